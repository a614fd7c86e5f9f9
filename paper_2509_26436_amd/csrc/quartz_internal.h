// Internal declarations shared by the HIP sources of libquartz.so (not part of
// the public ABI; see include/quartz.h for that).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "gemm_schedule.h"

namespace quartz {

// Packed weight layout: panels of kPanel output columns.  For each (panel p,
// group g), in [panel][group] order, one chunk of kPanel * 32 bytes of codes
// (column-major within the panel: column c's 64 codes at c * 32, eight per
// 32-bit weight word, see weight_word_store) followed by kPanel fp16 scales.
constexpr int kGroup = 64;
constexpr int kPanel = 64;
constexpr int kChunkCodeBytes = kPanel * kGroup / 2;          // 2048
constexpr int kChunkBytes = kChunkCodeBytes + kPanel * 2;     // 2176

inline int64_t packed_weight_bytes(int64_t N, int64_t K)
{
    const int64_t panels = (N + kPanel - 1) / kPanel;
    return panels * (K / kGroup) * kChunkBytes;
}

// Output tile per GEMM workgroup, and the most tiles one GEMM may have (the
// schedule indexes them with 32-bit integers; an output that large would not
// fit in device memory anyway).
constexpr int64_t kGemmBlockRows = 256;
constexpr int64_t kMaxGemmTiles = (int64_t(1) << 31) - 1;
constexpr int64_t kGemmBlockCols = 128;

// ---------------------------------------------------------------- launchers
// Each returns hipSuccess or the launch error.  Arguments are validated by the
// C-ABI layer before these are called.
hipError_t launch_quantize_act(const uint16_t* x, int64_t M, int64_t K, int64_t ldx,
                               int lzs_group, uint8_t* codes, uint8_t* flags,
                               uint16_t* scales, int8_t* zeros, bool asymmetric,
                               hipStream_t stream);

hipError_t launch_pack_weight(const uint16_t* w, int64_t N, int64_t K, uint8_t* w_packed,
                              uint16_t* w_scales, hipStream_t stream);

hipError_t launch_weight_group_sums(const uint8_t* w_packed, int64_t N, int64_t K,
                                    int16_t* sums, hipStream_t stream);

hipError_t launch_unpack_weight(const uint8_t* w_packed, int64_t N, int64_t K, int8_t* wq,
                                hipStream_t stream);

// Work schedule of the GEMM for a persistent grid of at most `blocks`
// workgroups (split: tiles of the last rounds may be cut along K, which needs
// a workspace; s.blocks == 0 when there is nothing to launch or blocks <= 0),
// its workspace size (0 when no tile is split) and the persistent grid size
// of the current device (CUs x resident workgroups per CU; 0 if there is no
// device).
GemmSchedule gemm_schedule(int64_t M, int64_t N, int64_t K, int blocks, bool split);
// the same for tiles of bm x bn
GemmSchedule gemm_schedule_tiles(int64_t M, int64_t N, int64_t K, int blocks, bool split,
                                 int64_t bm, int64_t bn);
// The per-group linear layer with a bf16 output runs its own kernel
// (w4a4_linear.hip, tiles of 128 x 256): its schedule, its persistent grid
// size on the current device, and its launch (a.sch from linear_schedule).
GemmSchedule linear_schedule(int64_t M, int64_t N, int64_t K, int blocks, bool split);
int linear_resident_blocks();
size_t gemm_workspace_bytes(const GemmSchedule& s);
int gemm_resident_blocks();
// bytes of the workspace's counter part (its start); the slots follow it
size_t gemm_counter_bytes(const GemmSchedule& s);

// The device scratch array of quartz_w4a4_linear_noalloc (scratch.hip): its
// size, its address on the current device (resolved once per device), and
// the fill kernel that zeroes its first counter_bytes on `stream`.
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(void** ptr);
hipError_t clear_noalloc_counters(void* ptr, size_t counter_bytes, hipStream_t stream);

// Compute units of the current device (queried once per device and cached;
// 256 if the query fails): the grid-stride kernels size their grids by it.
int device_compute_units();

// Destination of an output quantized for the next layer (its K is this
// layer's N): the arrays of quartz_quantize_act with M rows and N / 64
// groups; codes == nullptr means a plain bf16 output.
struct QuantOut {
    uint8_t* codes;
    uint8_t* flags;
    uint16_t* scales;
    int8_t* zeros;       // may be nullptr
    int32_t lzs;         // LZS subgroup size of the output: 8, 16, 32 or 64
};

// Geometry of a 3 x 3 convolution (stride 1, padding 1) run as an implicit
// GEMM: rows are output pixels m = (image * H + h) * W + w, the K-group g is
// tap t = g / cg (kh = t / 3, kw = t % 3) and channel block g % cg of the
// pixel (h + kh - 1, w + kw - 1), zero outside the image.  div_magic =
// floor(2^32 / cg) + 1 gives g / cg = mulhi(g, div_magic) for every g < 2^14
// (unused when cg == 1).  cg == 0: a plain GEMM.
struct ConvGeom {
    int32_t H, W;
    int32_t cg;            // C / 64
    uint32_t div_magic;
};

// The two products of LZS attention (ATTN kernels): B is an LZS-quantized
// activation, b_codes [G][b_plane][32], b_flags [G][b_plane][64/G_s],
// b_scales [G][b_plane] with the GEMM's rows n at plane row b_row0 + n; A's
// rows m are plane row a_row0 + m of planes of a_plane rows.  y32 and scale:
// the fp32 output of the scores (y32[m][ldy] = acc * scale), else unused.
struct AttnGeom {
    const uint8_t* b_codes;
    const uint8_t* b_flags;
    const uint16_t* b_scales;
    int64_t a_plane, a_row0, b_plane, b_row0;
    float* y32;
    float scale;
};

// Arguments of one GEMM launch (see the kernel template in w4a4_gemm_kernel.h).
struct GemmLaunch {
    const uint8_t* codes;
    const uint8_t* flags;
    const uint16_t* scales;
    const uint8_t* w_packed;
    const uint16_t* bias;
    uint16_t* y;
    int32_t* yi;
    int64_t M, N, K, ldy;
    int lzs_group;
    int epilogue;
    GemmSchedule sch;
    uint32_t* counters;
    float* slots;
    QuantOut qout;
    float act_scale;
    const int8_t* zeros;      // asymmetric mode only
    const int16_t* wsums;
    ConvGeom conv;            // implicit 3 x 3 convolution only
    AttnGeom attn;            // attention products only
};

// One output mode each (w4a4_gemm_<mode>.hip).
hipError_t launch_linear(const GemmLaunch& a, hipStream_t stream);
hipError_t launch_linear_static(const GemmLaunch& a, hipStream_t stream);
hipError_t launch_linear_asym(const GemmLaunch& a, hipStream_t stream);
hipError_t launch_gemm_i32(const GemmLaunch& a, hipStream_t stream);
hipError_t launch_gemm_conv(const GemmLaunch& a, hipStream_t stream);
hipError_t launch_gemm_conv_static(const GemmLaunch& a, hipStream_t stream);
hipError_t launch_gemm_attn_scores(const GemmLaunch& a, hipStream_t stream);
hipError_t launch_gemm_attn_pv(const GemmLaunch& a, hipStream_t stream);

// 3 x 3 convolution (stride 1, padding 1) as an implicit GEMM: codes, flags
// and scales of quartz_quantize_act for the feature map [images * H * W][C]
// (scales == nullptr: the static setting with act_scale and a per-channel
// packed weight), w_packed of the weight [N][9 C] with K ordered (kh, kw, c),
// y [images * H * W][ldy].
hipError_t launch_w4a4_conv3x3(const uint8_t* codes, const uint8_t* flags,
                               const uint16_t* scales, float act_scale, const uint8_t* w_packed,
                               const uint16_t* bias, uint16_t* y, int64_t images, int64_t H,
                               int64_t W, int64_t C, int64_t N, int64_t ldy, int lzs_group,
                               int epilogue, const GemmSchedule& sch, void* workspace,
                               hipStream_t stream);

// The asymmetric mode: zeros [K/64][M] from quartz_quantize_act, wsums
// [K/64][N] from launch_weight_group_sums.
hipError_t launch_w4a4_linear_asym(const uint8_t* codes, const uint8_t* flags,
                                   const uint16_t* scales, const int8_t* zeros,
                                   const uint8_t* w_packed, const int16_t* wsums,
                                   const uint16_t* bias, uint16_t* y, int64_t M, int64_t N,
                                   int64_t K, int64_t ldy, int lzs_group, int epilogue,
                                   const GemmSchedule& sch, void* workspace, hipStream_t stream);

// `workspace`: gemm_workspace_bytes(sch) bytes whose counter part is zero
// (left zero again by the launch); unused unless sch.sk_tiles > 0.  With
// qout.codes set, y is not written and N % 64 == 0.
hipError_t launch_w4a4_linear(const uint8_t* codes, const uint8_t* flags,
                              const uint16_t* scales, const uint8_t* w_packed,
                              const uint16_t* bias, uint16_t* y, int64_t M, int64_t N, int64_t K,
                              int64_t ldy, int lzs_group, int epilogue, const GemmSchedule& sch,
                              void* workspace, const QuantOut& qout, hipStream_t stream);

// The LDM setting: codes and flags of quartz_quantize_act_static, w_packed of
// the per-channel pack (the channel scale in every group's scale slot).
hipError_t launch_w4a4_linear_static(const uint8_t* codes, const uint8_t* flags, float act_scale,
                                     const uint8_t* w_packed, const uint16_t* bias, uint16_t* y,
                                     int64_t M, int64_t N, int64_t K, int64_t ldy, int lzs_group,
                                     int epilogue, const GemmSchedule& sch, void* workspace,
                                     hipStream_t stream);

hipError_t launch_quantize_act_static(const uint16_t* x, int64_t M, int64_t K, int64_t ldx,
                                      float scale, int lzs_group, uint8_t* codes,
                                      uint8_t* flags, hipStream_t stream);

hipError_t launch_pack_weight_per_channel(const uint16_t* w, int64_t N, int64_t K,
                                          uint8_t* w_packed, uint16_t* w_scales,
                                          hipStream_t stream);

hipError_t launch_w4a4_gemm_i32(const uint8_t* codes, const uint8_t* flags,
                                const uint8_t* w_packed, int32_t* acc, int64_t M, int64_t N,
                                int64_t K, int lzs_group, hipStream_t stream);

// LZS attention (attention.hip): V^T quantized along the keys from V
// [heads * L][ldv] (rows head * L + key) into codes [L/64][heads * d][32],
// flags [L/64][heads * d][64/G_s], scales [L/64][heads * d]; the row softmax of
// S [M][lds] (N columns) quantized into codes [N/64][M][32] ...; and the two
// products of one head (scores: fp32 s[Lq][lds] = scale * Q~ K~^T; PV: bf16
// o[Lq][ldo] = P~ V~, with a split workspace as for the linear layer).
hipError_t launch_quantize_vt(const uint16_t* v, int64_t heads, int64_t L, int64_t d, int64_t ldv,
                              int lzs_group, uint8_t* codes, uint8_t* flags, uint16_t* scales,
                              hipStream_t stream);
hipError_t launch_softmax_quantize(const float* S, int64_t M, int64_t N, int64_t lds, int lzs_group,
                                   uint8_t* codes, uint8_t* flags, uint16_t* scales,
                                   hipStream_t stream);
hipError_t launch_attn_scores(const uint8_t* qc, const uint8_t* qf, const uint16_t* qs,
                              int64_t q_plane, int64_t q_row0, const uint8_t* kc,
                              const uint8_t* kf, const uint16_t* ks, int64_t k_plane,
                              int64_t k_row0, int64_t Lq, int64_t Lk, int64_t d, int lzs_group,
                              float scale, float* s, int64_t lds, hipStream_t stream);
// LZS activation codes K-group-major -> fp8 e4m3 rows out[rows][K]
hipError_t launch_expand_fp8(const uint8_t* codes, const uint8_t* flags, int64_t rows, int64_t K,
                             int lzs_group, uint8_t* out, hipStream_t stream);
// fused LZS attention of all heads (d = 64 or 128) from the expanded operands
hipError_t launch_attention_fused(const uint8_t* qx, const uint16_t* qs, const uint8_t* kx,
                                  const uint16_t* ks, const uint8_t* vx, const uint16_t* vs,
                                  int64_t heads, int64_t L, int64_t d, int lzs_group, uint16_t* o,
                                  int64_t ldo, hipStream_t stream);
hipError_t launch_attn_pv(const uint8_t* pc, const uint8_t* pf, const uint16_t* ps,
                          const uint8_t* vc, const uint8_t* vf, const uint16_t* vs,
                          int64_t v_plane, int64_t v_row0, int64_t Lq, int64_t Lk, int64_t d,
                          int lzs_group, uint16_t* o, int64_t ldo, const GemmSchedule& sch,
                          void* workspace, hipStream_t stream);

// ------------------------------------------------------------ device helpers

// Nibble word -> 8 OCP fp8 e4m3 bytes of (+-|c|) * 2^flag.
// A word holds 8 sign-magnitude nibbles.  The result's low dword carries the
// values of nibbles 0, 2, 4, 6 (bytes 0..3) and its high dword those of
// nibbles 1, 3, 5, 7; weights and activations are decoded by this same
// routine, so the permutation of k it introduces is the same on both MFMA
// operands and leaves the dot product unchanged.
// |c| * 2^flag for |c| in 1..7 is exact in e4m3 (at most 3 significant bits,
// at most 112): the magnitudes index an 8-entry byte table (v_perm_b32)
// whose non-zero entries carry the exponent bias plus flag.
struct Fp8Table {
    uint32_t lo;   // e4m3 of 0, 1, 2, 3 (times 2^flag)
    uint32_t hi;   // e4m3 of 4, 5, 6, 7 (times 2^flag)
};

constexpr uint32_t kTabLo = 0x44403800u;
constexpr uint32_t kTabHi = 0x4E4C4A48u;

__device__ __forceinline__ uint2 decode_nibbles_fp8(uint32_t w, Fp8Table t)
{
    const uint32_t mag_even = w & 0x07070707u;
    const uint32_t mag_odd = (w >> 4) & 0x07070707u;
    uint2 r;
    r.x = __builtin_amdgcn_perm(t.hi, t.lo, mag_even) | ((w << 4) & 0x80808080u);
    r.y = __builtin_amdgcn_perm(t.hi, t.lo, mag_odd) | (w & 0x80808080u);
    return r;
}

// Weight words.  The pack writes each word of 8 sign-magnitude codes (the
// nibble word of decode_nibbles_fp8: byte i holds code E_i in its low nibble
// and O_i in its high nibble, E = elements 0, 4, 1, 5 and O = elements 2, 6,
// 3, 7 of the word's 8 consecutive k) with its sign bits moved: byte i keeps
// both magnitudes in bits 0-2 (E_i) and 4-6 (O_i), the sign of E_i in bit 7
// and the sign of O_(i-1 mod 4) in bit 3.  Then a mask gives the four E codes
// and a rotation by 4 bits plus the same mask the four O codes, each as the
// byte s * 128 + |c|: the OCP e4m3 subnormal of c * 2^-9, exact for |c| <= 7.
// A GEMM on these operands yields every weight product times 2^-9 exactly
// (all partial sums are integers times 2^-9), and the output code multiplies
// by 2^9 once (kWeightUnitInv), which is exact.
constexpr uint32_t kWeightCodeMask = 0x87878787u;
constexpr float kWeightUnitInv = 512.0f;     // 1 / 2^-9

__host__ __device__ __forceinline__ uint32_t rotl32(uint32_t x, int r)
{
    return (x << r) | (x >> (32 - r));
}

// nibble word (decode_nibbles_fp8 order) -> stored weight word
__host__ __device__ __forceinline__ uint32_t weight_word_store(uint32_t nib)
{
    return (nib & 0x77777777u) | ((nib & 0x08080808u) << 4) | rotl32(nib & 0x80808080u, 4);
}

// stored weight word -> nibble word
__host__ __device__ __forceinline__ uint32_t weight_word_nibbles(uint32_t w)
{
    return (w & 0x77777777u) | ((w & 0x80808080u) >> 4) | rotl32(w & 0x08080808u, 28);
}

// stored weight word -> 8 e4m3 bytes (of c * 2^-9) in the byte order of
// decode_nibbles_fp8 (E codes in the low dword, O codes in the high one)
__device__ __forceinline__ uint2 decode_weight_fp8(uint32_t w)
{
    return uint2{w & kWeightCodeMask, __builtin_amdgcn_alignbit(w, w, 4) & kWeightCodeMask};
}

}  // namespace quartz
