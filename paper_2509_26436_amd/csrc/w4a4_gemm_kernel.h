// W4A4 GEMM with in-register decode and CDNA4 fp8 MFMA: the kernel template
// (internal header; each output mode is instantiated in a translation unit of
// its own, w4a4_gemm_<mode>.hip, so they compile in parallel).
//
// For each 64-element K-group g the block stages its tiles of packed 4-bit
// activations (codes + per-subgroup FLAG + fp16 scale) and packed 4-bit
// weights (codes + fp16 scale) from global memory, decodes them in registers
// to OCP fp8 e4m3 operands -- activations as c * 2^FLAG in [-112, 112],
// weights as wq in [-7, 7], both exact in e4m3 -- and writes them to LDS
// (double-buffered: group g+1 is decoded while group g is multiplied).  Each
// wave then runs v_mfma_f32_32x32x64_f8f6f4 over the whole group, which yields
// the exact integer group product P_g (every partial sum is an integer below
// 2^24), and folds it into fp32 accumulators with the two group scales:
//   acc += P_g * (s_a[m,g] * s_w[n,g]).
// The 32 x 32 tile of scale products s_a (x) s_w is itself produced by one
// fp16 MFMA with a single non-zero k (fp16 x fp16 is exact in fp32), so the
// per-group dequantization costs one FMA per output element.
// The epilogue adds the bias, applies the optional GELU (tanh form) and
// stores bf16 (round to nearest even).
//
// The vector ALU is the scarce unit (one FMA per output and group, plus the
// decode), and one wave alone cannot issue it back to back, so the work is
// split by wave: per SIMD two "math" waves run only the MFMAs and the
// dequantization FMAs while a third "decode" wave streams the next group in
// (buffer loads, nibble -> fp8 decode, LDS stores).  Their instruction
// streams are independent, so the SIMD interleaves them.  All global
// addressing is scalar: buffer loads whose resource base advances by one
// group per iteration.
#pragma once

#include <algorithm>
#include <atomic>
#include <type_traits>

#include "gemm_schedule.h"
#include "lzs_device.h"
#include "quartz_internal.h"

namespace quartz {
namespace {


typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

// Buffer resource word 3 for raw (untyped, stride 0) loads on gfx9: a load at
// an offset >= num_records returns zero instead of touching memory.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

// GELU, tanh form: 0.5 v (1 + tanh(u)) with u = sqrt(2/pi) (v + 0.044715 v^3).
// Since 1 + tanh(u) = 2 / (1 + e^(-2u)), this equals v / (1 + 2^(w v)) with
// w = -2 log2(e) sqrt(2/pi) (1 + 0.044715 v^2): one hardware exp2 and one
// reciprocal instead of a tanh (relative error of a few fp32 ulps, far inside
// the output tolerance).  For large |u| the power saturates to 0 or +inf and
// the quotient to v or 0, the limits of GELU.
__device__ __forceinline__ float gelu_tanh(float v)
{
    constexpr float c0 = -2.0f * 1.4426950408889634f * 0.7978845608028654f;
    constexpr float c1 = c0 * 0.044715f;
    const float w = __builtin_fmaf(c1, v * v, c0);
    const float e = __builtin_amdgcn_exp2f(w * v);
    return v * __builtin_amdgcn_rcpf(1.0f + e);
}

// ------------------------------------------------------------------ layout
// Block tile BM x BN = 256 x 128.  12 waves: waves 0-7 are math waves as
// 4 (M) x 2 (N), wave tile 64 x 64 = 2 x 2 MFMA tiles of 32 x 32; waves 8-11
// are decode waves.  Waves are placed on the 4 SIMDs round robin, so each
// SIMD holds two math waves and one decode wave.
constexpr int BM = (int)kGemmBlockRows;
constexpr int BN = (int)kGemmBlockCols;
constexpr int kMathWaves = 8;
constexpr int kDecodeWaves = 4;
constexpr int kThreadsPerBlock = 64 * (kMathWaves + kDecodeWaves);
constexpr int kDecodeThreads = 64 * kDecodeWaves;
// The static whole-tile kernel's math waves fit in 128 registers, which
// leaves room for two decode waves per SIMD (16 waves): each decode thread
// then takes half an activation row and a quarter weight column, and the
// decode chain of a step is split over twice the waves.
constexpr int kSplitDecodeWaves = 8;
constexpr int kSplitThreadsPerBlock = 64 * (kMathWaves + kSplitDecodeWaves);
constexpr int WAVES_N = 2;
constexpr int WM = 64;
constexpr int WN = 64;
constexpr int TM = WM / 32;
constexpr int TN = WN / 32;
constexpr int kPanelsPerBlock = BN / kPanel;
constexpr int kStages = 3;

// 16-byte chunk c of decoded fp8 row r lives at chunk c ^ f(r) with
//   f(r) = (r1 ^ r2) | (r2 ^ r3) << 1      (r_i = bit i of r).
// Fragment reads (16 consecutive rows, one chunk) then touch distinct
// 16-byte bank groups within every 128-byte and every 256-byte window.
__device__ __forceinline__ int swz(int r, int c)
{
    const int f = (((r >> 1) ^ (r >> 2)) & 1) | ((((r >> 2) ^ (r >> 3)) & 1) << 1);
    return r * 64 + ((c ^ f) << 4);
}

// Workgroup barrier ordering LDS only: global loads still in flight (the
// prefetch ring) are not drained; their registers are waited on at first use.
__device__ __forceinline__ void lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The 64 / GS flag bytes of one (group, row), loaded as is and turned into
// decode tables only when the group is decoded, so the prefetch never waits
// for them.
template <int GS>
using FlagRaw = typename std::conditional<GS == 8, uint2,
                typename std::conditional<GS == 16, uint32_t, uint16_t>::type>::type;

template <int GS>
__device__ __forceinline__ FlagRaw<GS> load_flags_raw(Rsrc r, uint32_t off)
{
    if constexpr (GS == 8)
        return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
    else if constexpr (GS == 16)
        return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
    else if constexpr (GS == 32)
        return __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
    else
        return __builtin_amdgcn_raw_buffer_load_b8(r, (int)off, 0, 0);
}

// The decode table of flag k (byte k of the raw flags: bytes 0-3 in `lo`, 4-7
// in `hi`): FLAG replicated into every byte by one v_perm_b32 (selector 0x0C
// yields 0x00, which keeps the entry of magnitude 0 at zero), then shifted
// into the e4m3 exponent field and added to the base table in one
// v_lshl_add_u32 per dword (FLAG <= 4, so 8 FLAG stays inside its byte and
// no entry carries into the next).
template <int K>
__device__ __forceinline__ Fp8Table fp8_table_raw(uint32_t lo, uint32_t hi)
{
    static_assert(K >= 0 && K < 8, "flag byte");
    constexpr uint32_t rep = 0x01010101u * K;
    constexpr uint32_t rep_lo = (0x01010100u * K) | 0x0Cu;
    Fp8Table t;
    t.lo = (__builtin_amdgcn_perm(hi, lo, rep_lo) << 3) + kTabLo;
    t.hi = (__builtin_amdgcn_perm(hi, lo, rep) << 3) + kTabHi;
    return t;
}

// ATTN: the flags of half h of a B row (one activation row of 64 / G_s flag
// bytes): its first 32 elements are flags [0, 32 / G_s), the second half the
// rest (G_s = 64: the row's single flag covers both halves).  Returned in the
// low bytes of a dword, flag k of the half in byte k.
template <int GS>
__device__ __forceinline__ uint32_t load_half_flags(Rsrc r, uint32_t row_off, int h)
{
    if constexpr (GS == 8)
        return __builtin_amdgcn_raw_buffer_load_b32(r, (int)(row_off + 4u * (uint32_t)h), 0, 0);
    else if constexpr (GS == 16)
        return __builtin_amdgcn_raw_buffer_load_b16(r, (int)(row_off + 2u * (uint32_t)h), 0, 0);
    else if constexpr (GS == 32)
        return __builtin_amdgcn_raw_buffer_load_b8(r, (int)(row_off + (uint32_t)h), 0, 0);
    else
        return __builtin_amdgcn_raw_buffer_load_b8(r, (int)row_off, 0, 0);
}

template <int GS>
__device__ __forceinline__ uint2 flags_dwords(FlagRaw<GS> raw)
{
    if constexpr (GS == 8)
        return raw;
    else
        return uint2{(uint32_t)raw, 0u};
}

// One math wave's 64 x 64 bf16 output tile, staged in LDS by the epilogue
// that quantizes the output for the next layer (quantize_tile_out), addressed
// through LDS-typed pointers.
constexpr int kTransposeBytes = WM * WN * 2;
typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef __attribute__((address_space(3))) uint16_t lds_u16;
typedef __attribute__((address_space(3))) v4u lds_v4u;

// One math wave's 64 x 64 output tile (2 x 2 MFMA tiles of 32 x 32: lane l
// holds column l % 32, rows 8 (r/4) + 4 khalf + r%4 of register r) as the bf16
// values of the plain epilogue, fmaf(acc, cs[j], b[j]) then the optional
// GELU, written row-major into the wave's LDS region tb (8 KB, 128 bytes per
// row).  Row r's 16-byte chunk c (its elements 8c..8c+7) sits at chunk
// c ^ ((r >> 1) & 7) (tile_chunk_offset): the column-per-lane writes of one
// row, and a read of one chunk per row by 16 consecutive lanes (8 chunk
// positions x 2 row parities), both cover all 64 banks.  The caller waits for
// the writes before reading them back (the wave reads only its own region).
__device__ __forceinline__ uint32_t tile_chunk_offset(uint32_t row, uint32_t c)
{
    return row * 128u + ((c ^ ((row >> 1) & 7u)) << 4);
}

template <bool GELU>
__device__ __forceinline__ void stage_tile_bf16(const v16f (&out)[2][2], const float (&cs)[2],
                                                const float (&b)[2], lds_u8* tb, int lane)
{
    const uint32_t lane2 = (uint32_t)lane * 2u;
    typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
    typedef float f2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float v0 = fmaf(out[i][0][r], cs[0], b[0]);
            float v1 = fmaf(out[i][1][r], cs[1], b[1]);
            if constexpr (GELU) {
                v0 = gelu_tanh(v0);
                v1 = gelu_tanh(v1);
            }
            // after the swap lane l holds column l of rows row0, row0 + 4
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0),
                                                             __float_as_uint(v1), false, false);
            const f2 pair = {__uint_as_float(sw[0]), __uint_as_float(sw[1])};
            const uint32_t pk = __builtin_bit_cast(uint32_t, __builtin_convertvector(pair, bf2));
            const int row0 = i * 32 + 8 * (r >> 2) + (r & 3);
            const uint32_t x0 = (uint32_t)((row0 >> 1) & 7) << 4;
            const uint32_t x1 = (uint32_t)(((row0 + 4) >> 1) & 7) << 4;
            *(lds_u16*)(tb + row0 * 128 + (lane2 ^ x0)) = (uint16_t)pk;
            *(lds_u16*)(tb + (row0 + 4) * 128 + (lane2 ^ x1)) = (uint16_t)(pk >> 16);
        }
    }
}

// ---- output quantized for the next layer: one math wave's 64 x 64 tile (2 x 2
// MFMA tiles of 32 x 32: lane l holds column l % 32, rows 8 (r/4) + 4 khalf
// + r%4 of register r) becomes the bf16 values the plain epilogue would store,
// fmaf(acc, cs[j], b[j]) then the optional GELU, run through the activation
// quantizer with this layer's N as the next layer's K.  The wave's 64 columns
// are one 64-group of each of its 64 rows (N % 64 == 0).  The bf16 tile goes
// through the wave's own LDS region tb (stage_tile_bf16) and comes back one
// row per lane, so the group maximum, the subgroup ORs and the code packing
// are in-lane arithmetic (lzs_device.h); a chunk is one 8-element block.  The
// row is read once; per block the |q| pairs go back over the block's chunk
// (so they need no registers while the subgroup FLAGs are formed) and are
// read again for the code words.
// Outputs, K-group-major with g = column / 64: codes [g][M][32], flags
// [g][M][64 / lzs], scales [g][M], zeros [g][M]; rows past M fall outside the
// buffer ranges and are dropped.
template <bool GELU>
__device__ __forceinline__ void quantize_tile_out(const v16f (&out)[2][2], const float (&cs)[2],
                                                  const float (&b)[2], lds_u8* tb, int lane,
                                                  int64_t row_base, int64_t col_base, int64_t M,
                                                  int64_t N, const QuantOut& qout)
{
    if (col_base >= N)
        return;                              // wave-uniform
    stage_tile_bf16<GELU>(out, cs, b, tb, lane);
    // the wave reads back only what it wrote itself: LDS order within the
    // wave suffices, the clobber keeps the compiler's order
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    lds_u8* const row = tb + lane * 128;
    const uint32_t rx = (uint32_t)((lane >> 1) & 7) << 4;
    auto chunk = [&](int c) { return (lds_v4u*)(row + (((uint32_t)c << 4) ^ rx)); };
    uint32_t X[8][4];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const v4u v = *chunk(c);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            X[c][k] = v[k];
    }
    // max |x| on the bf16 magnitude bits (their unsigned order is the order
    // of |x|), two values per instruction
    lzs_us2 m2 = {0, 0};
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
        for (int k = 0; k < 4; ++k)
            m2 = __builtin_elementwise_max(m2, __builtin_bit_cast(lzs_us2, X[c][k] & 0x7FFF7FFFu));
    const uint32_t am = max((uint32_t)m2[0], (uint32_t)m2[1]);
    const GroupScale gsc = group_scale(__uint_as_float(am << 16));
    // |q| pairs of each 8-element block (written back over its chunk), their
    // OR and the sign bits; one branch for the wave
    uint32_t S[8], m8[8];
    auto pairs = [&](auto clamp) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            uint32_t p[4];
            mag_pairs8_t<decltype(clamp)::value>(X[c], gsc.r, p);
            m8[c] = pairs_or(p);
            S[c] = sign_nibbles(X[c]);
            *chunk(c) = v4u{p[0], p[1], p[2], p[3]};
        }
    };
    if (__builtin_amdgcn_ballot_w64(gsc.clamp))
        pairs(std::integral_constant<bool, true>());
    else
        pairs(std::integral_constant<bool, false>());
    // FLAG per block: the OR over its subgroup, built by OR-ing the blocks at
    // distance 1, 2 and 4 under wave-uniform masks that keep only partners in
    // the same subgroup
    const int qgs = qout.lzs;
    const uint32_t k16 = qgs >= 16 ? ~0u : 0u, k32 = qgs >= 32 ? ~0u : 0u, k64 = qgs >= 64 ? ~0u : 0u;
    uint32_t o1[8], o2[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
        o1[k] = m8[k] | (m8[k ^ 1] & k16);
#pragma unroll
    for (int k = 0; k < 8; ++k)
        o2[k] = o1[k] | (o1[k ^ 2] & k32);
    int fl[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
        fl[k] = lzs_flag(o2[k] | (o2[k ^ 4] & k64));
    // code words from the stored pairs
    uint32_t w[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const v4u v = *chunk(c);
        const uint32_t p[4] = {v[0], v[1], v[2], v[3]};
        w[c] = lzs_word(p, S[c], fl[c]);
    }

    const int64_t g = col_base / 64;
    const int64_t rg0 = g * M + row_base;           // (group, first row)
    const uint32_t rows_in = (uint32_t)max((int64_t)0, min(M - row_base, (int64_t)64));
    const Rsrc rc = make_rsrc(qout.codes + rg0 * 32, rows_in * 32u);
    __builtin_amdgcn_raw_buffer_store_b128(v4u{w[0], w[1], w[2], w[3]}, rc, lane * 32, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b128(v4u{w[4], w[5], w[6], w[7]}, rc, lane * 32 + 16, 0, 0);
    const uint32_t fb = (uint32_t)(64 / qgs);
    const Rsrc rf = make_rsrc(qout.flags + rg0 * fb, rows_in * fb);
    if (qgs == 8) {
        const uint32_t lo = fl[0] | fl[1] << 8 | fl[2] << 16 | fl[3] << 24;
        const uint32_t hi = fl[4] | fl[5] << 8 | fl[6] << 16 | fl[7] << 24;
        __builtin_amdgcn_raw_buffer_store_b64(v2u{lo, hi}, rf, lane * 8, 0, 0);
    } else if (qgs == 16) {
        __builtin_amdgcn_raw_buffer_store_b32(
            (uint32_t)(fl[0] | fl[2] << 8 | fl[4] << 16 | fl[6] << 24), rf, lane * 4, 0, 0);
    } else if (qgs == 32) {
        __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(fl[0] | fl[4] << 8), rf, lane * 2, 0, 0);
    } else {
        __builtin_amdgcn_raw_buffer_store_b8((uint8_t)fl[0], rf, lane, 0, 0);
    }
    const Rsrc rs = make_rsrc(qout.scales + rg0, rows_in * 2u);
    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)gsc.s16, rs, lane * 2, 0, 0);
    if (qout.zeros) {
        const Rsrc rz = make_rsrc(qout.zeros + rg0, rows_in);
        __builtin_amdgcn_raw_buffer_store_b8((uint8_t)0, rz, lane, 0, 0);
    }
}

// Decode roles (decode thread d = tid - 512, 0..255): A row d (32 code bytes,
// the row's 64 / G_s flags, s_a) and B column d/2, half d%2 (16 code bytes);
// threads d < 128 also carry s_w of column d.  Rows past M and columns past
// the packed panels fall outside the buffer ranges and read as zero: they
// only feed outputs that are never stored, so nothing needs a bounds check.
//
// Persistent workgroups: each one walks its segments (gemm_schedule.h) as a
// single pipeline.  The decode waves fetch and decode across segment
// boundaries without a break, so while the math waves write one tile's
// output the next tile's first groups are already being staged.  SPLIT
// instantiations carry the partial-sum code of shared tiles.
// STATIC instantiations are the LDM setting (the experimental-details
// appendix): one per-tensor activation scale and per-channel weight scales,
// so the K loop has no per-group scales at all: the fp8 MFMAs accumulate the
// exact integer sum in place and the epilogue applies act_scale * s_w[n].
// CONV instantiations are a 3 x 3 convolution (stride 1, padding 1) as an
// implicit GEMM (ConvGeom): codes, flags and scales are those of the feature
// map [M][C], and the A row of output pixel m for K-group g is the row of the
// pixel shifted by g's tap, read from channel block g % cg, or zero where the
// tap falls outside the image.  Every 64-group of an im2col row lies within
// one tap (C % 64 == 0), and a group's codes, FLAGs and scale depend on its
// 64 values only, so these are exactly the codes of the im2col matrix.
// ATTN instantiations are the two products of LZS attention: the B operand
// is itself an LZS-quantized activation (codes, FLAGs and fp16 scales in the
// quantizer's K-group-major layout, AttnGeom), decoded with its own FLAG
// tables like A, and A and B address one head's rows inside the arrays of
// all heads (plane stride and row offset).  With OUT32 the output is fp32,
// y32 = acc * scale (the scores); otherwise the bf16 output of the layer.
template <int GS, bool I32OUT, bool GELU, bool SPLIT, bool STATIC, bool CONV = false,
          bool ATTN = false, bool OUT32 = false>
__global__ __launch_bounds__(STATIC && !SPLIT ? kSplitThreadsPerBlock : kThreadsPerBlock) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ codes, const uint8_t* __restrict__ flags,
    const uint16_t* __restrict__ scales, const uint8_t* __restrict__ w_packed,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ yi,
    int64_t M, int64_t N, int64_t K, int64_t ldy, GemmSchedule sch,
    uint32_t* __restrict__ counters, float* __restrict__ slots, float act_scale, ConvGeom conv,
    AttnGeom attn)
{
    // per-group scales are staged and applied only by the per-group kernels
    constexpr bool kGroupScales = !I32OUT && !STATIC;
    // three LDS stages: group g + 2 is decoded into one while the math waves
    // read the operands of group g + 1 from another (and multiply group g
    // from registers)
    // One LDS array holds the operand stages, at the lowest addresses, where
    // every fragment address of the main loop is a lane offset plus an
    // immediate (a larger array placed first would push them past the 16-bit
    // immediate range and cost a register per stage).
    constexpr int kStageBytes = kStages * (BM + BN) * 64;
    __shared__ __attribute__((aligned(16))) uint8_t lds_main[kStageBytes];
    uint8_t (*const As)[BM * 64] = reinterpret_cast<uint8_t (*)[BM * 64]>(lds_main);
    uint8_t (*const Bs)[BN * 64] = reinterpret_cast<uint8_t (*)[BN * 64]>(lds_main + kStages * BM * 64);
    // group scales as fp16 bits; entries BM (BN) stay 0: the upper half-wave's
    // k = 8 operand slot of the outer-product MFMA reads them
    __shared__ uint16_t sas[kStages][BM + 8];
    __shared__ uint16_t sws[kStages][BN + 8];

    constexpr int FB = 64 / GS;                           // flag bytes per (group, row)
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int uwave = __builtin_amdgcn_readfirstlane(wave);
    const bool decoder = uwave >= kMathWaves;

    // Values that must not stay live across the loops pass through opaque
    // copies where they are used: the schedule (so the compiler re-derives
    // the reciprocals of its divisors per segment, a few scalar instructions,
    // instead of hoisting them into registers) and the thread index (so
    // per-lane indices are recomputed after each tile's output code instead
    // of occupying registers the main loop needs).
    auto fresh_schedule = [&] {
        GemmSchedule s = sch;
        asm volatile("" : "+s"(s.tiles_n), "+s"(s.groups), "+s"(s.blocks), "+s"(s.sk_first),
                          "+s"(s.sk_q), "+s"(s.sk_r), "+s"(s.sk_blocks), "+s"(s.sk_tiles));
        return s;
    };
    auto fresh_tid = [&] {
        int t = tid;
        asm volatile("" : "+v"(t));
        return t;
    };

    // ------------------------------------------------------ decode waves
    if (decoder) {
        static_assert(kDecodeThreads == BM && kDecodeThreads == 2 * BN, "decode roles");
        static_assert(64 * kSplitDecodeWaves == 2 * BM && 64 * kSplitDecodeWaves == 4 * BN,
                      "split decode roles");
        // STATIC whole-tile kernels: thread d decodes half ah of A row d / 2
        // and quarter bq of B column d / 4; otherwise all of A row d and half
        // bh of column d / 2 (the split kernels' partial-sum code needs more
        // than 128 registers)
        constexpr bool kSplit = STATIC && !SPLIT;
        const int d = tid - kMathWaves * 64;      // decode thread index
        const int dr = kSplit ? (d >> 1) & (BM - 1) : d & (BM - 1);   // A row
        const int ah = kSplit ? d & 1 : 0;                             // A half
        const int bc = kSplit ? (d >> 2) & (BN - 1) : (d >> 1) & (BN - 1);   // B column
        const int bh = kSplit ? d & 3 : d & 1;                         // B half / quarter
        const int swc = d & (BN - 1);             // column whose s_w this thread loads
        const int G = (int)(K / 64);
        const int64_t panels = (N + kPanel - 1) / kPanel;
        const uint32_t b_off =
            (uint32_t)((bc / kPanel) * G * kChunkBytes + (bc % kPanel) * 32 + bh * (kSplit ? 8 : 16));
        const uint32_t sw_off =
            (uint32_t)((swc / kPanel) * G * kChunkBytes + kChunkCodeBytes + (swc % kPanel) * 2);

        // fetch cursor: segment fc, step fg of it (steps past its groups are
        // no-ops), and the buffer ranges of its tile
        const int32_t blk = (int32_t)blockIdx.x;
        GemmCursor fc;
        int fg = 0, fend = 0;
        bool fdone = false;
        int64_t m0 = 0, panel0 = 0;
        uint32_t a_bytes = 0, s_bytes = 0, b_bytes = 0;
        // CONV: image row and column of this thread's output pixel m0 + dr
        // (M < 2^26, so 32-bit arithmetic holds)
        int conv_h = 0, conv_w = 0;
        auto set_ranges = [&] {
            m0 = (int64_t)fc.tm * BM;
            panel0 = (int64_t)fc.tn * (BN / kPanel);
            const int64_t rows = min(M - m0, (int64_t)BM);
            a_bytes = (uint32_t)(rows * 32);
            s_bytes = (uint32_t)(rows * 2);
            const int64_t blk_panels = min(panels - panel0, (int64_t)kPanelsPerBlock);
            b_bytes = (uint32_t)((blk_panels - 1) * G * kChunkBytes + kChunkBytes);
            if constexpr (CONV) {
                const uint32_t m = (uint32_t)m0 + (uint32_t)dr;
                const uint32_t q = m / (uint32_t)conv.W;
                conv_w = (int)(m - q * (uint32_t)conv.W);
                conv_h = (int)(q % (uint32_t)conv.H);
            }
        };
        if (!cursor_begin(fresh_schedule(), blk, fc))
            return;
        fg = fc.sg.g0;
        fend = fc.sg.g0 + padded_steps(fc.sg.g1 - fc.sg.g0);
        set_ranges();

        struct Raw {
            uint4 a0, a1;
            uint4 b;
            FlagRaw<GS> f;
            uint32_t fb;             // ATTN: flags of this thread's half B row
            uint16_t sa, sw;
        };
        // fetch the cursor's group into r, then advance the cursor by one step.
        // A no-op step (and any step past the end) reloads the segment's last
        // group: every step issues the same loads, so the compiler can wait
        // for exactly the ring slot being decoded (a conditional load would
        // make it wait for all of them), and staging the copy is harmless
        // since the stage a step writes is never read by another step.
        auto fetch_next = [&](Raw& r) {
            const int g = min(fg, fc.sg.g1 - 1);
            // A rows of group g: a plane of the K-group-major arrays, its first
            // row, the rows the buffer ranges cover, and this thread's row in
            // it (in == false: offset 2^31, outside every range, reads zero)
            int64_t plane = g, row0 = m0;
            uint32_t range_rows = a_bytes / 32, lrow = (uint32_t)dr;
            bool in = true;
            if constexpr (CONV) {
                // the channel block's whole plane, addressed by the pixel
                // that g's tap shifts this output pixel to
                const uint32_t tap = conv.cg == 1 ? (uint32_t)g : __umulhi((uint32_t)g, conv.div_magic);
                const int dh = (int)(tap / 3u) - 1, dw = (int)(tap % 3u) - 1;
                plane = g - (int)tap * conv.cg;
                row0 = 0;
                range_rows = (uint32_t)M;
                lrow = (uint32_t)((int)m0 + dr + dh * conv.W + dw);
                in = (uint32_t)(conv_h + dh) < (uint32_t)conv.H && (uint32_t)(conv_w + dw) < (uint32_t)conv.W;
            }
            const int64_t prow = ATTN ? plane * attn.a_plane + attn.a_row0 + row0 : plane * M + row0;
            const Rsrc ra = make_rsrc(codes + prow * 32, range_rows * 32u);
            const Rsrc rf = make_rsrc(flags + prow * FB, range_rows * (uint32_t)FB);
            const uint32_t ao = in ? lrow * 32u + (uint32_t)(ah * 16) : 0x80000000u;
            const uint32_t fo = in ? lrow * (uint32_t)FB : 0x80000000u;
            // ATTN: B rows n0 .. n0 + BN - 1 of group g's plane of the B
            // activation arrays (bh_rows of them inside N)
            const int64_t n0 = panel0 * kPanel;
            const int64_t bprow = (int64_t)g * attn.b_plane + attn.b_row0 + n0;
            const uint32_t bh_rows = (uint32_t)min(max(N - n0, (int64_t)0), (int64_t)BN);
            const Rsrc rb = ATTN ? make_rsrc(attn.b_codes + bprow * 32, bh_rows * 32u)
                                 : make_rsrc(w_packed + (panel0 * G + g) * kChunkBytes, b_bytes);
            r.a0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ra, (int)ao, 0, 0));
            if constexpr (kSplit)
                r.a1 = make_uint4(0, 0, 0, 0);
            else
                r.a1 = __builtin_bit_cast(uint4,
                                      __builtin_amdgcn_raw_buffer_load_b128(ra, (int)ao + 16, 0, 0));
            r.f = load_flags_raw<GS>(rf, fo);
            if constexpr (kSplit) {
                const uint2 b2 = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rb, (int)b_off, 0, 0));
                r.b = make_uint4(b2.x, b2.y, 0, 0);
            } else {
                r.b = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                                    rb, (int)(ATTN ? (uint32_t)(bc * 32 + bh * 16) : b_off), 0, 0));
            }
            if constexpr (kGroupScales) {   // the integer and static paths have none
                const Rsrc rs = make_rsrc(scales + prow, range_rows * 2u);
                r.sa = __builtin_amdgcn_raw_buffer_load_b16(rs, in ? (int)(lrow * 2u) : (int)0x80000000u, 0, 0);
                if constexpr (ATTN) {
                    const Rsrc rbs = make_rsrc(attn.b_scales + bprow, bh_rows * 2u);
                    r.sw = __builtin_amdgcn_raw_buffer_load_b16(rbs, swc * 2, 0, 0);
                } else {
                    r.sw = __builtin_amdgcn_raw_buffer_load_b16(rb, (int)sw_off, 0, 0);
                }
            } else {
                r.sa = 0;
                r.sw = 0;
            }
            if constexpr (ATTN) {
                const Rsrc rbf = make_rsrc(attn.b_flags + bprow * FB, bh_rows * (uint32_t)FB);
                r.fb = load_half_flags<GS>(rbf, (uint32_t)(bc * FB), bh);
            } else {
                r.fb = 0;
            }
            if (!fdone && ++fg == fend) {
                if (cursor_next(fresh_schedule(), blk, fc)) {
                    fg = fc.sg.g0;
                    fend = fc.sg.g0 + padded_steps(fc.sg.g1 - fc.sg.g0);
                    set_ranges();
                } else {
                    fdone = true;
                }
            }
        };
        // decode one group into LDS buffer `buf`
        auto stage = [&](const Raw& r, int buf) {
            uint2 fr = flags_dwords<GS>(r.f);
            if constexpr (kSplit) {
                // the half row's flags first: half ah starts at word 4 ah,
                // flag 4 ah / (G_s / 8)
                if constexpr (GS == 8) {
                    fr = ah ? uint2{fr.y, 0u} : fr;
                } else if constexpr (GS == 16) {
                    fr.x >>= 16 * ah;
                } else if constexpr (GS == 32) {
                    fr.x >>= 8 * ah;
                }
            }
            const uint32_t a[8] = {r.a0.x, r.a0.y, r.a0.z, r.a0.w, r.a1.x, r.a1.y, r.a1.z, r.a1.w};
            constexpr int kWordsPerFlag = GS / 8;
            constexpr int kChunks = kSplit ? 2 : 4;   // 16-byte fp8 chunks of the row this thread writes
            Fp8Table t = fp8_table_raw<0>(fr.x, fr.y);
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
                uint2 w[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int wi = 2 * c + h;           // word index within the thread's words
                    if (wi % kWordsPerFlag == 0 && wi > 0) {
                        switch (wi / kWordsPerFlag) {      // flag index, 1..7
                        case 1: t = fp8_table_raw<1>(fr.x, fr.y); break;
                        case 2: t = fp8_table_raw<2>(fr.x, fr.y); break;
                        case 3: t = fp8_table_raw<3>(fr.x, fr.y); break;
                        case 4: t = fp8_table_raw<4>(fr.x, fr.y); break;
                        case 5: t = fp8_table_raw<5>(fr.x, fr.y); break;
                        case 6: t = fp8_table_raw<6>(fr.x, fr.y); break;
                        default: t = fp8_table_raw<7>(fr.x, fr.y); break;
                        }
                    }
                    w[h] = decode_nibbles_fp8(a[wi], t);
                }
                *reinterpret_cast<uint4*>(As[buf] + swz(dr, kSplit ? 2 * ah + c : c)) =
                    make_uint4(w[0].x, w[0].y, w[1].x, w[1].y);
            }
            if constexpr (ATTN) {
                // the half B row's 4 words with the FLAG tables of its
                // subgroups (word w: flag w / (G_s / 8) of the half)
                const uint32_t bw[4] = {r.b.x, r.b.y, r.b.z, r.b.w};
                uint2 o[4];
                const Fp8Table t0 = fp8_table_raw<0>(r.fb, 0u);
                if constexpr (GS == 8) {
                    o[0] = decode_nibbles_fp8(bw[0], t0);
                    o[1] = decode_nibbles_fp8(bw[1], fp8_table_raw<1>(r.fb, 0u));
                    o[2] = decode_nibbles_fp8(bw[2], fp8_table_raw<2>(r.fb, 0u));
                    o[3] = decode_nibbles_fp8(bw[3], fp8_table_raw<3>(r.fb, 0u));
                } else if constexpr (GS == 16) {
                    const Fp8Table t1 = fp8_table_raw<1>(r.fb, 0u);
                    o[0] = decode_nibbles_fp8(bw[0], t0);
                    o[1] = decode_nibbles_fp8(bw[1], t0);
                    o[2] = decode_nibbles_fp8(bw[2], t1);
                    o[3] = decode_nibbles_fp8(bw[3], t1);
                } else {
#pragma unroll
                    for (int w = 0; w < 4; ++w)
                        o[w] = decode_nibbles_fp8(bw[w], t0);
                }
                *reinterpret_cast<uint4*>(Bs[buf] + swz(bc, 2 * bh)) = make_uint4(o[0].x, o[0].y, o[1].x, o[1].y);
                *reinterpret_cast<uint4*>(Bs[buf] + swz(bc, 2 * bh + 1)) = make_uint4(o[2].x, o[2].y, o[3].x, o[3].y);
            }
            // weight words: e4m3 of wq * 2^-9 (weight_word_store)
            const uint2 b0 = decode_weight_fp8(r.b.x);
            const uint2 b1 = decode_weight_fp8(r.b.y);
            if constexpr (ATTN) {
            } else if constexpr (kSplit) {
                *reinterpret_cast<uint4*>(Bs[buf] + swz(bc, bh)) = make_uint4(b0.x, b0.y, b1.x, b1.y);
            } else {
                const uint2 b2 = decode_weight_fp8(r.b.z);
                const uint2 b3 = decode_weight_fp8(r.b.w);
                *reinterpret_cast<uint4*>(Bs[buf] + swz(bc, 2 * bh)) = make_uint4(b0.x, b0.y, b1.x, b1.y);
                *reinterpret_cast<uint4*>(Bs[buf] + swz(bc, 2 * bh + 1)) = make_uint4(b2.x, b2.y, b3.x, b3.y);
            }
            if constexpr (kGroupScales) {
                sas[buf][dr] = r.sa;
                if (d < BN)
                    sws[buf][swc] = r.sw;
            }
        };

        // The decode of each group is on the critical path of the next ones:
        // these waves run at issue priority above the math waves' VALU work.
        // They keep a register ring of three groups in flight and decode two
        // groups ahead of the math waves, one workgroup barrier per group
        // (plus one before the first), the same count the math waves execute.
        // The ring is deeper for the static kernel: its steps are short
        // (fp8 MFMAs only), so three steps of prefetch no longer cover the
        // load latency.  Its depth is a multiple of the stage count.
        constexpr int kRing = STATIC ? 2 * kStages : kStages;
        Raw ring[kRing];
        __builtin_amdgcn_s_setprio(2);
        if (d < 8 * kStages) {
            sas[d >> 3][BM + (d & 7)] = 0;
            sws[d >> 3][BN + (d & 7)] = 0;
        }
        const int steps = gemm_steps(fresh_schedule(), blk);
#pragma unroll
        for (int i = 0; i < kRing; ++i)
            fetch_next(ring[i]);
        stage(ring[0], 0);
        fetch_next(ring[0]);
        stage(ring[1], 1);
        fetch_next(ring[1]);
        lds_sync();
        // Step s (u = s mod kRing): decode step s + 2 (ring slot (s + 2) mod
        // kRing, LDS stage (s + 2) mod 3) and refill the slot with step
        // s + 2 + kRing.  Straight-line code, so the compiler waits only for
        // the slot being decoded.
        auto dstep = [&](int u) {
            const int k = (u + 2) % kRing;
            stage(ring[k], (u + 2) % kStages);
            fetch_next(ring[k]);
            lds_sync();
        };
        int s = 0;
        for (; s + kRing <= steps; s += kRing) {
#pragma unroll
            for (int u = 0; u < kRing; ++u)
                dstep(u);
        }
#pragma unroll
        for (int u = 0; u < kRing - 1; ++u)
            if (s + u < steps)
                dstep(u);
        return;
    }

    // -------------------------------------------------------- math waves
    // Per-lane fragment indices, recomputed from fresh_tid after every tile's
    // output code (see above).
    // The swizzle depends on row bits 1-3 only, so the fragments of tile row 1
    // (column tile 1) sit exactly 32 rows = 2048 bytes after those of tile row
    // 0 (column tile 0): one pair of lane offsets per operand, the rest are
    // immediate offsets of the LDS reads.
    int lane, wm, wn, l32, khalf;
    uint32_t a_lo, a_hi, b_lo, b_hi;
    auto set_fragment_indices = [&] {
        const int t = fresh_tid();
        const int w = __builtin_amdgcn_readfirstlane(t >> 6) & (kMathWaves - 1);   // wave-uniform
        lane = t & 63;
        wm = w / WAVES_N;
        wn = w % WAVES_N;
        l32 = t & 31;
        khalf = (t >> 5) & 1;
        a_lo = (uint32_t)swz(wm * WM + l32, 2 * khalf);
        a_hi = (uint32_t)swz(wm * WM + l32, 2 * khalf + 1);
        b_lo = (uint32_t)swz(wn * WN + l32, 2 * khalf);
        b_hi = (uint32_t)swz(wn * WN + l32, 2 * khalf + 1);
    };
    static_assert(((32 >> 1) & 7) == 0, "32-row steps keep the swizzle");
    auto frag_at = [](const uint8_t* stage, uint32_t lo, uint32_t hi, int rows_off) {
        const uint4 l = *reinterpret_cast<const uint4*>(stage + lo + rows_off * 64);
        const uint4 h = *reinterpret_cast<const uint4*>(stage + hi + rows_off * 64);
        return v8i{(int)l.x, (int)l.y, (int)l.z, (int)l.w, (int)h.x, (int)h.y, (int)h.z, (int)h.w};
    };

    v16f acc[TM][TN];

    // Operands of the group being multiplied, held in registers; each one is
    // refilled with the next group's (from LDS stage nb) right after its last
    // use, so the LDS reads overlap the MFMAs instead of stalling the next
    // group's first MFMA.
    // a single weight-fragment register set: column 0 (prefetched) for tiles
    // (0,0) (1,0), then column 1, read from the current stage once column 0's
    // last product is issued
    // Operands of the scale outer-product MFMA (fp16, K = 16 with only k = 0
    // non-zero): dword 0 holds the scale in its low half (a zero-extending
    // 16-bit LDS load; the upper half-wave reads the zero pad, its k = 8), and
    // dwords 1-3 are zero once and never written again, so refilling an
    // operand is one LDS load and no packing instruction.
    // The split instantiation keeps the scales as plain fp16 values and packs
    // the operand per MFMA instead: its output code between segments (partial
    // sums) needs the 16 registers more than its main loop needs the saved
    // instructions (measured: 2.5 % either way).
    typedef int v4i __attribute__((ext_vector_type(4)));
    constexpr bool kKeepScaleOps = !SPLIT && kGroupScales;
    v8i bf, af[TM];
    v4i sa_op[TM], sw_op[TN];
    _Float16 sa_h[TM], sw_h[TN];
    auto load_a = [&](int i, int buf) {
        af[i] = frag_at(As[buf], a_lo, a_hi, i * 32);
        if constexpr (kGroupScales) {
            const uint16_t v = sas[buf][khalf ? BM : wm * WM + i * 32 + l32];
            if constexpr (kKeepScaleOps)
                sa_op[i][0] = (int)v;
            else
                sa_h[i] = __builtin_bit_cast(_Float16, v);
        }
    };
    auto load_b = [&](int j, int buf) {
        bf = frag_at(Bs[buf], b_lo, b_hi, j * 32);
        if constexpr (kGroupScales) {
            const uint16_t v = sws[buf][khalf ? BN : wn * WN + j * 32 + l32];
            if constexpr (kKeepScaleOps)
                sw_op[j][0] = (int)v;
            else
                sw_h[j] = __builtin_bit_cast(_Float16, v);
        }
    };

    // One group, tiles in the order (0,0) (1,0) (0,1) (1,1).  The fp8 product
    // of each tile is issued one step ahead: step t issues the scale MFMA of
    // tile t, then the FMAs of tile t (which wait only for the short scale
    // MFMA) with the fp8 MFMA of tile t + 1 issued between their two halves,
    // so the matrix unit works on the next product meanwhile and the other
    // math wave's MFMAs can slot in between.  The first product of a group is issued
    // right after the barrier, and the last tile's FMAs follow it (its
    // results stay live across the barrier).  Operands are prefetched for
    // the next group after their last use.  The asm statement pins each
    // tile's FMAs (without a use, LLVM sinks them to the end of the loop).
    static_assert(TM == 2 && TN == 2, "prefetch order assumes 2 x 2 tiles");
    v16f p_next, p_last, s_last;       // product of the next tile; last tile's P and S
    const v16f zero = {};
    // I32OUT: acc holds int32 bit patterns and each exact group product is
    // converted and added in int32, so the sum over K stays exact beyond 2^24
    // (|P_g| <= 50176 converts exactly; |sum| <= 784 K < 2^31 for K <= 2^20).
    auto add_i32 = [](float a, float p) {
        return __int_as_float(__float_as_int(a) + (int)(p * kWeightUnitInv));
    };
    auto fma_tile = [&](int i, int j, const v16f& p, const v16f& sc) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            if constexpr (I32OUT)
                acc[i][j][r] = add_i32(acc[i][j][r], p[r]);
            else
                acc[i][j][r] = fmaf(p[r], sc[r], acc[i][j][r]);
        }
        asm volatile("" : "+v"(acc[i][j]));
    };
    auto scale_tile = [&](int i, int j) {
        v16f sc = zero;
        if constexpr (!I32OUT) {
            typedef _Float16 v8h __attribute__((ext_vector_type(8)));
            v8h a, b;
            if constexpr (kKeepScaleOps) {
                a = __builtin_bit_cast(v8h, sa_op[i]);
                b = __builtin_bit_cast(v8h, sw_op[j]);
            } else {
                a = v8h{};
                b = v8h{};
                a[0] = sa_h[i];
                b[0] = sw_h[j];
            }
            __builtin_amdgcn_s_setprio(3);
            sc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, zero, 0, 0, 0);
            __builtin_amdgcn_s_setprio(0);
        }
        return sc;
    };
    // MFMA issue runs at raised wave priority (above the decode waves): the
    // matrix unit is the resource to keep fed, and a math wave whose MFMA is
    // held back also holds back the FMAs behind it.
    auto mfma_p = [&](int i, int j) {
        (void)j;
        __builtin_amdgcn_s_setprio(3);
        const v16f p = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[i], bf, zero, 0, 0, 0, 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
        return p;
    };
    auto fma_rows = [&](int i, int j, const v16f& p, const v16f& sc, int r0) {
#pragma unroll
        for (int r = r0; r < r0 + 8; ++r) {
            if constexpr (I32OUT)
                acc[i][j][r] = add_i32(acc[i][j][r], p[r]);
            else
                acc[i][j][r] = fmaf(p[r], sc[r], acc[i][j][r]);
        }
        asm volatile("" : "+v"(acc[i][j]));
    };
    // one group from LDS stage cb; the next group's operands are prefetched
    // from stage nb unless this is the last group of a segment (LAST)
    // STATIC: both weight columns in registers (bq), each fp8 MFMA adds its
    // product to the tile's accumulators in place (exact: every partial sum
    // is an integer; see include/quartz.h for the K range), and the operands
    // of the next group are read from stage nb after their last use here.
    v8i bq[TN];
    auto load_bq = [&](int j, int buf) { bq[j] = frag_at(Bs[buf], b_lo, b_hi, j * 32); };
    auto compute_static = [&](int cb, int nb, auto last) {
        constexpr bool LAST = decltype(last)::value;
        (void)cb;
        __builtin_amdgcn_s_setprio(3);
        acc[0][0] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[0], bq[0], acc[0][0], 0, 0, 0, 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[1], bq[0], acc[1][0], 0, 0, 0, 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
        if (!LAST)
            load_bq(0, nb);
        __builtin_amdgcn_s_setprio(3);
        acc[0][1] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[0], bq[1], acc[0][1], 0, 0, 0, 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
        if (!LAST)
            load_a(0, nb);
        __builtin_amdgcn_s_setprio(3);
        acc[1][1] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[1], bq[1], acc[1][1], 0, 0, 0, 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
        if (!LAST) {
            load_a(1, nb);
            load_bq(1, nb);
        }
    };
    auto compute = [&](int cb, int nb, auto last) {
        if constexpr (STATIC) {
            compute_static(cb, nb, last);
            return;
        }
        constexpr bool LAST = decltype(last)::value;
        // product of tile 0, then the last tile of the previous group
        p_next = mfma_p(0, 0);
        __builtin_amdgcn_sched_barrier(0);
        fma_tile(TM - 1, TN - 1, p_last, s_last);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < TM * TN; ++t) {
            // step t: scale MFMA of tile t, half of tile t's FMAs, fp8 MFMA of
            // tile t + 1, operand refills, the other half of the FMAs (so a
            // wave never issues two MFMAs back to back)
            const int i = t % TM, j = t / TM;
            const v16f p = p_next;
            const v16f sc = scale_tile(i, j);
            __builtin_amdgcn_sched_barrier(0);
            if (t + 1 < TM * TN)
                fma_rows(i, j, p, sc, 0);
            __builtin_amdgcn_sched_barrier(0);
            if (t + 1 < TM * TN)
                p_next = mfma_p((t + 1) % TM, (t + 1) / TM);
            __builtin_amdgcn_sched_barrier(0);
            // refills after the last use of each operand: af[i] by the product of
            // tile (i,1) (issued one step ahead), sa_op[i] by the scale of tile
            // (i,1), bf / sw_op[0] by column 0's products and scales
            if (t == 0)
                load_b(1, cb);          // column 1 of this group (column 0's products are issued)
            if (t == 2 && !LAST) {
                load_a(0, nb);
                load_b(0, nb);          // column 0 of the next group
            }
            if (t == 3 && !LAST)
                load_a(1, nb);
            __builtin_amdgcn_sched_barrier(0);
            if (t + 1 < TM * TN) {
                fma_rows(i, j, p, sc, 8);
            } else {
                p_last = p;
                s_last = sc;
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // The math waves' barrier: their own outstanding LDS reads (the prefetch)
    // may cross it, since the stage they read is not rewritten until two
    // barriers later; the memory clobber keeps the compiler from moving LDS
    // accesses across it.
    auto math_barrier = [] { asm volatile("s_barrier" ::: "memory"); };

    // the first n groups of a segment (its first group is in LDS stage 0),
    // each followed by the next one's operand prefetch
    using NotLast = std::integral_constant<bool, false>;
    auto run_groups = [&](int n) {
        int g = 0;
        for (; g + kStages <= n; g += kStages) {
#pragma unroll
            for (int u = 0; u < kStages; ++u) {
                compute(u, (u + 1) % kStages, NotLast());
                math_barrier();
            }
        }
#pragma unroll
        for (int u = 0; u < kStages - 1; ++u) {
            if (g + u < n) {
                compute(u, (u + 1) % kStages, NotLast());
                math_barrier();
            }
        }
    };

    GemmCursor cur;
    const int32_t blk = (int32_t)blockIdx.x;
    // this lane's bias values of the current tile (bf16 bits), loaded when the
    // segment starts so that the output code does not wait for them
    // STATIC: also the channel scales s_w[n] of its columns (fp16 bits, from
    // the scale slot of group 0 in the packed weight)
    uint16_t bias_bits[TN], cscale_bits[TN];
    auto load_bias = [&] {
        if constexpr (!I32OUT) {
            const Rsrc rb = make_rsrc(bias, bias ? (uint32_t)(N * 2) : 0u);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bias_bits[j] = __builtin_amdgcn_raw_buffer_load_b16(
                    rb, (int)(((int64_t)cur.tn * BN + wn * WN + j * 32 + l32) * 2), 0, 0);
        }
        if constexpr (STATIC) {
            // the wave's 64 columns are one panel: its group-0 chunk
            const int64_t panel = (int64_t)cur.tn * (BN / kPanel) + wn;
            const Rsrc rs = make_rsrc(w_packed + panel * (K / 64) * kChunkBytes + kChunkCodeBytes,
                                      panel < (N + kPanel - 1) / kPanel ? (uint32_t)(kPanel * 2) : 0u);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                cscale_bits[j] = __builtin_amdgcn_raw_buffer_load_b16(rs, (j * 32 + l32) * 2, 0, 0);
        }
    };
    // the value of acc before bias and activation: acc times 2^9 (its unit is
    // that of the weight operands), or for STATIC the integer sum times
    // act_scale * s_w[n] (the 2^9 folded into cs)
    float cs[TN];
    auto set_out_scale = [&] {
        if constexpr (STATIC) {
#pragma unroll
            for (int j = 0; j < TN; ++j)
                cs[j] = act_scale * (float)__builtin_bit_cast(_Float16, cscale_bits[j]) * kWeightUnitInv;
        }
    };
    // acc is in units of the weight operands (2^-9, see decode_weight_fp8)
    // except for ATTN, whose B operand is an activation: the factor 2^9 is
    // exact, so fmaf(a, 2^9, b) rounds exactly like the sum of the unscaled
    // accumulator and the bias
    auto out_value = [&](float a, int j, float bj) {
        if constexpr (STATIC)
            return fmaf(a, cs[j], bj);
        else if constexpr (ATTN)
            return a + bj;
        else
            return fmaf(a, kWeightUnitInv, bj);
    };
    // ---- output.  Lane l holds column l % 32 of each 32 x 32 tile, rows
    // 8 (r/4) + 4 khalf + r%4 of register r.
    auto store_tile = [&](const v16f (&out)[TM][TN]) {
        if constexpr (OUT32) {
            // fp32 y32[row][ldy] = acc * scale; lane l holds column l % 32,
            // so each store instruction writes two rows' 32 consecutive floats
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int64_t col = (int64_t)cur.tn * BN + wn * WN + j * 32 + l32;
                if (col >= N)
                    continue;
#pragma unroll
                for (int i = 0; i < TM; ++i) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int64_t row = (int64_t)cur.tm * BM + wm * WM + i * 32 + 8 * (r >> 2) + 4 * khalf + (r & 3);
                        if (row < M)
                            attn.y32[row * ldy + col] = out[i][j][r] * attn.scale;
                    }
                }
            }
        } else if constexpr (I32OUT) {
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int64_t col = (int64_t)cur.tn * BN + wn * WN + j * 32 + l32;
                if (col >= N)
                    continue;
#pragma unroll
                for (int i = 0; i < TM; ++i) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int64_t row = (int64_t)cur.tm * BM + wm * WM + i * 32 + 8 * (r >> 2) + 4 * khalf + (r & 3);
                        if (row < M)
                            yi[row * N + col] = __float_as_int(out[i][j][r]);
                    }
                }
            }
        } else {
            // bias and activation per element, then one lane-half swap between the
            // two column tiles: afterwards lane l holds column l of the wave's 64
            // columns for one row (tile 0's rows in the first register, tile 1's
            // khalf = 1 rows in the second), so every store covers a full 128-byte
            // row segment; the pair is rounded to bf16 (RNE) by one conversion.
            // Stores go through one buffer range per wave (its 64 rows from its
            // first column), with the whole offset, row included, in the lane
            // operand: the bounds check covers that operand and the immediate
            // only, never the scalar one.  Rows past M then fall outside the
            // range and are dropped, and lanes whose column is past N start
            // at 2^31, outside it for every row (the range is at most 2^31
            // bytes: 64 rows of at most 2^25).
            static_assert(TN == 2, "the swap pairs the two column tiles");
            set_out_scale();
            const int64_t row_base = (int64_t)cur.tm * BM + wm * WM;
            const int64_t col_base = (int64_t)cur.tn * BN + wn * WN;
            float b[TN];
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[j] = __uint_as_float((uint32_t)bias_bits[j] << 16);
            const int64_t rows_in = max((int64_t)0, min(M - row_base, (int64_t)WM));
            const uint32_t row_bytes = (uint32_t)ldy * 2u;
            const Rsrc out_r = make_rsrc(y + row_base * ldy + col_base, (uint32_t)rows_in * row_bytes);
            const uint32_t voff = col_base + lane < N ? (uint32_t)lane * 2u : 0x80000000u;
            typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
            typedef float f2 __attribute__((ext_vector_type(2)));
#pragma unroll
            for (int i = 0; i < TM; ++i) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float v0 = out_value(out[i][0][r], 0, b[0]);
                    float v1 = out_value(out[i][1][r], 1, b[1]);
                    if constexpr (GELU) {
                        v0 = gelu_tanh(v0);
                        v1 = gelu_tanh(v1);
                    }
                    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0),
                                                                     __float_as_uint(v1), false, false);
                    const f2 pair = {__uint_as_float(sw[0]), __uint_as_float(sw[1])};
                    const uint32_t pk = __builtin_bit_cast(uint32_t, __builtin_convertvector(pair, bf2));
                    const uint32_t row0 = (uint32_t)(i * 32 + 8 * (r >> 2) + (r & 3));
                    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)pk, out_r,
                                                          (int)(voff + row0 * row_bytes), 0, 0);
                    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(pk >> 16), out_r,
                                                          (int)(voff + (row0 + 4) * row_bytes), 0, 0);
                }
            }
        }
    };

    // Partial sums of a shared tile.  Each math wave handles its own 64 x 64
    // region independently: it stores its registers to its slot (float4 runs
    // in register order, 1 KB per instruction), waits until those stores are
    // complete, and counts itself in the region's counter.  The wave that
    // completes the count adds every contributor's slot in workgroup order,
    // so the result does not depend on which one arrives last, resets the
    // counter for the next call and writes the output.  Nobody waits for
    // another wave.
    // Coherence across the XCDs' separate L2 caches comes from the accesses
    // themselves, not from fences: slot stores and loads carry the sc1 cache
    // policy (device-coherent: the stores write through, the loads do not
    // hit stale lines), the same instructions the compiler emits for relaxed
    // device-scope atomic loads and stores, and the counter is a device-scope
    // atomic.  A device-scope release / acquire fence would instead write back
    // and invalidate the whole L2 of the XCD (buffer_wbl2 / buffer_inv),
    // evicting the operands of every other workgroup on it.  Ordering: the
    // stores are waited for (vmcnt) before the counter increment, and the
    // finisher issues its loads only after the increment has returned.
    constexpr int kRegionFloats = WM * WN;
    constexpr int kCoherent = 16;      // sc1 cache-policy bit of buffer loads / stores
    auto slot_rsrc = [&](int slot) {
        return make_rsrc(slots + ((int64_t)slot * kMathWaves + uwave) * kRegionFloats,
                         kRegionFloats * (uint32_t)sizeof(float));
    };
    typedef float v4f __attribute__((ext_vector_type(4)));
    // Returns true for the wave that completes the region (acc then holds
    // the whole sum and the caller writes the output).
    auto finish_partial = [&]() -> bool {
        if constexpr (SPLIT && !I32OUT) {
            const uint32_t lane_off = (uint32_t)lane * 16u;
            const Rsrc mine = slot_rsrc(cur.sg.slot);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const v4f v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                       acc[i][j][4 * q + 3]};
                        __builtin_amdgcn_raw_buffer_store_b128(
                            v, mine, (int)(lane_off + ((i * TN + j) * 4 + q) * 1024), 0, kCoherent);
                    }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            uint32_t* ctr = counters + (int64_t)cur.sg.sk_tile * kMathWaves + uwave;
            uint32_t arrived = 0;
            if (lane == 0)
                arrived = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            arrived = __builtin_amdgcn_readfirstlane(arrived);
            const GemmSchedule sch_ = fresh_schedule();
            int32_t b_first, b_last;
            sk_contributors(sch_, cur.sg.sk_tile, b_first, b_last);
            if (arrived != (uint32_t)(b_last - b_first))
                return false;
            asm volatile("" ::: "memory");
            if (b_last - b_first == 1) {
                // two contributors (the usual case): add the other one's slot
                // to the registers; a + b == b + a in floating point, so the
                // result is the same whichever of the two finishes
                const int32_t other = b_first == blk ? b_last : b_first;
                const Rsrc part = slot_rsrc(sk_slot(sch_, other, cur.sg.sk_tile));
                // in two halves (tile row i), to bound the registers in flight
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    v4f v[TN][4];
#pragma unroll
                    for (int j = 0; j < TN; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            v[j][q] = __builtin_amdgcn_raw_buffer_load_b128(
                                part, (int)(lane_off + ((i * TN + j) * 4 + q) * 1024), 0, kCoherent);
#pragma unroll
                    for (int j = 0; j < TN; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q)
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                acc[i][j][4 * q + e] += v[j][q][e];
                    __builtin_amdgcn_sched_barrier(0);
                }
                if (lane == 0)
                    __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                return true;
            }
            // more contributors: acc = sum of their slots in workgroup order
            // (this wave's own slot included, re-read: it holds the same values),
            // per 32 x 32 tile, with two contributors' loads in flight at a time
            // (a lone slot read per step left the finisher waiting on each
            // round trip in turn)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int toff = (int)(lane_off + (i * TN + j) * 4 * 1024);
                    for (int32_t bb = b_first; bb <= b_last; bb += 2) {
                        const bool two = bb < b_last;
                        v4f va[4], vb[4];
                        const Rsrc pa = slot_rsrc(sk_slot(sch_, bb, cur.sg.sk_tile));
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            va[q] = __builtin_amdgcn_raw_buffer_load_b128(pa, toff + q * 1024, 0, kCoherent);
                        if (two) {
                            const Rsrc pb = slot_rsrc(sk_slot(sch_, bb + 1, cur.sg.sk_tile));
#pragma unroll
                            for (int q = 0; q < 4; ++q)
                                vb[q] = __builtin_amdgcn_raw_buffer_load_b128(pb, toff + q * 1024, 0, kCoherent);
                        }
#pragma unroll
                        for (int q = 0; q < 4; ++q)
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                if (bb == b_first)
                                    acc[i][j][4 * q + e] = va[q][e];
                                else
                                    acc[i][j][4 * q + e] += va[q][e];
                                if (two)
                                    acc[i][j][4 * q + e] += vb[q][e];
                            }
                    }
                }
            if (lane == 0)
                __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return true;
        }
        return false;
    };

    auto reset_tile = [&] {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc[i][j][r] = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            p_last[r] = 0.0f;          // the "last tile" before a segment's first group adds 0
            s_last[r] = 0.0f;
        }
    };

    // Segment by segment: the first group's operands are read from LDS stage
    // 0, the groups but the last run with the next group's prefetch, the last
    // one prefetches nothing (so no operand is live across the output code),
    // the no-op steps that round the segment up to whole 3-step rounds are
    // barriers only, then the tile's output.  The decode waves meanwhile
    // stage the next segment's first groups.
    if (!cursor_begin(fresh_schedule(), blk, cur))
        return;
    if constexpr (kKeepScaleOps) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
            sa_op[i] = v4i{0, 0, 0, 0};
#pragma unroll
        for (int j = 0; j < TN; ++j)
            sw_op[j] = v4i{0, 0, 0, 0};
    }
    lds_sync();
    for (;;) {
        const int L = cur.sg.g1 - cur.sg.g0;
        set_fragment_indices();
        load_bias();
        reset_tile();
        load_a(0, 0);
        load_a(1, 0);
        if constexpr (STATIC) {
            load_bq(0, 0);
            load_bq(1, 0);
        } else {
            load_b(0, 0);
        }
        run_groups(L - 1);
        compute((L - 1) % kStages, 0, std::integral_constant<bool, true>());
        math_barrier();
        for (int p = L; p < padded_steps(L); ++p)
            math_barrier();
        if constexpr (!STATIC)
            fma_tile(TM - 1, TN - 1, p_last, s_last);
        set_fragment_indices();
        // one output call site, so the epilogue is inlined once
        if (!SPLIT || cur.sg.sk_tile < 0 || finish_partial())
            store_tile(acc);
        if (!cursor_next(fresh_schedule(), blk, cur))
            break;
    }
}

template <bool B>
using bool_c = std::integral_constant<bool, B>;

// Launch of one output mode, every G_s / epilogue / split combination of it.
template <bool I32OUT, bool STATIC, bool CONV = false, bool ATTN = false, bool OUT32 = false>
hipError_t launch_mode(const GemmLaunch& a, hipStream_t stream)
{
    const dim3 grid((unsigned)a.sch.blocks);
    const dim3 block(STATIC && a.sch.sk_tiles == 0 ? kSplitThreadsPerBlock : kThreadsPerBlock);
    auto go = [&](auto gs, auto gelu, auto split) {
        w4a4_gemm_kernel<decltype(gs)::value, I32OUT, decltype(gelu)::value, decltype(split)::value,
                         STATIC, CONV, ATTN, OUT32><<<grid, block, 0, stream>>>(
            a.codes, a.flags, a.scales, a.w_packed, a.bias, a.y, a.yi, a.M, a.N, a.K, a.ldy, a.sch,
            a.counters, a.slots, a.act_scale, a.conv, a.attn);
    };
    auto with_split = [&](auto gs, auto gelu) {
        if (!I32OUT && !OUT32 && a.sch.sk_tiles > 0)
            go(gs, gelu, bool_c<!I32OUT && !OUT32>());
        else
            go(gs, gelu, bool_c<false>());
    };
    auto with_gelu = [&](auto gs) {
        if (!I32OUT && !ATTN && a.epilogue == 1)
            with_split(gs, bool_c<!I32OUT && !ATTN>());
        else
            with_split(gs, bool_c<false>());
    };
    switch (a.lzs_group) {
    case 8:
        with_gelu(std::integral_constant<int, 8>());
        break;
    case 16:
        with_gelu(std::integral_constant<int, 16>());
        break;
    case 32:
        with_gelu(std::integral_constant<int, 32>());
        break;
    default:
        with_gelu(std::integral_constant<int, 64>());
        break;
    }
    return hipGetLastError();
}

}  // namespace
}  // namespace quartz
