// W4A4 GEMM with in-register decode and CDNA4 fp8 MFMA.
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
#include <type_traits>

#include "quartz_internal.h"

namespace quartz {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

// Buffer resource word 3 for raw (untyped, stride 0) loads on gfx9: a load at
// an offset >= num_records returns zero instead of touching memory.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float v)
{
    uint32_t u = __float_as_uint(v);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
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

__device__ __forceinline__ v8i load_frag(const uint8_t* lds, int r, int khalf)
{
    const uint4 lo = *reinterpret_cast<const uint4*>(lds + swz(r, 2 * khalf));
    const uint4 hi = *reinterpret_cast<const uint4*>(lds + swz(r, 2 * khalf + 1));
    return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z,
               (int)hi.w};
}

// Workgroup barrier ordering LDS only: global loads still in flight (the
// prefetch ring) are not drained; their registers are waited on at first use.
__device__ __forceinline__ void lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The 64 / GS flag bytes of one (group, row), loaded as is; expanded to
// 8 * FLAG per 8-element word (words 0-3 in `lo`, 4-7 in `hi`, one per byte)
// only when the group is decoded, so the prefetch never waits for them.
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

template <int GS>
__device__ __forceinline__ uint2 expand_flags8(FlagRaw<GS> raw)
{
    uint2 f;
    if constexpr (GS == 8) {
        f = raw;
    } else if constexpr (GS == 16) {
        f.x = __builtin_amdgcn_perm(0u, raw, 0x01010000u);
        f.y = __builtin_amdgcn_perm(0u, raw, 0x03030202u);
    } else if constexpr (GS == 32) {
        f.x = __builtin_amdgcn_perm(0u, (uint32_t)raw, 0x00000000u);
        f.y = __builtin_amdgcn_perm(0u, (uint32_t)raw, 0x01010101u);
    } else {
        f.x = __builtin_amdgcn_perm(0u, (uint32_t)raw, 0x00000000u);
        f.y = f.x;
    }
    f.x <<= 3;      // FLAG <= 4, so 8 * FLAG stays inside its byte
    f.y <<= 3;
    return f;
}

// Decode roles (decode thread d = tid - 512, 0..255): A row d (32 code bytes,
// the row's 64 / G_s flags, s_a) and B column d/2, half d%2 (16 code bytes);
// threads d < 128 also carry s_w of column d.  Rows past M and columns past
// the packed panels fall outside the buffer ranges and read as zero: they
// only feed outputs that are never stored, so nothing needs a bounds check.
template <int GS, bool I32OUT, bool GELU>
__global__ __launch_bounds__(kThreadsPerBlock) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ codes, const uint8_t* __restrict__ flags,
    const uint16_t* __restrict__ scales, const uint8_t* __restrict__ w_packed,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ yi,
    int64_t M, int64_t N, int64_t K, int64_t ldy)
{
    // three LDS stages: group g + 2 is decoded into one while the math waves
    // read the operands of group g + 1 from another (and multiply group g
    // from registers)
    __shared__ __attribute__((aligned(16))) uint8_t As[kStages][BM * 64];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[kStages][BN * 64];
    // group scales as fp16 bits; entries BM (BN) stay 0: the upper half-wave's
    // k = 8 operand slot of the outer-product MFMA reads them
    __shared__ uint16_t sas[kStages][BM + 8];
    __shared__ uint16_t sws[kStages][BN + 8];

    constexpr int FB = 64 / GS;                           // flag bytes per (group, row)
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t m0 = (int64_t)blockIdx.y * BM;
    const int64_t n0 = (int64_t)blockIdx.x * BN;
    const int G = (int)(K / 64);
    const int uwave = __builtin_amdgcn_readfirstlane(wave);
    const bool decoder = uwave >= kMathWaves;

    // ------------------------------------------------------ decode waves
    static_assert(kDecodeThreads == BM && kDecodeThreads == 2 * BN, "decode roles");
    const int d = tid - kMathWaves * 64;          // decode thread index (math waves: < 0)
    const int dr = d & (BM - 1);                  // A row
    const int bc = (d >> 1) & (BN - 1);           // B column
    const int bh = d & 1;                         // B half
    const int swc = d & (BN - 1);                 // column whose s_w this thread loads
    const int64_t panels = (N + kPanel - 1) / kPanel;
    const int64_t panel0 = n0 / kPanel;
    const int64_t rows = min(M - m0, (int64_t)BM);
    const uint32_t a_bytes = (uint32_t)(rows * 32);
    const uint32_t f_bytes = (uint32_t)(rows * FB);
    const uint32_t s_bytes = (uint32_t)(rows * 2);
    const int64_t blk_panels = min(panels - panel0, (int64_t)kPanelsPerBlock);
    const uint32_t b_bytes = (uint32_t)((blk_panels - 1) * G * kChunkBytes + kChunkBytes);
    const uint32_t a_off = (uint32_t)(dr * 32);
    const uint32_t f_off = (uint32_t)(dr * FB);
    const uint32_t b_off = (uint32_t)((bc / kPanel) * G * kChunkBytes + (bc % kPanel) * 32 + bh * 16);
    const uint32_t sw_off =
        (uint32_t)((swc / kPanel) * G * kChunkBytes + kChunkCodeBytes + (swc % kPanel) * 2);

    struct Raw {
        uint4 a0, a1;
        uint4 b;
        FlagRaw<GS> f;
        uint16_t sa, sw;
    };
    auto fetch = [&](Raw& r, int g) {
        const Rsrc ra = make_rsrc(codes + ((int64_t)g * M + m0) * 32, a_bytes);
        const Rsrc rf = make_rsrc(flags + ((int64_t)g * M + m0) * FB, f_bytes);
        const Rsrc rb = make_rsrc(w_packed + (panel0 * G + g) * kChunkBytes, b_bytes);
        r.a0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ra, (int)a_off, 0, 0));
        r.a1 = __builtin_bit_cast(uint4,
                                  __builtin_amdgcn_raw_buffer_load_b128(ra, (int)a_off + 16, 0, 0));
        r.f = load_flags_raw<GS>(rf, f_off);
        r.b = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rb, (int)b_off, 0, 0));
        if constexpr (!I32OUT) {       // the integer path has no scales (scales == nullptr)
            const Rsrc rs = make_rsrc(scales + (int64_t)g * M + m0, s_bytes);
            r.sa = __builtin_amdgcn_raw_buffer_load_b16(rs, (int)(dr * 2), 0, 0);
            r.sw = __builtin_amdgcn_raw_buffer_load_b16(rb, (int)sw_off, 0, 0);
        } else {
            r.sa = 0;
            r.sw = 0;
        }
    };
    // decode one group into LDS buffer `buf`
    auto stage = [&](const Raw& r, int buf) {
        const uint2 fl8 = expand_flags8<GS>(r.f);
        const uint32_t a[8] = {r.a0.x, r.a0.y, r.a0.z, r.a0.w, r.a1.x, r.a1.y, r.a1.z, r.a1.w};
        constexpr int kWordsPerFlag = GS / 8;
        Fp8Table t = fp8_table<0>(fl8.x);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            uint2 w[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int wi = 2 * c + h;           // word index 0..7
                if (wi % kWordsPerFlag == 0 && wi > 0) {
                    const uint32_t f = wi < 4 ? fl8.x : fl8.y;
                    switch (wi & 3) {
                    case 0: t = fp8_table<0>(f); break;
                    case 1: t = fp8_table<1>(f); break;
                    case 2: t = fp8_table<2>(f); break;
                    default: t = fp8_table<3>(f); break;
                    }
                }
                w[h] = decode_nibbles_fp8(a[wi], t);
            }
            *reinterpret_cast<uint4*>(As[buf] + swz(dr, c)) = make_uint4(w[0].x, w[0].y, w[1].x, w[1].y);
        }
        const Fp8Table tw{kTabLo, kTabHi};
        const uint2 b0 = decode_nibbles_fp8(r.b.x, tw);
        const uint2 b1 = decode_nibbles_fp8(r.b.y, tw);
        const uint2 b2 = decode_nibbles_fp8(r.b.z, tw);
        const uint2 b3 = decode_nibbles_fp8(r.b.w, tw);
        *reinterpret_cast<uint4*>(Bs[buf] + swz(bc, 2 * bh)) = make_uint4(b0.x, b0.y, b1.x, b1.y);
        *reinterpret_cast<uint4*>(Bs[buf] + swz(bc, 2 * bh + 1)) = make_uint4(b2.x, b2.y, b3.x, b3.y);
        if constexpr (!I32OUT) {
            sas[buf][dr] = r.sa;
            if (d < BN)
                sws[buf][swc] = r.sw;
        }
    };

    // -------------------------------------------------------- math waves
    const int wm = (wave & (kMathWaves - 1)) / WAVES_N;
    const int wn = (wave & (kMathWaves - 1)) % WAVES_N;
    const int l32 = lane & 31;
    const int khalf = lane >> 5;
    int sa_idx[TM], sw_idx[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
        sa_idx[i] = khalf ? BM : wm * WM + i * 32 + l32;
#pragma unroll
    for (int j = 0; j < TN; ++j)
        sw_idx[j] = khalf ? BN : wn * WN + j * 32 + l32;

    v16f acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][j][r] = 0.0f;

    // Operands of the group being multiplied, held in registers; each one is
    // refilled with the next group's (from LDS stage nb) right after its last
    // use, so the LDS reads overlap the MFMAs instead of stalling the next
    // group's first MFMA.
    // a single weight-fragment register set: column 0 (prefetched) for tiles
    // (0,0) (1,0), then column 1, read from the current stage once column 0's
    // last product is issued
    v8i bf, af[TM];
    _Float16 sw_h[TN], sa_h[TM];
    auto load_a = [&](int i, int buf) {
        af[i] = load_frag(As[buf], wm * WM + i * 32 + l32, khalf);
        if constexpr (!I32OUT)
            sa_h[i] = __builtin_bit_cast(_Float16, sas[buf][sa_idx[i]]);
    };
    auto load_b = [&](int j, int buf) {
        bf = load_frag(Bs[buf], wn * WN + j * 32 + l32, khalf);
        if constexpr (!I32OUT)
            sw_h[j] = __builtin_bit_cast(_Float16, sws[buf][sw_idx[j]]);
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
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        p_last[r] = 0.0f;              // the "last tile" before the first group adds 0
        s_last[r] = 0.0f;
    }
    const v16f zero = {};
    auto fma_tile = [&](int i, int j, const v16f& p, const v16f& sc) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            if constexpr (I32OUT)
                acc[i][j][r] += p[r];
            else
                acc[i][j][r] = fmaf(p[r], sc[r], acc[i][j][r]);
        }
        asm volatile("" : "+v"(acc[i][j]));
    };
    auto scale_tile = [&](int i, int j) {
        v16f sc = zero;
        if constexpr (!I32OUT) {
            // fp16 operands of the scale outer product: only k = 0 is non-zero
            v8h sa_op = {}, sw_op = {};
            sa_op[0] = sa_h[i];
            sw_op[0] = sw_h[j];
            __builtin_amdgcn_s_setprio(3);
            sc = __builtin_amdgcn_mfma_f32_32x32x16_f16(sa_op, sw_op, zero, 0, 0, 0);
            __builtin_amdgcn_s_setprio(0);
        }
        return sc;
    };
    // MFMA issue runs at raised wave priority (above the decode waves): the
    // matrix unit is the resource to keep fed, and a math wave whose MFMA is
    // held back also holds back the FMAs behind it.
    auto mfma_p = [&](int i) {
        __builtin_amdgcn_s_setprio(3);
        const v16f p = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[i], bf, zero, 0, 0, 0, 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
        return p;
    };
    auto fma_rows = [&](int i, int j, const v16f& p, const v16f& sc, int r0) {
#pragma unroll
        for (int r = r0; r < r0 + 8; ++r) {
            if constexpr (I32OUT)
                acc[i][j][r] += p[r];
            else
                acc[i][j][r] = fmaf(p[r], sc[r], acc[i][j][r]);
        }
        asm volatile("" : "+v"(acc[i][j]));
    };
    auto compute = [&](int cb, int nb) {
        // product of tile 0, then the last tile of the previous group
        p_next = mfma_p(0);
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
                p_next = mfma_p((t + 1) % TM);
            __builtin_amdgcn_sched_barrier(0);
            // refills after the last use of each operand: af[i] by the product of
            // tile (i,1) (issued one step ahead), sa_h[i] by the scale of tile
            // (i,1), bf / sw_h[0] by column 0's products and scales
            if (t == 0)
                load_b(1, cb);          // column 1 of this group (column 0's products are issued)
            if (t == 2) {
                load_a(0, nb);
                load_b(0, nb);          // column 0 of the next group
            }
            if (t == 3)
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

    // ---- pipeline: decode waves keep a register ring of two groups in flight
    // and decode two groups ahead of the math waves.  The two roles run
    // separate loops with the same barriers (one before the first group and
    // one after each), so their registers never overlap in liveness.
    if (decoder) {
        Raw ring[2];
        // the decode of each group is on the critical path of the next ones:
        // give these waves issue priority over the math waves
        __builtin_amdgcn_s_setprio(2);
        if (d < 8 * kStages) {
            sas[d >> 3][BM + (d & 7)] = 0;
            sws[d >> 3][BN + (d & 7)] = 0;
        }
        fetch(ring[0], 0);
        fetch(ring[1], min(1, G - 1));
        stage(ring[0], 0);
        fetch(ring[0], min(2, G - 1));
        stage(ring[1], 1);
        fetch(ring[1], min(3, G - 1));
        lds_sync();
        // Iteration g: decode group g + 2 (ring slot g % 2) into stage
        // (g + 2) % 3 and refill the slot with group g + 4.  Straight-line
        // code with clamped prefetch indices (harmless reloads at the end),
        // so the compiler waits only for the slot being decoded.
        auto dstep = [&](int u, int g) {
            stage(ring[u & 1], (u + 2) % kStages);
            fetch(ring[u & 1], min(g + 4, G - 1));
            lds_sync();
        };
        constexpr int kU = 2 * kStages;
        int g = 0;
        for (; g + kU <= G; g += kU) {
#pragma unroll
            for (int u = 0; u < kU; ++u)
                dstep(u, g + u);
        }
#pragma unroll
        for (int u = 0; u < kU - 1; ++u)
            if (g + u < G)
                dstep(u, g + u);
        return;
    }
    lds_sync();
    load_a(0, 0);
    load_a(1, 0);
    load_b(0, 0);
    {
        // iteration g multiplies group g and prefetches group g + 1 from
        // stage (g + 1) % 3 (at the last group: a harmless read of a stale stage)
        int g = 0;
        for (; g + kStages <= G; g += kStages) {
#pragma unroll
            for (int u = 0; u < kStages; ++u) {
                compute(u % kStages, (u + 1) % kStages);
                math_barrier();
            }
        }
#pragma unroll
        for (int u = 0; u < kStages - 1; ++u) {
            if (g + u < G) {
                compute(u % kStages, (u + 1) % kStages);
                math_barrier();
            }
        }
    }

    fma_tile(TM - 1, TN - 1, p_last, s_last);

    // ---- epilogue.  Lane l holds column l % 32 of each 32 x 32 tile, rows
    // 8 (r/4) + 4 khalf + r%4 of register r.
    if constexpr (I32OUT) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int64_t col = n0 + wn * WN + j * 32 + l32;
            if (col >= N)
                continue;
#pragma unroll
            for (int i = 0; i < TM; ++i) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t row = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * khalf + (r & 3);
                    if (row < M)
                        yi[row * N + col] = (int32_t)acc[i][j][r];
                }
            }
        }
    } else {
        // bias and activation per element, then one lane-half swap between the
        // two column tiles: afterwards lane l holds column l of the wave's 64
        // columns for one row (tile 0's rows in the first register, tile 1's
        // khalf = 1 rows in the second), so every store covers a full 128-byte
        // row segment; the pair is rounded to bf16 (RNE) by one conversion
        static_assert(TN == 2, "the swap pairs the two column tiles");
        float b[TN] = {0.0f, 0.0f};
        if (bias) {
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int64_t c = n0 + wn * WN + j * 32 + l32;
                b[j] = c < N ? __uint_as_float((uint32_t)bias[c] << 16) : 0.0f;
            }
        }
        const int64_t col = n0 + wn * WN + lane;
        typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
        typedef float f2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float v0 = acc[i][0][r] + b[0];
                float v1 = acc[i][1][r] + b[1];
                if constexpr (GELU) {
                    v0 = gelu_tanh(v0);
                    v1 = gelu_tanh(v1);
                }
                const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0),
                                                                 __float_as_uint(v1), false, false);
                const f2 pair = {__uint_as_float(sw[0]), __uint_as_float(sw[1])};
                const uint32_t pk = __builtin_bit_cast(uint32_t, __builtin_convertvector(pair, bf2));
                const int64_t row0 = m0 + wm * WM + i * 32 + 8 * (r >> 2) + (r & 3);
                const int64_t row1 = row0 + 4;
                if (col < N) {
                    if (row0 < M)
                        y[row0 * ldy + col] = (uint16_t)pk;
                    if (row1 < M)
                        y[row1 * ldy + col] = (uint16_t)(pk >> 16);
                }
            }
        }
    }
}

template <bool I32OUT, int GS>
hipError_t launch_gs(const uint8_t* codes, const uint8_t* flags, const uint16_t* scales,
                     const uint8_t* w_packed, const uint16_t* bias, uint16_t* y, int32_t* yi,
                     int64_t M, int64_t N, int64_t K, int64_t ldy, int epilogue,
                     hipStream_t stream)
{
    const dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM));
    // the epilogue is a compile-time choice, so the plain kernel carries no GELU code
    if (!I32OUT && epilogue == 1)
        w4a4_gemm_kernel<GS, false, true><<<grid, dim3(kThreadsPerBlock), 0, stream>>>(
            codes, flags, scales, w_packed, bias, y, yi, M, N, K, ldy);
    else
        w4a4_gemm_kernel<GS, I32OUT, false><<<grid, dim3(kThreadsPerBlock), 0, stream>>>(
            codes, flags, scales, w_packed, bias, y, yi, M, N, K, ldy);
    return hipGetLastError();
}

template <bool I32OUT>
hipError_t launch(const uint8_t* codes, const uint8_t* flags, const uint16_t* scales,
                  const uint8_t* w_packed, const uint16_t* bias, uint16_t* y, int32_t* yi,
                  int64_t M, int64_t N, int64_t K, int64_t ldy, int lzs_group, int epilogue,
                  hipStream_t stream)
{
    switch (lzs_group) {
    case 8:
        return launch_gs<I32OUT, 8>(codes, flags, scales, w_packed, bias, y, yi, M, N, K, ldy,
                                    epilogue, stream);
    case 16:
        return launch_gs<I32OUT, 16>(codes, flags, scales, w_packed, bias, y, yi, M, N, K, ldy,
                                     epilogue, stream);
    case 32:
        return launch_gs<I32OUT, 32>(codes, flags, scales, w_packed, bias, y, yi, M, N, K, ldy,
                                     epilogue, stream);
    default:
        return launch_gs<I32OUT, 64>(codes, flags, scales, w_packed, bias, y, yi, M, N, K, ldy,
                                     epilogue, stream);
    }
}

}  // namespace

hipError_t launch_w4a4_linear(const uint8_t* codes, const uint8_t* flags,
                              const uint16_t* scales, const uint8_t* w_packed,
                              const uint16_t* bias, uint16_t* y, int64_t M, int64_t N, int64_t K,
                              int64_t ldy, int lzs_group, int epilogue, hipStream_t stream)
{
    return launch<false>(codes, flags, scales, w_packed, bias, y, nullptr, M, N, K, ldy, lzs_group,
                         epilogue, stream);
}

hipError_t launch_w4a4_gemm_i32(const uint8_t* codes, const uint8_t* flags,
                                const uint8_t* w_packed, int32_t* acc, int64_t M, int64_t N,
                                int64_t K, int lzs_group, hipStream_t stream)
{
    return launch<true>(codes, flags, nullptr, w_packed, nullptr, nullptr, acc, M, N, K, N,
                        lzs_group, 0, stream);
}

}  // namespace quartz
