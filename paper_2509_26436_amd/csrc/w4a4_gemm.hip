// W4A4 GEMM with in-register decode and CDNA4 fp8 MFMA.
//
// For each 64-element K-group g the block stages its tiles of packed 4-bit
// activations (codes + per-subgroup FLAG + fp16 scale) and packed 4-bit
// weights (codes + fp16 scale) from global memory, decodes them in registers
// to OCP fp8 e4m3 operands -- activations as c * 2^FLAG in [-112, 112],
// weights as wq in [-7, 7], both exact in e4m3 -- and writes them to LDS
// (double-buffered: group g+1 is fetched from global memory while group g is
// multiplied).  Each wave then runs v_mfma_f32_32x32x64_f8f6f4 over the whole
// group, which yields the exact integer group product P_g (every partial sum
// is an integer below 2^24), and folds it into fp32 accumulators with the two
// group scales:
//   acc += P_g * (s_a[m,g] * s_w[n,g]).
// The 32 x 32 tile of scale products s_a (x) s_w is itself produced by one
// fp16 MFMA with a single non-zero k (fp16 x fp16 is exact in fp32), so the
// per-group dequantization costs one FMA per output element.
// The epilogue adds the bias, applies the optional GELU (tanh form) and
// stores bf16 (round to nearest even).
#include <type_traits>

#include "quartz_internal.h"

namespace quartz {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));


__device__ __forceinline__ uint16_t f32_to_bf16_rne(float v)
{
    uint32_t u = __float_as_uint(v);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float gelu_tanh(float v)
{
    const float k = 0.7978845608028654f;   // sqrt(2 / pi)
    return 0.5f * v * (1.0f + tanhf(k * (v + 0.044715f * v * v * v)));
}

// ------------------------------------------------------------------ layout
// Block tile BM x BN = 256 x 128, 8 waves as 4 (M) x 2 (N), wave tile 64 x 64
// = 2 x 2 MFMA tiles of 32 x 32.  Two waves share each SIMD, so one wave's
// VALU work (decode, dequantization) overlaps the other's MFMAs.
constexpr int BM = (int)kGemmBlockRows;
constexpr int BN = 128;
constexpr int kWaves = 8;
constexpr int kThreadsPerBlock = 64 * kWaves;
constexpr int WAVES_N = 2;
constexpr int WM = 64;
constexpr int WN = 64;
constexpr int TM = WM / 32;
constexpr int TN = WN / 32;
constexpr int kDepth = 3;      // groups held in the register prefetch ring

// 16-byte chunk c of decoded fp8 row r lives at chunk c ^ f(r) with
//   f(r) = (r1 ^ r2) | (r2 ^ r3) << 1      (r_i = bit i of r).
// Fragment reads (16 consecutive rows, one chunk) and decode writes (8 rows,
// both halves) then touch distinct 16-byte bank groups within every 128-byte
// and every 256-byte window, whether the LDS serves 8 or 16 lanes per cycle.
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

// Raw flag bytes of the 32 elements [32 h, 32 h + 32) of one (group, row),
// whose 64 / GS flag bytes start at `p` (loaded as is: expanding them right
// after the load would make the prefetch wait for it).
// (kept in a 16-bit type where 16 bits suffice, so that the zero extension
// happens when the ring slot is decoded, not right after the load).
template <int GS>
using FlagRaw = typename std::conditional<GS == 8, uint32_t, uint16_t>::type;

template <int GS>
__device__ __forceinline__ FlagRaw<GS> load_flags_raw(const uint8_t* __restrict__ p)
{
    if constexpr (GS == 8)
        return *reinterpret_cast<const uint32_t*>(p);
    else if constexpr (GS == 16)
        return *reinterpret_cast<const uint16_t*>(p);
    else
        return *p;
}

// Raw flags -> 8 * FLAG of each 8-element word i (0..3) of the half, one per byte.
template <int GS>
__device__ __forceinline__ uint32_t expand_flags8(uint32_t raw)
{
    uint32_t f;
    if constexpr (GS == 8)
        f = raw;
    else if constexpr (GS == 16)
        f = __builtin_amdgcn_perm(0u, raw, 0x01010000u);
    else
        f = __builtin_amdgcn_perm(0u, raw, 0x00000000u);
    return f << 3;    // FLAG <= 4, so 8 * FLAG stays inside its byte
}

// Staging roles: thread t decodes A row t/2, half t%2 (16 code bytes) and
// B column t/4, quarter t%4 (8 code bytes); threads < BM carry s_a of row t
// and BM <= t < BM + BN s_w of column t - BM.  Every thread issues the same
// four loads per group (the rest load a scale they do not use), so the
// compiler can count them and wait only for the group being decoded.  Rows
// past M and columns past the padded N read a clamped, valid row / column:
// they only feed outputs that are never stored, so the main loop needs no
// bounds checks.
template <int GS, bool I32OUT>
__global__ __launch_bounds__(kThreadsPerBlock) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ codes, const uint8_t* __restrict__ flags,
    const uint16_t* __restrict__ scales, const uint8_t* __restrict__ w_packed,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ yi,
    int64_t M, int64_t N, int64_t K, int64_t ldy, int epilogue)
{
    __shared__ __attribute__((aligned(16))) uint8_t As[2][BM * 64];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[2][BN * 64];
    // group scales as fp16 bits; entries BM (BN) stay 0: the upper half-wave's
    // k = 8 operand slot of the outer-product MFMA reads them
    __shared__ uint16_t sas[2][BM + 8];
    __shared__ uint16_t sws[2][BN + 8];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t m0 = (int64_t)blockIdx.y * BM;
    const int64_t n0 = (int64_t)blockIdx.x * BN;
    const int G = (int)(K / 64);
    const int64_t padded_n = (N + kPanel - 1) / kPanel * kPanel;

    static_assert(2 * BM == kThreadsPerBlock && 4 * BN == kThreadsPerBlock, "staging roles");
    const int sr = tid >> 1;          // A row
    const int sh = tid & 1;           // A half
    const int bc = tid >> 2;          // B column
    const int bq = tid & 3;           // B quarter
    // Global addresses = a wave-uniform base for group g and this block
    // (scalar registers) plus a small 32-bit per-lane offset.  Activations
    // are K-group-major: group g of row m at (g * M + m).
    const int64_t am = min(m0 + sr, M - 1);
    const uint32_t a_code_off = (uint32_t)((am - m0) * 32 + sh * 16);
    constexpr int kFlagHalf = GS == 64 ? 0 : 32 / GS;   // flag bytes of the first half
    const uint32_t a_flag_off = (uint32_t)((am - m0) * (64 / GS) + sh * kFlagHalf);
    // the block's columns n0 .. n0 + BN - 1 span two 64-column panels
    const int64_t panel0 = n0 / kPanel;
    const int64_t bn = min(n0 + bc, padded_n - 1);
    const uint32_t b_code_off = (uint32_t)((bn / kPanel - panel0) * G * kChunkBytes +
                                           (bn % kPanel) * 32 + bq * 8);
    // scales: waves 0-3 carry s_a of row tid (K-group-major, stride M per
    // group), waves 4-5 s_w of column tid - BM (inside the packed chunk,
    // stride kChunkBytes per group); waves 6-7 load an s_a they do not use
    const int uwave = __builtin_amdgcn_readfirstlane(wave);
    const bool sa_role = uwave < 4;
    const bool sw_role = uwave == 4 || uwave == 5;
    const int64_t sam = min(m0 + (tid & (BM - 1)), M - 1);
    const int64_t swn = min(n0 + (tid & (BN - 1)), padded_n - 1);
    const uint32_t s_off = sw_role ? (uint32_t)((swn / kPanel - panel0) * G * kChunkBytes +
                                                kChunkCodeBytes + (swn % kPanel) * 2)
                                   : (uint32_t)((sam - m0) * 2);
    const uint8_t* a_blk = codes + m0 * 32;
    const uint8_t* f_blk = flags + m0 * (64 / GS);
    const uint8_t* b_blk = w_packed + panel0 * G * kChunkBytes;
    const uint8_t* s_base =
        sw_role || I32OUT ? b_blk : reinterpret_cast<const uint8_t*>(scales + m0);
    const int64_t s_stride = sw_role ? (int64_t)kChunkBytes : M * 2;

    struct Raw {
        uint4 a;
        uint2 b;
        FlagRaw<GS> f;
        uint16_t s;
    };
    auto fetch = [&](Raw& r, int g) {
        const uint8_t* ca = a_blk + (int64_t)g * (M * 32);
        const uint8_t* cf = f_blk + (int64_t)g * (M * (64 / GS));
        const uint8_t* cb = b_blk + (int64_t)g * kChunkBytes;
        const uint8_t* cs = s_base + (int64_t)g * s_stride;
        r.a = *reinterpret_cast<const uint4*>(ca + a_code_off);
        r.f = load_flags_raw<GS>(cf + a_flag_off);
        r.b = *reinterpret_cast<const uint2*>(cb + b_code_off);
        if constexpr (!I32OUT)       // the integer path has no scales (scales == nullptr)
            r.s = *reinterpret_cast<const uint16_t*>(cs + s_off);
        else
            r.s = 0;
    };
    // ---- compute roles
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;
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

    // Decode of the next group, cut into four slices so that each slice's VALU
    // work is issued while the matrix unit runs one tile's MFMAs.
    // Decode of the next group in eight pieces, two per MFMA tile: piece 2t
    // goes between tile t's fp8 MFMA and its scale MFMA, piece 2t+1 right
    // before its FMAs.  Tiles 0 and 1 decode the two words pairs of the
    // activation row half, tile 2 the weight column quarter, tile 3 stores
    // the scales.
    uint32_t fl8 = 0;      // 8 * FLAG per activation word of this half
    Fp8Table t_lo, t_hi;   // tables of the two words being decoded
    uint2 d_first;         // first word of a pair, decoded
    auto stage_piece = [&](const Raw& r, int buf, int piece) {
        switch (piece) {
        case 0:
            fl8 = expand_flags8<GS>((uint32_t)r.f);
            t_lo = fp8_table<0>(fl8);
            t_hi = GS == 8 ? fp8_table<1>(fl8) : t_lo;
            d_first = decode_nibbles_fp8(r.a.x, t_lo);
            break;
        case 1: {
            const uint2 d = decode_nibbles_fp8(r.a.y, t_hi);
            *reinterpret_cast<uint4*>(As[buf] + swz(sr, 2 * sh)) =
                make_uint4(d_first.x, d_first.y, d.x, d.y);
            break;
        }
        case 2:
            t_lo = GS <= 16 ? fp8_table<2>(fl8) : t_lo;
            t_hi = GS == 8 ? fp8_table<3>(fl8) : t_lo;
            d_first = decode_nibbles_fp8(r.a.z, t_lo);
            break;
        case 3: {
            const uint2 d = decode_nibbles_fp8(r.a.w, t_hi);
            *reinterpret_cast<uint4*>(As[buf] + swz(sr, 2 * sh + 1)) =
                make_uint4(d_first.x, d_first.y, d.x, d.y);
            break;
        }
        case 4:
            d_first = decode_nibbles_fp8(r.b.x, Fp8Table{kTabLo, kTabHi});
            break;
        case 5: {
            const uint2 d = decode_nibbles_fp8(r.b.y, Fp8Table{kTabLo, kTabHi});
            *reinterpret_cast<uint4*>(Bs[buf] + swz(bc, bq)) =
                make_uint4(d_first.x, d_first.y, d.x, d.y);
            break;
        }
        case 6:
            if (sa_role)
                sas[buf][tid] = r.s;
            else if (sw_role)
                sws[buf][tid - BM] = r.s;
            break;
        default:
            break;
        }
    };
    auto stage = [&](const Raw& r, int buf) {
#pragma unroll
        for (int q = 0; q < 8; ++q)
            stage_piece(r, buf, q);
    };

    // One group: per tile, the MFMAs, then a decode slice of the next group
    // (VALU work that runs while the matrix unit computes), then the tile's
    // FMAs.  Scheduling barriers keep this order; the asm statement pins each
    // tile's FMAs (without a use, LLVM sinks them to the end of the loop and
    // keeps every tile's results live).
    auto compute = [&](int buf, const Raw& next, bool more, int next_buf) {
        v8i bf[TN];
        v8h sw_op[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            bf[j] = load_frag(Bs[buf], wn * WN + j * 32 + l32, khalf);
            sw_op[j] = v8h{};
            if constexpr (!I32OUT)
                sw_op[j][0] = __builtin_bit_cast(_Float16, sws[buf][sw_idx[j]]);
        }
        constexpr int T = TM * TN;
        static_assert(T == 4, "four decode slices per group");
        const v16f zero = {};
        v8i af[TM];
        v8h sa_op[TM];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            af[i] = load_frag(As[buf], wm * WM + i * 32 + l32, khalf);
            // fp16 operand of the scale outer product: only k = 0 is non-zero
            sa_op[i] = v8h{};
            if constexpr (!I32OUT)
                sa_op[i][0] = __builtin_bit_cast(_Float16, sas[buf][sa_idx[i]]);
        }
        auto tile = [&](int i, int j, bool interleave) {
            // in-order issue: VALU work between the two MFMAs keeps the wave
            // busy while the matrix unit finishes the first one
            const v16f p = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                af[i], bf[j], zero, 0, 0, 0, 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            if (interleave && more)
                stage_piece(next, next_buf, 2 * (i * TN + j));
            __builtin_amdgcn_sched_barrier(0);
            v16f sc;
            if constexpr (!I32OUT)
                sc = __builtin_amdgcn_mfma_f32_32x32x16_f16(sa_op[i], sw_op[j], zero, 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            if (interleave && more)
                stage_piece(next, next_buf, 2 * (i * TN + j) + 1);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                if constexpr (I32OUT)
                    acc[i][j][r] += p[r];
                else
                    acc[i][j][r] = fmaf(p[r], sc[r], acc[i][j][r]);
            }
            asm volatile("" : "+v"(acc[i][j]));
            __builtin_amdgcn_sched_barrier(0);
        };
#pragma unroll
        for (int t = 0; t < T; ++t)
            tile(t / TN, t % TN, true);
    };

    // ---- pipeline: register ring of kDepth groups, fp8 LDS double buffer
    if (tid < 8) {
        sas[tid & 1][BM + (tid >> 1)] = 0;
        sws[tid & 1][BN + (tid >> 1)] = 0;
    }
    Raw ring[kDepth];
#pragma unroll
    for (int u = 0; u < kDepth; ++u)
        fetch(ring[u], min(u, G - 1));
    stage(ring[0], 0);
    lds_sync();

    // Main loop over chunks of 2 * kDepth groups (ring slot and LDS buffer are
    // then compile-time constants in every unrolled copy): straight-line code
    // with the same loads on every path (prefetch indices past the end are
    // clamped to the last group: a harmless reload), so the compiler waits
    // only for the ring slot being decoded, not for the loads just issued.
    constexpr int kUnroll = 2 * kDepth;
    {
        int g0 = 0;
        for (; g0 + kUnroll <= G; g0 += kUnroll) {
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int g = g0 + u;
                // ring slot u % kDepth held group g (staged one iteration ago): refill it
                fetch(ring[u % kDepth], min(g + kDepth, G - 1));
                compute(u & 1, ring[(u + 1) % kDepth], true, (u + 1) & 1);
                lds_sync();
            }
        }
        // Tail: the last G % kUnroll groups (their prefetches are issued above
        // or inside this loop in the same ring order).
#pragma unroll
        for (int u = 0; u < kUnroll - 1; ++u) {
            const int g = g0 + u;
            if (g < G) {
                if (g + kDepth < G)
                    fetch(ring[u % kDepth], g + kDepth);
                compute(u & 1, ring[(u + 1) % kDepth], g + 1 < G, (u + 1) & 1);
                lds_sync();
            }
        }
    }

    // ---- epilogue: lane holds column l32 of each 32 x 32 tile, rows 8 (r/4) + 4 khalf + r%4
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int64_t col = n0 + wn * WN + j * 32 + l32;
        if (col >= N)
            continue;
        float b = 0.0f;
        if (!I32OUT && bias)
            b = __uint_as_float((uint32_t)bias[col] << 16);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * khalf + (r & 3);
                if (row >= M)
                    continue;
                if constexpr (I32OUT) {
                    yi[row * N + col] = (int32_t)acc[i][j][r];
                } else {
                    float v = acc[i][j][r] + b;
                    if (epilogue == 1)
                        v = gelu_tanh(v);
                    y[row * ldy + col] = f32_to_bf16_rne(v);
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
    w4a4_gemm_kernel<GS, I32OUT><<<grid, dim3(kThreadsPerBlock), 0, stream>>>(
        codes, flags, scales, w_packed, bias, y, yi, M, N, K, ldy, epilogue);
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
