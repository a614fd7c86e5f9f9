// Host side of the W4A4 GEMM: the work schedule of the persistent grid, the
// split workspace layout, and the launch entry points (the kernels are
// instantiated in w4a4_gemm_<mode>.hip).
#include "w4a4_gemm_kernel.h"

namespace quartz {
namespace {

// Split only when it saves each workgroup at least kMinSplitSaving groups of
// work on average (the idle part of the last round of whole tiles): below
// that, the split's own costs (segments that start mid-tile, partial sums,
// operands shared less well in L2) eat the gain.  With fewer tiles than
// workgroups, every workgroup takes at least kMinSplitGroups groups and a
// tile is shared by about kMaxSplitWays workgroups at most (each extra one
// costs the finisher a slot read), and nothing is split when that leaves
// fewer than two workgroups per tile on average: the exchange of partial
// sums then costs more than the balance gains (9 tiles of 18 groups: 36 us
// split over 40 workgroups against 20 us whole).
constexpr int64_t kMinSplitSaving = 16;
constexpr int64_t kMinSplitGroups = 16;
constexpr int64_t kMaxSplitWays = 8;

size_t counter_bytes(const GemmSchedule& s)
{
    return ((size_t)s.sk_tiles * kMathWaves * sizeof(uint32_t) + 255) / 256 * 256;
}

}  // namespace

GemmSchedule gemm_schedule_tiles(int64_t M, int64_t N, int64_t K, int blocks, bool split,
                                 int64_t bm, int64_t bn)
{
    GemmSchedule s{};
    const int64_t tiles_m = (M + bm - 1) / bm;
    const int64_t tiles_n = (N + bn - 1) / bn;
    const int64_t T = tiles_m * tiles_n;
    const int64_t G = K / 64;
    s.tiles_n = (int32_t)tiles_n;
    s.groups = (int32_t)G;
    if (blocks <= 0 || T <= 0 || G <= 0 || T > kMaxGemmTiles)
        return s;                              // blocks == 0: nothing to launch
    // whole tiles only: tile b + r * blocks for r = 0, 1, ...
    s.blocks = (int32_t)std::min<int64_t>(blocks, T);
    s.sk_first = (int32_t)T;
    if (!split || T % blocks == 0)
        return s;
    const int64_t rounds = (T + blocks - 1) / blocks;
    if ((rounds * blocks - T) * G < kMinSplitSaving * blocks)
        return s;
    int64_t sk_first, sk_blocks;
    if (T > blocks) {
        sk_first = (T / blocks - 1) * blocks;  // leaves between 1 and 2 rounds of tiles to split
        sk_blocks = blocks;
    } else {
        sk_first = 0;
        const int64_t min_units = std::max(kMinSplitGroups, (G + kMaxSplitWays - 1) / kMaxSplitWays);
        sk_blocks = std::max<int64_t>(1, std::min<int64_t>(blocks, T * G / min_units));
        if (sk_blocks < 2 * T)
            return s;                          // under two workgroups per tile: not worth the exchange
    }
    const int64_t units = (T - sk_first) * G;
    if (units >= (int64_t(1) << 30))
        return s;
    s.blocks = (int32_t)(T > blocks ? blocks : sk_blocks);
    s.sk_first = (int32_t)sk_first;
    s.sk_tiles = (int32_t)(T - sk_first);
    s.sk_blocks = (int32_t)sk_blocks;
    s.sk_q = (int32_t)(units / sk_blocks);
    s.sk_r = (int32_t)(units % sk_blocks);
    return s;
}

GemmSchedule gemm_schedule(int64_t M, int64_t N, int64_t K, int blocks, bool split)
{
    return gemm_schedule_tiles(M, N, K, blocks, split, BM, BN);
}

size_t gemm_counter_bytes(const GemmSchedule& s)
{
    return s.sk_tiles > 0 ? counter_bytes(s) : 0;
}

size_t gemm_workspace_bytes(const GemmSchedule& s)
{
    if (s.sk_tiles == 0)
        return 0;
    return counter_bytes(s) + (size_t)2 * s.sk_blocks * kMathWaves * WM * WN * sizeof(float);
}

static void split_workspace(const GemmSchedule& sch, void* workspace, uint32_t*& counters,
                            float*& slots)
{
    counters = static_cast<uint32_t*>(workspace);
    slots = sch.sk_tiles > 0
                ? reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + counter_bytes(sch))
                : nullptr;
}

hipError_t launch_w4a4_linear(const uint8_t* codes, const uint8_t* flags,
                              const uint16_t* scales, const uint8_t* w_packed,
                              const uint16_t* bias, uint16_t* y, int64_t M, int64_t N, int64_t K,
                              int64_t ldy, int lzs_group, int epilogue, const GemmSchedule& sch,
                              void* workspace, const QuantOut& qout, hipStream_t stream)
{
    if (sch.blocks <= 0)
        return hipErrorInvalidConfiguration;
    GemmLaunch a{codes, flags, scales, w_packed, bias, y, nullptr, M, N, K, ldy, lzs_group,
                 epilogue, sch, nullptr, nullptr, qout, 0.0f};
    split_workspace(sch, workspace, a.counters, a.slots);
    // the kernel of w4a4_linear.hip (tiles of 128 x 256, schedule from
    // linear_schedule), bf16 or quantized output
    return launch_linear(a, stream);
}

hipError_t launch_w4a4_linear_static(const uint8_t* codes, const uint8_t* flags, float act_scale,
                                     const uint8_t* w_packed, const uint16_t* bias, uint16_t* y,
                                     int64_t M, int64_t N, int64_t K, int64_t ldy, int lzs_group,
                                     int epilogue, const GemmSchedule& sch, void* workspace,
                                     hipStream_t stream)
{
    if (sch.blocks <= 0)
        return hipErrorInvalidConfiguration;
    GemmLaunch a{codes, flags, nullptr, w_packed, bias, y, nullptr, M, N, K, ldy, lzs_group,
                 epilogue, sch, nullptr, nullptr, QuantOut{}, act_scale};
    split_workspace(sch, workspace, a.counters, a.slots);
    // the kernel of w4a4_linear.hip (schedule from linear_schedule)
    return launch_linear_static(a, stream);
}

hipError_t launch_w4a4_linear_asym(const uint8_t* codes, const uint8_t* flags,
                                   const uint16_t* scales, const int8_t* zeros,
                                   const uint8_t* w_packed, const int16_t* wsums,
                                   const uint16_t* bias, uint16_t* y, int64_t M, int64_t N,
                                   int64_t K, int64_t ldy, int lzs_group, int epilogue,
                                   const GemmSchedule& sch, void* workspace, hipStream_t stream)
{
    if (sch.blocks <= 0)
        return hipErrorInvalidConfiguration;
    GemmLaunch a{codes, flags, scales, w_packed, bias, y, nullptr, M, N, K, ldy, lzs_group,
                 epilogue, sch, nullptr, nullptr, QuantOut{}, 0.0f, zeros, wsums};
    split_workspace(sch, workspace, a.counters, a.slots);
    // the kernel of w4a4_linear_asym.hip (schedule from linear_schedule)
    return launch_linear_asym(a, stream);
}

hipError_t launch_w4a4_conv3x3(const uint8_t* codes, const uint8_t* flags,
                               const uint16_t* scales, float act_scale, const uint8_t* w_packed,
                               const uint16_t* bias, uint16_t* y, int64_t images, int64_t H,
                               int64_t W, int64_t C, int64_t N, int64_t ldy, int lzs_group,
                               int epilogue, const GemmSchedule& sch, void* workspace,
                               hipStream_t stream)
{
    if (sch.blocks <= 0)
        return hipErrorInvalidConfiguration;
    const int64_t M = images * H * W;
    const int32_t cg = (int32_t)(C / kGroup);
    const ConvGeom conv{(int32_t)H, (int32_t)W, cg,
                        cg > 1 ? (uint32_t)((uint64_t(1) << 32) / (uint64_t)cg + 1) : 0u};
    GemmLaunch a{codes, flags, scales, w_packed, bias, y, nullptr, M, N, 9 * C, ldy, lzs_group,
                 epilogue, sch, nullptr, nullptr, QuantOut{}, act_scale, nullptr, nullptr, conv};
    split_workspace(sch, workspace, a.counters, a.slots);
    return scales ? launch_gemm_conv(a, stream) : launch_gemm_conv_static(a, stream);
}

hipError_t launch_attn_scores(const uint8_t* qc, const uint8_t* qf, const uint16_t* qs,
                              int64_t q_plane, int64_t q_row0, const uint8_t* kc,
                              const uint8_t* kf, const uint16_t* ks, int64_t k_plane,
                              int64_t k_row0, int64_t Lq, int64_t Lk, int64_t d, int lzs_group,
                              float scale, float* s, int64_t lds, hipStream_t stream)
{
    const GemmSchedule sch = gemm_schedule(Lq, Lk, d, gemm_resident_blocks(), false);
    if (sch.blocks <= 0)
        return hipErrorInvalidConfiguration;
    GemmLaunch a{qc, qf, qs, nullptr, nullptr, nullptr, nullptr, Lq, Lk, d, lds, lzs_group, 0,
                 sch, nullptr, nullptr, QuantOut{}, 0.0f};
    a.attn = AttnGeom{kc, kf, ks, q_plane, q_row0, k_plane, k_row0, s, scale};
    return launch_gemm_attn_scores(a, stream);
}

hipError_t launch_attn_pv(const uint8_t* pc, const uint8_t* pf, const uint16_t* ps,
                          const uint8_t* vc, const uint8_t* vf, const uint16_t* vs,
                          int64_t v_plane, int64_t v_row0, int64_t Lq, int64_t Lk, int64_t d,
                          int lzs_group, uint16_t* o, int64_t ldo, const GemmSchedule& sch,
                          void* workspace, hipStream_t stream)
{
    if (sch.blocks <= 0)
        return hipErrorInvalidConfiguration;
    GemmLaunch a{pc, pf, ps, nullptr, nullptr, o, nullptr, Lq, d, Lk, ldo, lzs_group, 0,
                 sch, nullptr, nullptr, QuantOut{}, 0.0f};
    a.attn = AttnGeom{vc, vf, vs, Lq, 0, v_plane, v_row0, nullptr, 0.0f};
    split_workspace(sch, workspace, a.counters, a.slots);
    return launch_gemm_attn_pv(a, stream);
}

hipError_t launch_w4a4_gemm_i32(const uint8_t* codes, const uint8_t* flags,
                                const uint8_t* w_packed, int32_t* acc, int64_t M, int64_t N,
                                int64_t K, int lzs_group, hipStream_t stream)
{
    const GemmSchedule sch = gemm_schedule(M, N, K, gemm_resident_blocks(), false);
    if (sch.blocks <= 0)
        return hipErrorInvalidConfiguration;
    const GemmLaunch a{codes, flags, nullptr, w_packed, nullptr, nullptr, acc, M, N, K, N,
                       lzs_group, 0, sch, nullptr, nullptr, QuantOut{}, 0.0f};
    return launch_gemm_i32(a, stream);
}

}  // namespace quartz
