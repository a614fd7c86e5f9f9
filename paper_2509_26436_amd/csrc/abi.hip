// C-ABI entry points of libquartz.so: host-side validation, then the launch on
// the caller's stream.  See include/quartz.h for the contract of each call.
#include <cfloat>
#include <cmath>

#include "quartz.h"
#include "quartz_internal.h"

namespace {

constexpr int64_t kMaxK = int64_t(1) << 20;       // at most 16384 groups per row
// rows x groups of one call (M x K/64 or N x K/64): 2^34 elements, 32 GiB of
// bf16 input; keeps every grid below 2^32 threads
constexpr int64_t kMaxRowGroups = int64_t(1) << 28;
// leading dimension of the activations and of the output (elements): 64 bf16
// rows of it stay below 2^31 bytes (one buffer range per wave of output rows)
constexpr int64_t kMaxLd = int64_t(1) << 24;
// pixels of one implicit convolution (images * H * W): the GEMM addresses a
// channel block's codes by pixel with 32-bit offsets (32 bytes per pixel)
constexpr int64_t kMaxConvPixels = int64_t(1) << 26;

// sizes that every entry point accepts: rows >= 0, 0 <= K <= kMaxK, K % 64 == 0
// and rows * K / 64 <= kMaxRowGroups
bool size_ok(int64_t rows, int64_t K)
{
    if (rows < 0 || K < 0 || K % 64 != 0 || K > kMaxK)
        return false;
    return K == 0 || rows <= kMaxRowGroups / (K / 64);
}

bool aligned16(const void* p)
{
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

bool lzs_ok(int32_t g)
{
    return g == 8 || g == 16 || g == 32 || g == 64;
}

quartz_status from_hip(hipError_t e)
{
    return e == hipSuccess ? QUARTZ_OK : QUARTZ_ERR_HIP;
}

}  // namespace

extern "C" {

const char* quartz_status_string(quartz_status s)
{
    switch (s) {
    case QUARTZ_OK:
        return "ok";
    case QUARTZ_ERR_NULL:
        return "a required pointer is NULL";
    case QUARTZ_ERR_SHAPE:
        return "invalid shape (negative size, K not a multiple of 64, leading dimension too small, or too large)";
    case QUARTZ_ERR_UNSUPPORTED:
        return "unsupported group_size, lzs_group, mode or epilogue";
    case QUARTZ_ERR_ALIGN:
        return "a pointer is not 16-byte aligned";
    case QUARTZ_ERR_HIP:
        return "HIP kernel launch failed";
    case QUARTZ_ERR_WORKSPACE:
        return "workspace smaller than quartz_w4a4_linear_workspace_bytes";
    }
    return "unknown status";
}

quartz_status quartz_quantize_act(const void* x_bf16, int64_t M, int64_t K, int64_t ldx,
                                  int32_t group_size, int32_t lzs_group, int32_t mode,
                                  uint8_t* codes, uint8_t* flags, uint16_t* scales,
                                  int8_t* zeros, hipStream_t stream)
{
    if (group_size != 64 || !lzs_ok(lzs_group) ||
        (mode != QUARTZ_MODE_SYMMETRIC && mode != QUARTZ_MODE_ASYMMETRIC))
        return QUARTZ_ERR_UNSUPPORTED;
    if (!size_ok(M, K) || ldx < K || ldx > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (ldx % 8 != 0)
        return QUARTZ_ERR_ALIGN;       // 16-byte aligned rows for the vector loads
    if (M == 0 || K == 0)
        return QUARTZ_OK;
    if (!x_bf16 || !codes || !flags || !scales || (mode == QUARTZ_MODE_ASYMMETRIC && !zeros))
        return QUARTZ_ERR_NULL;
    if (!aligned16(x_bf16) || !aligned16(codes) || !aligned16(flags) || !aligned16(scales) ||
        (zeros && !aligned16(zeros)))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_quantize_act(static_cast<const uint16_t*>(x_bf16), M, K, ldx,
                                                lzs_group, codes, flags, scales, zeros,
                                                mode == QUARTZ_MODE_ASYMMETRIC, stream));
}

quartz_status quartz_quantize_act_static(const void* x_bf16, int64_t M, int64_t K, int64_t ldx,
                                         float scale, int32_t lzs_group, uint8_t* codes,
                                         uint8_t* flags, hipStream_t stream)
{
    if (!lzs_ok(lzs_group) || !(scale >= FLT_MIN) || !std::isfinite(scale))
        return QUARTZ_ERR_UNSUPPORTED;
    if (!size_ok(M, K) || ldx < K || ldx > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (ldx % 8 != 0)
        return QUARTZ_ERR_ALIGN;
    if (M == 0 || K == 0)
        return QUARTZ_OK;
    if (!x_bf16 || !codes || !flags)
        return QUARTZ_ERR_NULL;
    if (!aligned16(x_bf16) || !aligned16(codes) || !aligned16(flags))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_quantize_act_static(static_cast<const uint16_t*>(x_bf16), M, K,
                                                       ldx, scale, lzs_group, codes, flags,
                                                       stream));
}

size_t quartz_packed_weight_bytes(int64_t N, int64_t K, int32_t group_size)
{
    if (group_size != 64 || N < 0 || K < 0 || K % 64 != 0)
        return 0;
    return (size_t)quartz::packed_weight_bytes(N, K);
}

quartz_status quartz_pack_weight(const void* w_bf16, int64_t N, int64_t K, int32_t group_size,
                                 void* w_packed, uint16_t* w_scales, hipStream_t stream)
{
    if (group_size != 64)
        return QUARTZ_ERR_UNSUPPORTED;
    if (!size_ok(N, K))
        return QUARTZ_ERR_SHAPE;
    if (N == 0 || K == 0)
        return QUARTZ_OK;
    if (!w_bf16 || !w_packed)
        return QUARTZ_ERR_NULL;
    if (!aligned16(w_bf16) || !aligned16(w_packed) || (w_scales && !aligned16(w_scales)))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_pack_weight(static_cast<const uint16_t*>(w_bf16), N, K,
                                               static_cast<uint8_t*>(w_packed), w_scales, stream));
}

quartz_status quartz_pack_weight_per_channel(const void* w_bf16, int64_t N, int64_t K,
                                             void* w_packed, uint16_t* w_scales,
                                             hipStream_t stream)
{
    if (!size_ok(N, K))
        return QUARTZ_ERR_SHAPE;
    if (N == 0 || K == 0)
        return QUARTZ_OK;
    if (!w_bf16 || !w_packed)
        return QUARTZ_ERR_NULL;
    if (!aligned16(w_bf16) || !aligned16(w_packed) || (w_scales && !aligned16(w_scales)))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_pack_weight_per_channel(static_cast<const uint16_t*>(w_bf16), N,
                                                           K, static_cast<uint8_t*>(w_packed),
                                                           w_scales, stream));
}

quartz_status quartz_weight_group_sums(const void* w_packed, int64_t N, int64_t K,
                                      int32_t group_size, int16_t* w_sums, hipStream_t stream)
{
    if (group_size != 64)
        return QUARTZ_ERR_UNSUPPORTED;
    if (!size_ok(N, K))
        return QUARTZ_ERR_SHAPE;
    if (N == 0 || K == 0)
        return QUARTZ_OK;
    if (!w_packed || !w_sums)
        return QUARTZ_ERR_NULL;
    if (!aligned16(w_packed) || !aligned16(w_sums))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_weight_group_sums(static_cast<const uint8_t*>(w_packed), N, K,
                                                     w_sums, stream));
}

quartz_status quartz_unpack_weight(const void* w_packed, int64_t N, int64_t K,
                                   int32_t group_size, int8_t* wq_out, hipStream_t stream)
{
    if (group_size != 64)
        return QUARTZ_ERR_UNSUPPORTED;
    if (!size_ok(N, K))
        return QUARTZ_ERR_SHAPE;
    if (N == 0 || K == 0)
        return QUARTZ_OK;
    if (!w_packed || !wq_out)
        return QUARTZ_ERR_NULL;
    if (!aligned16(w_packed) || !aligned16(wq_out))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_unpack_weight(static_cast<const uint8_t*>(w_packed), N, K,
                                                 wq_out, stream));
}

static quartz_status check_gemm(const uint8_t* codes, const uint8_t* flags, const void* w_packed,
                                int64_t M, int64_t N, int64_t K, int32_t group_size,
                                int32_t lzs_group)
{
    if (group_size != 64 || !lzs_ok(lzs_group))
        return QUARTZ_ERR_UNSUPPORTED;
    if (K <= 0 || !size_ok(M, K) || !size_ok(N, K) ||
        ((M + quartz::kGemmBlockRows - 1) / quartz::kGemmBlockRows) *
                ((N + quartz::kGemmBlockCols - 1) / quartz::kGemmBlockCols) >
            quartz::kMaxGemmTiles)
        return QUARTZ_ERR_SHAPE;
    if (M == 0 || N == 0)
        return QUARTZ_OK;
    if (!codes || !flags || !w_packed)
        return QUARTZ_ERR_NULL;
    if (!aligned16(codes) || !aligned16(flags) || !aligned16(w_packed))
        return QUARTZ_ERR_ALIGN;
    return QUARTZ_OK;
}

// qout == nullptr: bf16 output y_bf16 [M][ldy]; otherwise the output goes
// to qout (quantized for the next layer) and y_bf16 / ldy are not used
static quartz_status linear_impl(const uint8_t* codes, const uint8_t* flags,
                                 const uint16_t* scales, const void* w_packed,
                                 const void* bias_bf16, void* y_bf16, int64_t M, int64_t N,
                                 int64_t K, int64_t ldy, int32_t group_size, int32_t lzs_group,
                                 int32_t epilogue, void* workspace, size_t workspace_bytes,
                                 const quartz::QuantOut* qout, hipStream_t stream,
                                 bool use_scratch = false)
{
    if (epilogue != QUARTZ_EPI_NONE && epilogue != QUARTZ_EPI_GELU_TANH)
        return QUARTZ_ERR_UNSUPPORTED;
    quartz_status st = check_gemm(codes, flags, w_packed, M, N, K, group_size, lzs_group);
    if (st != QUARTZ_OK)
        return st;
    if (!qout && (ldy < N || ldy > kMaxLd))
        return QUARTZ_ERR_SHAPE;
    if (qout && N % 64 != 0)
        return QUARTZ_ERR_SHAPE;        // the output is the next layer's K
    if (M == 0 || N == 0)
        return QUARTZ_OK;
    if (!scales || (!qout && !y_bf16) ||
        (qout && (!qout->codes || !qout->flags || !qout->scales)))
        return QUARTZ_ERR_NULL;
    if (!aligned16(scales) || (!qout && !aligned16(y_bf16)) ||
        (bias_bf16 && !aligned16(bias_bf16)) || (workspace && !aligned16(workspace)) ||
        (qout && (!aligned16(qout->codes) || !aligned16(qout->flags) ||
                  !aligned16(qout->scales) || (qout->zeros && !aligned16(qout->zeros)))))
        return QUARTZ_ERR_ALIGN;
    // the linear kernel (tiles of 128 x 256), bf16 or quantized output
    const quartz::GemmSchedule sch = quartz::linear_schedule(
        M, N, K, quartz::linear_resident_blocks(), workspace != nullptr || use_scratch);
    if (sch.blocks <= 0)
        return QUARTZ_ERR_HIP;          // no usable device
    if (use_scratch) {
        // the device's own scratch array in place of a workspace: nothing is
        // allocated; its counters are cleared by a kernel on this stream
        workspace_bytes = quartz::noalloc_scratch_bytes();
        if (quartz::gemm_workspace_bytes(sch) > workspace_bytes)
            return QUARTZ_ERR_WORKSPACE;
        if (quartz::noalloc_scratch(&workspace) != hipSuccess)
            return QUARTZ_ERR_HIP;
        if (quartz::clear_noalloc_counters(workspace, quartz::gemm_counter_bytes(sch), stream) !=
            hipSuccess)
            return QUARTZ_ERR_HIP;
    }
    if (quartz::gemm_workspace_bytes(sch) > workspace_bytes)
        return QUARTZ_ERR_WORKSPACE;
    return from_hip(quartz::launch_w4a4_linear(
        codes, flags, scales, static_cast<const uint8_t*>(w_packed),
        static_cast<const uint16_t*>(bias_bf16), static_cast<uint16_t*>(y_bf16), M, N, K, ldy,
        lzs_group, epilogue, sch, workspace, qout ? *qout : quartz::QuantOut{}, stream));
}

quartz_status quartz_w4a4_linear(const uint8_t* codes, const uint8_t* flags,
                                 const uint16_t* scales, const int8_t* zeros,
                                 const void* w_packed, const void* bias_bf16, void* y_bf16,
                                 int64_t M, int64_t N, int64_t K, int64_t ldy,
                                 int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                 hipStream_t stream)
{
    (void)zeros;   // the symmetric mode has zero points 0 by construction
    return linear_impl(codes, flags, scales, w_packed, bias_bf16, y_bf16, M, N, K, ldy,
                       group_size, lzs_group, epilogue, nullptr, 0, nullptr, stream);
}

size_t quartz_w4a4_linear_workspace_bytes(int64_t M, int64_t N, int64_t K, int32_t group_size)
{
    if (group_size != 64 || M <= 0 || N <= 0 || K <= 0 || !size_ok(M, K) || !size_ok(N, K))
        return 0;
    // the larger of the two kernels' needs: the same size query serves the
    // linear layer (tiles of 128 x 256) and the entry points that run the
    // template (256 x 128: asymmetric mode, convolution)
    return std::max(
        quartz::gemm_workspace_bytes(
            quartz::gemm_schedule(M, N, K, quartz::gemm_resident_blocks(), true)),
        quartz::gemm_workspace_bytes(
            quartz::linear_schedule(M, N, K, quartz::linear_resident_blocks(), true)));
}

quartz_status quartz_w4a4_linear_ws(const uint8_t* codes, const uint8_t* flags,
                                    const uint16_t* scales, const int8_t* zeros,
                                    const void* w_packed, const void* bias_bf16, void* y_bf16,
                                    int64_t M, int64_t N, int64_t K, int64_t ldy,
                                    int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    (void)zeros;
    return linear_impl(codes, flags, scales, w_packed, bias_bf16, y_bf16, M, N, K, ldy,
                       group_size, lzs_group, epilogue, workspace, workspace_bytes, nullptr,
                       stream);
}

quartz_status quartz_w4a4_linear_noalloc(const uint8_t* codes, const uint8_t* flags,
                                         const uint16_t* scales, const int8_t* zeros,
                                         const void* w_packed, const void* bias_bf16, void* y_bf16,
                                         int64_t M, int64_t N, int64_t K, int64_t ldy,
                                         int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                         hipStream_t stream)
{
    (void)zeros;
    return linear_impl(codes, flags, scales, w_packed, bias_bf16, y_bf16, M, N, K, ldy,
                       group_size, lzs_group, epilogue, nullptr, 0, nullptr, stream, true);
}

size_t quartz_w4a4_linear_noalloc_max_bytes(void)
{
    return quartz::noalloc_scratch_bytes();
}

quartz_status quartz_w4a4_linear_static(const uint8_t* codes, const uint8_t* flags,
                                        float act_scale, const void* w_packed,
                                        const void* bias_bf16, void* y_bf16, int64_t M, int64_t N,
                                        int64_t K, int64_t ldy, int32_t lzs_group,
                                        int32_t epilogue, void* workspace, size_t workspace_bytes,
                                        hipStream_t stream)
{
    if ((epilogue != QUARTZ_EPI_NONE && epilogue != QUARTZ_EPI_GELU_TANH) ||
        !std::isfinite(act_scale))
        return QUARTZ_ERR_UNSUPPORTED;
    quartz_status st = check_gemm(codes, flags, w_packed, M, N, K, 64, lzs_group);
    if (st != QUARTZ_OK)
        return st;
    if (ldy < N || ldy > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (M == 0 || N == 0)
        return QUARTZ_OK;
    if (!y_bf16)
        return QUARTZ_ERR_NULL;
    if (!aligned16(y_bf16) || (bias_bf16 && !aligned16(bias_bf16)) ||
        (workspace && !aligned16(workspace)))
        return QUARTZ_ERR_ALIGN;
    const quartz::GemmSchedule sch =
        quartz::linear_schedule(M, N, K, quartz::linear_resident_blocks(), workspace != nullptr);
    if (sch.blocks <= 0)
        return QUARTZ_ERR_HIP;
    if (quartz::gemm_workspace_bytes(sch) > workspace_bytes)
        return QUARTZ_ERR_WORKSPACE;
    return from_hip(quartz::launch_w4a4_linear_static(
        codes, flags, act_scale, static_cast<const uint8_t*>(w_packed),
        static_cast<const uint16_t*>(bias_bf16), static_cast<uint16_t*>(y_bf16), M, N, K, ldy,
        lzs_group, epilogue, sch, workspace, stream));
}

quartz_status quartz_w4a4_linear_asym(const uint8_t* codes, const uint8_t* flags,
                                      const uint16_t* scales, const int8_t* zeros,
                                      const void* w_packed, const int16_t* w_sums,
                                      const void* bias_bf16, void* y_bf16, int64_t M, int64_t N,
                                      int64_t K, int64_t ldy, int32_t group_size,
                                      int32_t lzs_group, int32_t epilogue, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream)
{
    if (epilogue != QUARTZ_EPI_NONE && epilogue != QUARTZ_EPI_GELU_TANH)
        return QUARTZ_ERR_UNSUPPORTED;
    quartz_status st = check_gemm(codes, flags, w_packed, M, N, K, group_size, lzs_group);
    if (st != QUARTZ_OK)
        return st;
    if (ldy < N || ldy > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (M == 0 || N == 0)
        return QUARTZ_OK;
    if (!scales || !zeros || !w_sums || !y_bf16)
        return QUARTZ_ERR_NULL;
    if (!aligned16(scales) || !aligned16(zeros) || !aligned16(w_sums) || !aligned16(y_bf16) ||
        (bias_bf16 && !aligned16(bias_bf16)) || (workspace && !aligned16(workspace)))
        return QUARTZ_ERR_ALIGN;
    const quartz::GemmSchedule sch =
        quartz::linear_schedule(M, N, K, quartz::linear_resident_blocks(), workspace != nullptr);
    if (sch.blocks <= 0)
        return QUARTZ_ERR_HIP;
    if (quartz::gemm_workspace_bytes(sch) > workspace_bytes)
        return QUARTZ_ERR_WORKSPACE;
    return from_hip(quartz::launch_w4a4_linear_asym(
        codes, flags, scales, zeros, static_cast<const uint8_t*>(w_packed), w_sums,
        static_cast<const uint16_t*>(bias_bf16), static_cast<uint16_t*>(y_bf16), M, N, K, ldy,
        lzs_group, epilogue, sch, workspace, stream));
}

quartz_status quartz_w4a4_linear_quantize(const uint8_t* codes, const uint8_t* flags,
                                          const uint16_t* scales, const int8_t* zeros,
                                          const void* w_packed, const void* bias_bf16, int64_t M,
                                          int64_t N, int64_t K, int32_t group_size,
                                          int32_t lzs_group, int32_t epilogue,
                                          int32_t out_lzs_group, int32_t out_mode,
                                          uint8_t* out_codes, uint8_t* out_flags,
                                          uint16_t* out_scales, int8_t* out_zeros, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream)
{
    (void)zeros;
    if (!lzs_ok(out_lzs_group) || out_mode != QUARTZ_MODE_SYMMETRIC)
        return QUARTZ_ERR_UNSUPPORTED;
    // the output is the next layer's activation with K = N
    if (!size_ok(M, N))
        return QUARTZ_ERR_SHAPE;
    const quartz::QuantOut q{out_codes, out_flags, out_scales, out_zeros, out_lzs_group};
    return linear_impl(codes, flags, scales, w_packed, bias_bf16, nullptr, M, N, K, 0,
                       group_size, lzs_group, epilogue, workspace, workspace_bytes, &q, stream);
}

int64_t quartz_w4a4_linear_schedule(int64_t M, int64_t N, int64_t K, int32_t blocks,
                                    int32_t split, int32_t tiles, int32_t* schedule,
                                    int32_t* segments, int64_t capacity)
{
    if (M <= 0 || N <= 0 || K <= 0 || !size_ok(M, K) || !size_ok(N, K) || blocks <= 0 ||
        !schedule || capacity < 0 || (capacity > 0 && !segments) || (tiles != 0 && tiles != 1))
        return -1;
    const quartz::GemmSchedule s = tiles == 0 ? quartz::linear_schedule(M, N, K, blocks, split != 0)
                                              : quartz::gemm_schedule(M, N, K, blocks, split != 0);
    if (s.blocks <= 0)
        return -1;
    const int32_t fields[10] = {s.tiles_n, s.groups, s.sk_tiles > 0 ? 1 : 0, s.blocks,
                                quartz::dp_count(s, 0), s.sk_first, s.sk_tiles, s.sk_blocks,
                                s.sk_q, s.sk_r};
    for (int i = 0; i < 10; ++i)
        schedule[i] = fields[i];
    int64_t n = 0;
    for (int32_t b = 0; b < s.blocks; ++b) {
        quartz::GemmSegment sg;
        int32_t steps = 0;
        for (int32_t j = 0; quartz::gemm_segment(s, b, j, sg); ++j, ++n) {
            steps += sg.g1 - sg.g0;
            if (n >= capacity)
                continue;
            int32_t b_first = -1, b_last = -1, other_slot = -1;
            if (sg.sk_tile >= 0) {
                quartz::sk_contributors(s, sg.sk_tile, b_first, b_last);
                other_slot = quartz::sk_slot(s, b, sg.sk_tile);
            }
            const int32_t row[10] = {b, j, sg.tile, sg.g0, sg.g1, sg.sk_tile, sg.slot, b_first,
                                     b_last, other_slot};
            for (int i = 0; i < 10; ++i)
                segments[n * 10 + i] = row[i];
        }
        // the kernel walks the same segments incrementally
        quartz::GemmCursor c;
        int32_t jc = 0, padded = 0;
        for (bool ok = quartz::cursor_begin(s, b, c); ok; ok = quartz::cursor_next(s, b, c), ++jc) {
            quartz::GemmSegment ref;
            if (!quartz::gemm_segment(s, b, jc, ref) || ref.tile != c.sg.tile || ref.g0 != c.sg.g0 ||
                ref.g1 != c.sg.g1 || ref.sk_tile != c.sg.sk_tile || ref.slot != c.sg.slot ||
                c.j != jc || (int64_t)c.tm * s.tiles_n + c.tn != c.sg.tile)
                return -2;
            padded += quartz::padded_steps(c.sg.g1 - c.sg.g0);
        }
        quartz::GemmSegment extra;
        if (quartz::gemm_segment(s, b, jc, extra) || padded != quartz::gemm_steps(s, b) ||
            padded < steps)
            return -2;
    }
    return n;
}

quartz_status quartz_w4a4_gemm_i32(const uint8_t* codes, const uint8_t* flags,
                                   const void* w_packed, int32_t* acc_out, int64_t M, int64_t N,
                                   int64_t K, int32_t group_size, int32_t lzs_group,
                                   hipStream_t stream)
{
    quartz_status st = check_gemm(codes, flags, w_packed, M, N, K, group_size, lzs_group);
    if (st != QUARTZ_OK)
        return st;
    if (M == 0 || N == 0)
        return QUARTZ_OK;
    if (!acc_out)
        return QUARTZ_ERR_NULL;
    if (!aligned16(acc_out))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_w4a4_gemm_i32(codes, flags,
                                                 static_cast<const uint8_t*>(w_packed), acc_out, M,
                                                 N, K, lzs_group, stream));
}

// ------------------------------------------------------------ LZS attention

static bool attn_dims_ok(int64_t L, int64_t d)
{
    return L > 0 && d > 0 && L % 64 == 0 && d % 64 == 0 && L <= kMaxK && d <= kMaxK;
}

quartz_status quartz_quantize_vt(const void* v_bf16, int64_t heads, int64_t L, int64_t d,
                                 int64_t ldv, int32_t lzs_group, uint8_t* codes, uint8_t* flags,
                                 uint16_t* scales, hipStream_t stream)
{
    if (!lzs_ok(lzs_group))
        return QUARTZ_ERR_UNSUPPORTED;
    if (heads < 0 || !attn_dims_ok(L, d) || ldv < d || ldv > kMaxLd ||
        !size_ok(heads * d, L) || (heads > 0 && L > kMaxRowGroups / heads))
        return QUARTZ_ERR_SHAPE;
    if (ldv % 8 != 0)
        return QUARTZ_ERR_ALIGN;
    if (heads == 0)
        return QUARTZ_OK;
    if (!v_bf16 || !codes || !flags || !scales)
        return QUARTZ_ERR_NULL;
    if (!aligned16(v_bf16) || !aligned16(codes) || !aligned16(flags) || !aligned16(scales))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_quantize_vt(static_cast<const uint16_t*>(v_bf16), heads, L, d,
                                               ldv, lzs_group, codes, flags, scales, stream));
}

quartz_status quartz_softmax_quantize(const float* s, int64_t M, int64_t N, int64_t lds,
                                      int32_t lzs_group, uint8_t* codes, uint8_t* flags,
                                      uint16_t* scales, hipStream_t stream)
{
    if (!lzs_ok(lzs_group))
        return QUARTZ_ERR_UNSUPPORTED;
    if (M < 0 || N <= 0 || N % 64 != 0 || !size_ok(M, N) || lds < N || lds > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (lds % 4 != 0)
        return QUARTZ_ERR_ALIGN;
    if (M == 0)
        return QUARTZ_OK;
    if (!s || !codes || !flags || !scales)
        return QUARTZ_ERR_NULL;
    if (!aligned16(s) || !aligned16(codes) || !aligned16(flags) || !aligned16(scales))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_softmax_quantize(s, M, N, lds, lzs_group, codes, flags, scales,
                                                    stream));
}

// rows [row0, row0 + n) of planes of `plane` rows
static bool rows_ok(int64_t plane, int64_t row0, int64_t n)
{
    return plane > 0 && row0 >= 0 && n >= 0 && row0 <= plane - n && plane <= kMaxRowGroups;
}

quartz_status quartz_attn_scores(const uint8_t* q_codes, const uint8_t* q_flags,
                                 const uint16_t* q_scales, int64_t q_plane, int64_t q_row0,
                                 const uint8_t* k_codes, const uint8_t* k_flags,
                                 const uint16_t* k_scales, int64_t k_plane, int64_t k_row0,
                                 int64_t Lq, int64_t Lk, int64_t d, int32_t lzs_group, float scale,
                                 float* s, int64_t lds, hipStream_t stream)
{
    if (!lzs_ok(lzs_group) || !std::isfinite(scale))
        return QUARTZ_ERR_UNSUPPORTED;
    if (Lq < 0 || Lk < 0 || d <= 0 || d % 64 != 0 || d > kMaxK || !rows_ok(q_plane, q_row0, Lq) ||
        !rows_ok(k_plane, k_row0, Lk) || !size_ok(q_plane, d) || !size_ok(k_plane, d) ||
        lds < Lk || lds > kMaxLd ||
        ((Lq + quartz::kGemmBlockRows - 1) / quartz::kGemmBlockRows) *
                ((Lk + quartz::kGemmBlockCols - 1) / quartz::kGemmBlockCols) > quartz::kMaxGemmTiles)
        return QUARTZ_ERR_SHAPE;
    if (Lq == 0 || Lk == 0)
        return QUARTZ_OK;
    if (!q_codes || !q_flags || !q_scales || !k_codes || !k_flags || !k_scales || !s)
        return QUARTZ_ERR_NULL;
    if (!aligned16(q_codes) || !aligned16(q_flags) || !aligned16(q_scales) || !aligned16(k_codes) ||
        !aligned16(k_flags) || !aligned16(k_scales) || !aligned16(s))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_attn_scores(q_codes, q_flags, q_scales, q_plane, q_row0, k_codes,
                                               k_flags, k_scales, k_plane, k_row0, Lq, Lk, d,
                                               lzs_group, scale, s, lds, stream));
}

size_t quartz_attn_pv_workspace_bytes(int64_t Lq, int64_t Lk, int64_t d)
{
    if (Lq <= 0 || d <= 0 || Lk <= 0 || Lk % 64 != 0 || !size_ok(Lq, Lk) || !size_ok(d, Lk))
        return 0;
    return quartz::gemm_workspace_bytes(
        quartz::gemm_schedule(Lq, d, Lk, quartz::gemm_resident_blocks(), true));
}

quartz_status quartz_attn_pv(const uint8_t* p_codes, const uint8_t* p_flags,
                             const uint16_t* p_scales, const uint8_t* vt_codes,
                             const uint8_t* vt_flags, const uint16_t* vt_scales, int64_t vt_plane,
                             int64_t vt_row0, int64_t Lq, int64_t Lk, int64_t d,
                             int32_t lzs_group, void* o_bf16, int64_t ldo, void* workspace,
                             size_t workspace_bytes, hipStream_t stream)
{
    if (!lzs_ok(lzs_group))
        return QUARTZ_ERR_UNSUPPORTED;
    if (Lq < 0 || d <= 0 || Lk <= 0 || Lk % 64 != 0 || Lk > kMaxK || !size_ok(Lq, Lk) ||
        !rows_ok(vt_plane, vt_row0, d) || !size_ok(vt_plane, Lk) || ldo < d || ldo > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (Lq == 0)
        return QUARTZ_OK;
    if (!p_codes || !p_flags || !p_scales || !vt_codes || !vt_flags || !vt_scales || !o_bf16)
        return QUARTZ_ERR_NULL;
    if (!aligned16(p_codes) || !aligned16(p_flags) || !aligned16(p_scales) ||
        !aligned16(vt_codes) || !aligned16(vt_flags) || !aligned16(vt_scales) ||
        !aligned16(o_bf16) || (workspace && !aligned16(workspace)))
        return QUARTZ_ERR_ALIGN;
    const quartz::GemmSchedule sch =
        quartz::gemm_schedule(Lq, d, Lk, quartz::gemm_resident_blocks(), workspace != nullptr);
    if (sch.blocks <= 0)
        return QUARTZ_ERR_HIP;
    if (quartz::gemm_workspace_bytes(sch) > workspace_bytes)
        return QUARTZ_ERR_WORKSPACE;
    return from_hip(quartz::launch_attn_pv(p_codes, p_flags, p_scales, vt_codes, vt_flags,
                                           vt_scales, vt_plane, vt_row0, Lq, Lk, d, lzs_group,
                                           static_cast<uint16_t*>(o_bf16), ldo, sch, workspace,
                                           stream));
}

// Workspace of quartz_lzs_attention.  Head dimensions 64 and 128 (the fused
// kernel): Q, K and V^T codes / flags / scales of all heads, then the three
// expanded to fp8 e4m3.  Other d (the unfused pipeline), in order: the PV
// split workspace (must start zero-filled; every call leaves it so), the
// codes / flags / scales, the scores of one head and its quantized softmax
// output.
namespace {
struct AttnLayout {
    size_t split, qc, qf, qs, kc, kf, ks, vc, vf, vs, qx, kx, vx, s, pc, pf, ps, total;
};
size_t align256(size_t x) { return (x + 255) / 256 * 256; }
bool attention_fused(int64_t d) { return d == 64 || d == 128; }
AttnLayout attn_layout(int64_t heads, int64_t L, int64_t d, int32_t gs)
{
    AttnLayout w{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align256(bytes);
        return at;
    };
    const bool fused = attention_fused(d);
    const size_t rows = (size_t)(heads * L);
    const size_t vrows = (size_t)(heads * d);
    if (!fused)
        w.split = take(quartz::gemm_workspace_bytes(
            quartz::gemm_schedule(L, d, L, quartz::gemm_resident_blocks(), true)));
    w.qc = take(rows * (size_t)d / 2);
    w.qf = take(rows * (size_t)d / (size_t)gs);
    w.qs = take(rows * (size_t)d / 64 * 2);
    w.kc = take(rows * (size_t)d / 2);
    w.kf = take(rows * (size_t)d / (size_t)gs);
    w.ks = take(rows * (size_t)d / 64 * 2);
    w.vc = take(vrows * (size_t)L / 2);
    w.vf = take(vrows * (size_t)L / (size_t)gs);
    w.vs = take(vrows * (size_t)L / 64 * 2);
    if (fused) {
        w.qx = take(rows * (size_t)d);
        w.kx = take(rows * (size_t)d);
        w.vx = take(vrows * (size_t)L);
    } else {
        w.s = take((size_t)L * (size_t)L * 4);
        w.pc = take((size_t)L * (size_t)L / 2);
        w.pf = take((size_t)L * (size_t)L / (size_t)gs);
        w.ps = take((size_t)L * (size_t)L / 64 * 2);
    }
    w.total = off;
    return w;
}
}  // namespace

static bool attention_shape_ok(int64_t heads, int64_t L, int64_t d)
{
    return heads >= 0 && attn_dims_ok(L, d) && L <= (int64_t(1) << 16) &&
           (heads == 0 || (heads <= kMaxRowGroups / L && size_ok(heads * L, d) &&
                           size_ok(heads * d, L)));
}

size_t quartz_lzs_attention_workspace_bytes(int64_t heads, int64_t L, int64_t d,
                                            int32_t lzs_group)
{
    if (!lzs_ok(lzs_group) || heads <= 0 || !attention_shape_ok(heads, L, d))
        return 0;
    return attn_layout(heads, L, d, lzs_group).total;
}

quartz_status quartz_lzs_attention(const void* q_bf16, const void* k_bf16, const void* v_bf16,
                                   int64_t heads, int64_t L, int64_t d, int32_t lzs_group,
                                   void* o_bf16, int64_t ldo, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream)
{
    if (!lzs_ok(lzs_group))
        return QUARTZ_ERR_UNSUPPORTED;
    if (!attention_shape_ok(heads, L, d) || ldo < heads * d || ldo > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (heads == 0)
        return QUARTZ_OK;
    if (!q_bf16 || !k_bf16 || !v_bf16 || !o_bf16 || !workspace)
        return QUARTZ_ERR_NULL;
    if (!aligned16(q_bf16) || !aligned16(k_bf16) || !aligned16(v_bf16) || !aligned16(o_bf16) ||
        !aligned16(workspace) || ldo % 4 != 0)
        return QUARTZ_ERR_ALIGN;
    const AttnLayout w = attn_layout(heads, L, d, lzs_group);
    if (w.total > workspace_bytes)
        return QUARTZ_ERR_WORKSPACE;
    uint8_t* base = static_cast<uint8_t*>(workspace);
    auto u8 = [&](size_t off) { return base + off; };
    auto u16 = [&](size_t off) { return reinterpret_cast<uint16_t*>(base + off); };
    const int64_t rows = heads * L;
    hipError_t e = quartz::launch_quantize_act(static_cast<const uint16_t*>(q_bf16), rows, d, d,
                                               lzs_group, u8(w.qc), u8(w.qf), u16(w.qs), nullptr,
                                               false, stream);
    if (e == hipSuccess)
        e = quartz::launch_quantize_act(static_cast<const uint16_t*>(k_bf16), rows, d, d,
                                        lzs_group, u8(w.kc), u8(w.kf), u16(w.ks), nullptr, false,
                                        stream);
    if (e == hipSuccess)
        e = quartz::launch_quantize_vt(static_cast<const uint16_t*>(v_bf16), heads, L, d, d,
                                       lzs_group, u8(w.vc), u8(w.vf), u16(w.vs), stream);
    if (attention_fused(d)) {
        if (e == hipSuccess)
            e = quartz::launch_expand_fp8(u8(w.qc), u8(w.qf), rows, d, lzs_group, u8(w.qx), stream);
        if (e == hipSuccess)
            e = quartz::launch_expand_fp8(u8(w.kc), u8(w.kf), rows, d, lzs_group, u8(w.kx), stream);
        if (e == hipSuccess)
            e = quartz::launch_expand_fp8(u8(w.vc), u8(w.vf), heads * d, L, lzs_group, u8(w.vx),
                                          stream);
        if (e == hipSuccess)
            e = quartz::launch_attention_fused(u8(w.qx), u16(w.qs), u8(w.kx), u16(w.ks), u8(w.vx),
                                               u16(w.vs), heads, L, d, lzs_group,
                                               static_cast<uint16_t*>(o_bf16), ldo, stream);
        return from_hip(e);
    }
    const quartz::GemmSchedule pv =
        quartz::gemm_schedule(L, d, L, quartz::gemm_resident_blocks(), true);
    const float scale = (float)(1.0 / std::sqrt((double)d));
    float* S = reinterpret_cast<float*>(base + w.s);
    for (int64_t h = 0; h < heads && e == hipSuccess; ++h) {
        e = quartz::launch_attn_scores(u8(w.qc), u8(w.qf), u16(w.qs), rows, h * L, u8(w.kc),
                                       u8(w.kf), u16(w.ks), rows, h * L, L, L, d, lzs_group,
                                       scale, S, L, stream);
        if (e == hipSuccess)
            e = quartz::launch_softmax_quantize(S, L, L, L, lzs_group, u8(w.pc), u8(w.pf),
                                                u16(w.ps), stream);
        if (e == hipSuccess)
            e = quartz::launch_attn_pv(u8(w.pc), u8(w.pf), u16(w.ps), u8(w.vc), u8(w.vf),
                                       u16(w.vs), heads * d, h * d, L, L, d, lzs_group,
                                       static_cast<uint16_t*>(o_bf16) + h * d, ldo, pv,
                                       u8(w.split), stream);
    }
    return from_hip(e);
}

static quartz_status conv_impl(const uint8_t* codes, const uint8_t* flags,
                               const uint16_t* scales, float act_scale, bool is_static,
                               const void* w_packed, const void* bias_bf16, void* y_bf16,
                               int64_t images, int64_t H, int64_t W, int64_t C, int64_t N,
                               int64_t ldy, int32_t group_size, int32_t lzs_group,
                               int32_t epilogue, void* workspace, size_t workspace_bytes,
                               hipStream_t stream)
{
    if ((epilogue != QUARTZ_EPI_NONE && epilogue != QUARTZ_EPI_GELU_TANH) ||
        (is_static && !std::isfinite(act_scale)))
        return QUARTZ_ERR_UNSUPPORTED;
    if (images < 0 || H <= 0 || W <= 0 || C <= 0 || C % 64 != 0 || N < 0 ||
        H >= kMaxConvPixels || W >= kMaxConvPixels || H > kMaxConvPixels / W ||
        (images > 0 && images > (kMaxConvPixels - 1) / (H * W)) || C > kMaxK / 9)
        return QUARTZ_ERR_SHAPE;
    const int64_t M = images * H * W;
    const int64_t K = 9 * C;
    quartz_status st = check_gemm(codes, flags, w_packed, M, N, K, group_size, lzs_group);
    if (st != QUARTZ_OK)
        return st;
    if (ldy < N || ldy > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (M == 0 || N == 0)
        return QUARTZ_OK;
    if ((!is_static && !scales) || !y_bf16)
        return QUARTZ_ERR_NULL;
    if ((!is_static && !aligned16(scales)) || !aligned16(y_bf16) ||
        (bias_bf16 && !aligned16(bias_bf16)) || (workspace && !aligned16(workspace)))
        return QUARTZ_ERR_ALIGN;
    const quartz::GemmSchedule sch =
        quartz::gemm_schedule(M, N, K, quartz::gemm_resident_blocks(), workspace != nullptr);
    if (sch.blocks <= 0)
        return QUARTZ_ERR_HIP;
    if (quartz::gemm_workspace_bytes(sch) > workspace_bytes)
        return QUARTZ_ERR_WORKSPACE;
    return from_hip(quartz::launch_w4a4_conv3x3(
        codes, flags, is_static ? nullptr : scales, act_scale,
        static_cast<const uint8_t*>(w_packed), static_cast<const uint16_t*>(bias_bf16),
        static_cast<uint16_t*>(y_bf16), images, H, W, C, N, ldy, lzs_group, epilogue, sch,
        workspace, stream));
}

quartz_status quartz_w4a4_conv3x3(const uint8_t* codes, const uint8_t* flags,
                                  const uint16_t* scales, const void* w_packed,
                                  const void* bias_bf16, void* y_bf16, int64_t images, int64_t H,
                                  int64_t W, int64_t C, int64_t N, int64_t ldy,
                                  int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    return conv_impl(codes, flags, scales, 0.0f, false, w_packed, bias_bf16, y_bf16, images, H,
                     W, C, N, ldy, group_size, lzs_group, epilogue, workspace, workspace_bytes,
                     stream);
}

quartz_status quartz_w4a4_conv3x3_static(const uint8_t* codes, const uint8_t* flags,
                                         float act_scale, const void* w_packed,
                                         const void* bias_bf16, void* y_bf16, int64_t images,
                                         int64_t H, int64_t W, int64_t C, int64_t N, int64_t ldy,
                                         int32_t lzs_group, int32_t epilogue, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream)
{
    return conv_impl(codes, flags, nullptr, act_scale, true, w_packed, bias_bf16, y_bf16, images,
                     H, W, C, N, ldy, 64, lzs_group, epilogue, workspace, workspace_bytes,
                     stream);
}

}  // extern "C"
