// C-ABI entry points of libquartz.so: host-side validation, then the launch on
// the caller's stream.  See include/quartz.h for the contract of each call.
#include "quartz.h"
#include "quartz_internal.h"

namespace {

constexpr int64_t kMaxK = int64_t(1) << 20;       // at most 16384 groups per row
// rows x groups of one call (M x K/64 or N x K/64): 2^34 elements, 32 GiB of
// bf16 input; keeps every grid below 2^32 threads
constexpr int64_t kMaxRowGroups = int64_t(1) << 28;
// leading dimension of the activations (elements): 8 rows of it stay below 2^32 bytes
constexpr int64_t kMaxLd = int64_t(1) << 24;

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
    }
    return "unknown status";
}

quartz_status quartz_quantize_act(const void* x_bf16, int64_t M, int64_t K, int64_t ldx,
                                  int32_t group_size, int32_t lzs_group, int32_t mode,
                                  uint8_t* codes, uint8_t* flags, uint16_t* scales,
                                  int8_t* zeros, hipStream_t stream)
{
    if (group_size != 64 || !lzs_ok(lzs_group) || mode != QUARTZ_MODE_SYMMETRIC)
        return QUARTZ_ERR_UNSUPPORTED;
    if (!size_ok(M, K) || ldx < K || ldx > kMaxLd)
        return QUARTZ_ERR_SHAPE;
    if (ldx % 8 != 0)
        return QUARTZ_ERR_ALIGN;       // 16-byte aligned rows for the vector loads
    if (M == 0 || K == 0)
        return QUARTZ_OK;
    if (!x_bf16 || !codes || !flags || !scales)
        return QUARTZ_ERR_NULL;
    if (!aligned16(x_bf16) || !aligned16(codes) || !aligned16(flags) || !aligned16(scales) ||
        (zeros && !aligned16(zeros)))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_quantize_act(static_cast<const uint16_t*>(x_bf16), M, K, ldx,
                                                lzs_group, codes, flags, scales, zeros, stream));
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
        (M + quartz::kGemmBlockRows - 1) / quartz::kGemmBlockRows > 65535)
        return QUARTZ_ERR_SHAPE;
    if (M == 0 || N == 0)
        return QUARTZ_OK;
    if (!codes || !flags || !w_packed)
        return QUARTZ_ERR_NULL;
    if (!aligned16(codes) || !aligned16(flags) || !aligned16(w_packed))
        return QUARTZ_ERR_ALIGN;
    return QUARTZ_OK;
}

quartz_status quartz_w4a4_linear(const uint8_t* codes, const uint8_t* flags,
                                 const uint16_t* scales, const int8_t* zeros,
                                 const void* w_packed, const void* bias_bf16, void* y_bf16,
                                 int64_t M, int64_t N, int64_t K, int64_t ldy,
                                 int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                 hipStream_t stream)
{
    (void)zeros;   // the symmetric mode has zero points 0 by construction
    if (epilogue != QUARTZ_EPI_NONE && epilogue != QUARTZ_EPI_GELU_TANH)
        return QUARTZ_ERR_UNSUPPORTED;
    quartz_status st = check_gemm(codes, flags, w_packed, M, N, K, group_size, lzs_group);
    if (st != QUARTZ_OK)
        return st;
    if (ldy < N)
        return QUARTZ_ERR_SHAPE;
    if (M == 0 || N == 0)
        return QUARTZ_OK;
    if (!scales || !y_bf16)
        return QUARTZ_ERR_NULL;
    if (!aligned16(scales) || !aligned16(y_bf16) || (bias_bf16 && !aligned16(bias_bf16)))
        return QUARTZ_ERR_ALIGN;
    return from_hip(quartz::launch_w4a4_linear(
        codes, flags, scales, static_cast<const uint8_t*>(w_packed),
        static_cast<const uint16_t*>(bias_bf16), static_cast<uint16_t*>(y_bf16), M, N, K, ldy,
        lzs_group, epilogue, stream));
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

}  // extern "C"
