// W4A4 GEMM with in-register decode and CDNA4 fp8 MFMA.
//
// For each 64-element K-group g the block stages its tiles of packed 4-bit
// activations (codes + per-subgroup FLAG + fp16 scale) and packed 4-bit
// weights (codes + fp16 scale) from global memory, decodes them in registers
// to OCP fp8 e4m3 operands -- activations as c * 2^FLAG in [-112, 112],
// weights as wq in [-7, 7], both exact in e4m3 -- and writes them to LDS.
// Each wave then runs v_mfma_f32_32x32x64_f8f6f4 over the whole group, which
// yields the exact integer group product P_g (all partial sums are integers
// below 2^24), and folds it into fp32 accumulators with the two group scales:
//   acc += P_g * (s_a[m,g] * s_w[n,g])      (s_a * s_w is exact in fp32).
// The epilogue adds the bias, applies the optional GELU (tanh form) and
// stores bf16 (round to nearest even).
#include "quartz_internal.h"

namespace quartz {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int kThreads = 256;
constexpr int kRowBytes = 64;   // one decoded fp8 row of a group in LDS

__device__ __forceinline__ float f16_to_f32(uint16_t h)
{
    return (float)__builtin_bit_cast(_Float16, h);
}

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

// Flags of the 32 elements [32 h, 32 h + 32) of group g of row m: the flag of
// 8-element word i (0..3) of that half.
template <int GS>
__device__ __forceinline__ void load_flags(const uint8_t* __restrict__ flags, int64_t m, int64_t K,
                                           int g, int h, uint32_t fl[4])
{
    const uint8_t* row = flags + m * (K / GS);
    if constexpr (GS == 8) {
        const uint32_t f4 = *reinterpret_cast<const uint32_t*>(row + g * 8 + h * 4);
        for (int i = 0; i < 4; ++i)
            fl[i] = (f4 >> (8 * i)) & 0xFFu;
    } else if constexpr (GS == 16) {
        const uint32_t f2 = *reinterpret_cast<const uint16_t*>(row + g * 4 + h * 2);
        fl[0] = fl[1] = f2 & 0xFFu;
        fl[2] = fl[3] = f2 >> 8;
    } else if constexpr (GS == 32) {
        const uint32_t f1 = row[g * 2 + h];
        fl[0] = fl[1] = fl[2] = fl[3] = f1;
    } else {
        const uint32_t f1 = row[g];
        fl[0] = fl[1] = fl[2] = fl[3] = f1;
    }
}

template <int GS, bool I32OUT>
__global__ __launch_bounds__(kThreads) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ codes, const uint8_t* __restrict__ flags,
    const uint16_t* __restrict__ scales, const uint8_t* __restrict__ w_packed,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int32_t* __restrict__ yi,
    int64_t M, int64_t N, int64_t K, int64_t ldy, int epilogue)
{
    __shared__ __attribute__((aligned(16))) uint8_t As[BM * kRowBytes];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[BN * kRowBytes];
    __shared__ float sa_s[BM];
    __shared__ float sw_s[BN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t m0 = (int64_t)blockIdx.y * BM;
    const int64_t n0 = (int64_t)blockIdx.x * BN;
    const int G = (int)(K / 64);
    const int64_t panels = (N + kPanel - 1) / kPanel;

    // staging role: row / column (tid / 2) and half of the group (tid % 2)
    const int sr = tid >> 1;
    const int sh = tid & 1;
    const int64_t am = m0 + sr;
    const int64_t bn = n0 + sr;
    const bool a_ok = am < M;
    const bool b_ok = bn < panels * kPanel;
    const uint8_t* a_codes = codes + am * (K / 2) + sh * 16;
    const uint8_t* b_base = w_packed + (bn / kPanel) * G * kChunkBytes;
    const int b_col = (int)(bn % kPanel);

    // compute role: 2 x 2 waves, each 64 x 64 = 2 x 2 MFMA tiles of 32 x 32
    const int wm = wave >> 1;
    const int wn = wave & 1;

    v16f acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][j][r] = 0.0f;

    for (int g = 0; g < G; ++g) {
        // ---- stage A: 32 codes of row am -> fp8 in LDS
        {
            uint4 c4 = make_uint4(0, 0, 0, 0);
            uint32_t fl[4] = {0, 0, 0, 0};
            float sa = 0.0f;
            if (a_ok) {
                c4 = *reinterpret_cast<const uint4*>(a_codes + g * 32);
                load_flags<GS>(flags, am, K, g, sh, fl);
                sa = f16_to_f32(scales[am * G + g]);
            }
            const uint2 d0 = decode_nibbles_fp8(c4.x, fl[0]);
            const uint2 d1 = decode_nibbles_fp8(c4.y, fl[1]);
            const uint2 d2 = decode_nibbles_fp8(c4.z, fl[2]);
            const uint2 d3 = decode_nibbles_fp8(c4.w, fl[3]);
            uint4* dst = reinterpret_cast<uint4*>(As + sr * kRowBytes + sh * 32);
            dst[0] = make_uint4(d0.x, d0.y, d1.x, d1.y);
            dst[1] = make_uint4(d2.x, d2.y, d3.x, d3.y);
            if (sh == 0)
                sa_s[sr] = sa;
        }
        // ---- stage B: 32 weight codes of column bn -> fp8 in LDS
        {
            uint4 c4 = make_uint4(0, 0, 0, 0);
            float sw = 0.0f;
            if (b_ok) {
                const uint8_t* chunk = b_base + (int64_t)g * kChunkBytes;
                c4 = *reinterpret_cast<const uint4*>(chunk + b_col * 32 + sh * 16);
                sw = f16_to_f32(reinterpret_cast<const uint16_t*>(chunk + kChunkCodeBytes)[b_col]);
            }
            const uint2 d0 = decode_nibbles_fp8(c4.x, 0);
            const uint2 d1 = decode_nibbles_fp8(c4.y, 0);
            const uint2 d2 = decode_nibbles_fp8(c4.z, 0);
            const uint2 d3 = decode_nibbles_fp8(c4.w, 0);
            uint4* dst = reinterpret_cast<uint4*>(Bs + sr * kRowBytes + sh * 32);
            dst[0] = make_uint4(d0.x, d0.y, d1.x, d1.y);
            dst[1] = make_uint4(d2.x, d2.y, d3.x, d3.y);
            if (sh == 0)
                sw_s[sr] = sw;
        }
        __syncthreads();

        // ---- MFMA over the group + per-group dequantization
        v8i a_frag[2], b_frag[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const uint4* src = reinterpret_cast<const uint4*>(
                As + (wm * 64 + i * 32 + (lane & 31)) * kRowBytes + (lane >> 5) * 32);
            const uint4 lo = src[0], hi = src[1];
            a_frag[i] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w,
                            (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const uint4* src = reinterpret_cast<const uint4*>(
                Bs + (wn * 64 + j * 32 + (lane & 31)) * kRowBytes + (lane >> 5) * 32);
            const uint4 lo = src[0], hi = src[1];
            b_frag[j] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w,
                            (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            float sa_r[16];
            if constexpr (!I32OUT) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    sa_r[r] = sa_s[wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)];
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                v16f zero;
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    zero[r] = 0.0f;
                const v16f p = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                    a_frag[i], b_frag[j], zero, 0, 0, 0, 0, 0, 0);
                if constexpr (I32OUT) {
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        acc[i][j][r] += p[r];
                } else {
                    const float sw = sw_s[wn * 64 + j * 32 + (lane & 31)];
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        acc[i][j][r] = fmaf(p[r], sa_r[r] * sw, acc[i][j][r]);
                }
            }
        }
        __syncthreads();
    }

    // ---- epilogue
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn * 64 + j * 32 + (lane & 31);
            if (col >= N)
                continue;
            float b = 0.0f;
            if (!I32OUT && bias)
                b = __uint_as_float((uint32_t)bias[col] << 16);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
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

template <bool I32OUT>
hipError_t launch(const uint8_t* codes, const uint8_t* flags, const uint16_t* scales,
                  const uint8_t* w_packed, const uint16_t* bias, uint16_t* y, int32_t* yi,
                  int64_t M, int64_t N, int64_t K, int64_t ldy, int lzs_group, int epilogue,
                  hipStream_t stream)
{
    const dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM));
    const dim3 block(kThreads);
    switch (lzs_group) {
    case 8:
        w4a4_gemm_kernel<8, I32OUT><<<grid, block, 0, stream>>>(codes, flags, scales, w_packed,
                                                                bias, y, yi, M, N, K, ldy, epilogue);
        break;
    case 16:
        w4a4_gemm_kernel<16, I32OUT><<<grid, block, 0, stream>>>(codes, flags, scales, w_packed,
                                                                 bias, y, yi, M, N, K, ldy, epilogue);
        break;
    case 32:
        w4a4_gemm_kernel<32, I32OUT><<<grid, block, 0, stream>>>(codes, flags, scales, w_packed,
                                                                 bias, y, yi, M, N, K, ldy, epilogue);
        break;
    default:
        w4a4_gemm_kernel<64, I32OUT><<<grid, block, 0, stream>>>(codes, flags, scales, w_packed,
                                                                 bias, y, yi, M, N, K, ldy, epilogue);
        break;
    }
    return hipGetLastError();
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
