// Weight pre-pack: symmetric round-to-nearest int4 per 64-element group along
// K with an fp16 group scale (the weight setting of Appendix C), written in
// the GEMM's panel layout (see quartz_internal.h), plus the debug unpack.
//
// A team of 8 lanes owns one (column n, group g): each lane loads 8 bf16,
// the team reduces max|w| with DPP, every lane computes
//   s_w = fp16_rne_sat(max|w| / 7),  r = 1/s_w,  |wq| = min(rne(|w| * r), 7)
// and stores one 32-bit word of 8 sign-magnitude nibbles, in the same nibble
// order as the activation codes.
#include "quartz_internal.h"

namespace quartz {
namespace {

constexpr float kMagic = 12582912.0f;          // 1.5 * 2^23, see quantize_lzs.hip
constexpr uint32_t kMagicBits = 0x4B400000u;

__device__ __forceinline__ uint32_t dpp_xor1(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
}
__device__ __forceinline__ uint32_t dpp_xor2(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
}
__device__ __forceinline__ uint32_t dpp_half_mirror(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);
}

__device__ __forceinline__ uint32_t f16_bits_rne_sat(float s)
{
    _Float16 h = (_Float16)s;
    uint32_t b = (uint32_t)__builtin_bit_cast(uint16_t, h);
    if ((b & 0x7FFFu) == 0x7C00u)
        b = (b & 0x8000u) | 0x7BFFu;
    return b;
}

// grid covers panels * 64 columns x G groups; one team per (column, group)
__global__ __launch_bounds__(256) void pack_weight_kernel(
    const uint16_t* __restrict__ w, int64_t N, int64_t K, int64_t padded_cols,
    uint8_t* __restrict__ w_packed, uint16_t* __restrict__ w_scales)
{
    const int lane = threadIdx.x & 63;
    const int u = lane & 7;
    const int64_t G = K / 64;
    const int64_t team = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 3;
    const int64_t total = padded_cols * G;
    const bool live = team < total;
    // team -> (panel, group, column in panel); consecutive teams walk the
    // columns of one (panel, group) chunk so the chunk is written contiguously
    const int64_t cpan = team % kPanel;
    const int64_t pg = team / kPanel;
    const int64_t g = pg % G;
    const int64_t panel = pg / G;
    const int64_t n = panel * kPanel + cpan;
    const bool real = live && n < N;

    uint4 v = make_uint4(0, 0, 0, 0);
    if (real)
        v = *reinterpret_cast<const uint4*>(w + n * K + g * 64 + u * 8);
    const uint32_t d[4] = {v.x, v.y, v.z, v.w};
    float f[8];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        f[2 * p] = __uint_as_float(d[p] << 16);
        f[2 * p + 1] = __uint_as_float(d[p] & 0xFFFF0000u);
    }
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        amax = fmaxf(amax, fabsf(f[i]));
    uint32_t ab = __float_as_uint(amax);
    ab = max(ab, dpp_xor1(ab));
    ab = max(ab, dpp_xor2(ab));
    ab = max(ab, dpp_half_mirror(ab));
    const float beta = __uint_as_float(ab);
    const uint32_t s16 = f16_bits_rne_sat(beta / 7.0f);
    const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)s16);
    const float r = (s == 0.0f) ? 0.0f : 1.0f / s;

    uint32_t T = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float prod = fabsf(f[i]) * r;
        const uint32_t b = min(__float_as_uint(prod + kMagic), kMagicBits + 7u);
        T |= (b & 7u) << (4 * ((i >> 1) + 4 * (i & 1)));
    }
    uint32_t S = 0;
#pragma unroll
    for (int p = 0; p < 4; ++p)
        S |= (d[p] & 0x80008000u) >> (12 - 4 * p);
    const uint32_t word = T | (S & (T + 0x77777777u));

    if (live) {
        uint8_t* chunk = w_packed + (panel * G + g) * kChunkBytes;
        reinterpret_cast<uint32_t*>(chunk + cpan * 32)[u] = word;
        if (u == 0) {
            reinterpret_cast<uint16_t*>(chunk + kChunkCodeBytes)[cpan] = (uint16_t)s16;
            if (real && w_scales)
                w_scales[n * G + g] = (uint16_t)s16;
        }
    }
}

// one thread per 8 weights: decode a nibble word back to int8 values
__global__ __launch_bounds__(256) void unpack_weight_kernel(
    const uint8_t* __restrict__ w_packed, int64_t N, int64_t K, int8_t* __restrict__ wq)
{
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t words_per_row = K / 8;
    if (t >= N * words_per_row)
        return;
    const int64_t n = t / words_per_row;
    const int64_t j = t - n * words_per_row;
    const int64_t G = K / 64;
    const int64_t g = j / 8;
    const int64_t panel = n / kPanel;
    const int64_t cpan = n % kPanel;
    const uint32_t word = reinterpret_cast<const uint32_t*>(
        w_packed + (panel * G + g) * kChunkBytes + cpan * 32)[j % 8];
    uint32_t out[2] = {0, 0};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const uint32_t nib = (word >> (4 * ((i >> 1) + 4 * (i & 1)))) & 0xFu;
        const int mag = (int)(nib & 7u);
        const int val = (nib & 8u) ? -mag : mag;
        out[i >> 2] |= ((uint32_t)val & 0xFFu) << (8 * (i & 3));
    }
    reinterpret_cast<uint2*>(wq + n * K + j * 8)[0] = make_uint2(out[0], out[1]);
}

}  // namespace

hipError_t launch_pack_weight(const uint16_t* w, int64_t N, int64_t K, uint8_t* w_packed,
                              uint16_t* w_scales, hipStream_t stream)
{
    const int64_t padded = (N + kPanel - 1) / kPanel * kPanel;
    const int64_t teams = padded * (K / 64);
    const int64_t blocks = (teams * 8 + 255) / 256;
    pack_weight_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(w, N, K, padded, w_packed,
                                                                          w_scales);
    return hipGetLastError();
}

hipError_t launch_unpack_weight(const uint8_t* w_packed, int64_t N, int64_t K, int8_t* wq,
                                hipStream_t stream)
{
    const int64_t threads = N * (K / 8);
    const int64_t blocks = (threads + 255) / 256;
    unpack_weight_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(w_packed, N, K, wq);
    return hipGetLastError();
}

}  // namespace quartz
