// Fused activation quantizer: Stage 1 (Eq. 1, symmetric reading) and Stage 2
// (Eq. 2 leading-zero suppression + right shift, Section 3) in one pass.
//
// One 64-element group is handled by a team of 8 lanes, each lane owning 8
// consecutive bf16 values (one 16-byte load).  A wave covers 8 consecutive rows
// (one per team) and 4 consecutive groups (4 rounds): every load instruction
// reads one full 128-byte line per row, and since the outputs are stored
// K-group-major (codes [K/64][M][32], flags [K/64][M][64/G_s], scales
// [K/64][M]) every code store of a wave writes 256 contiguous bytes.
//
// Per group:  alpha = max|x| (exact, 8-lane DPP max)
//             s = fp16_rne_sat(alpha / 127), r = 1/s (IEEE fp32 divisions)
//             |q| = min(rne(fp32(|x| * r)), 127)     (sign kept aside)
// Per subgroup of G_s: FLAG = max(29 - clz(OR |q|), 0)   (DPP OR across lanes)
//                      c = sgn * (|q| >> FLAG)           (truncation toward 0)
// rne(p) for 0 <= p < 2^22 is read from the low bits of fp32(p + 1.5 * 2^23):
// that sum has an ulp of 1, so its rounding is round-half-even of p.
#include "quartz_internal.h"

namespace quartz {
namespace {

constexpr float kMagic = 12582912.0f;          // 1.5 * 2^23
constexpr uint32_t kMagicBits = 0x4B400000u;

// DPP controls (gfx9 encoding).
constexpr int kQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141;  // row_half_mirror: lane i <-> 7 - i within 8

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// max over the 8 lanes of a team (all lanes receive it)
__device__ __forceinline__ uint32_t team8_max(uint32_t v)
{
    v = max(v, dpp<kQuadXor1>(v));
    v = max(v, dpp<kQuadXor2>(v));
    v = max(v, dpp<kHalfMirror>(v));
    return v;
}

// OR over the lanes that share one LZS subgroup (G_s / 8 lanes)
template <int GS>
__device__ __forceinline__ uint32_t subgroup_or(uint32_t v)
{
    if constexpr (GS >= 16)
        v |= dpp<kQuadXor1>(v);
    if constexpr (GS >= 32)
        v |= dpp<kQuadXor2>(v);
    if constexpr (GS >= 64)
        v |= dpp<kHalfMirror>(v);
    return v;
}

// fp32 -> fp16 bits, round to nearest even, overflow saturates to 65504.
__device__ __forceinline__ uint32_t f16_bits_rne_sat(float s)
{
    _Float16 h = (_Float16)s;
    uint32_t b = (uint32_t)__builtin_bit_cast(uint16_t, h);
    if ((b & 0x7FFFu) == 0x7C00u)
        b = (b & 0x8000u) | 0x7BFFu;
    return b;
}

template <int GS>
__global__ __launch_bounds__(256) void quantize_act_kernel(
    const uint16_t* __restrict__ x, int64_t M, int64_t G, int64_t ldx, int64_t quads,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ flags, uint16_t* __restrict__ scales,
    int8_t* __restrict__ zeros)
{
    constexpr int FB = 64 / GS;     // flag bytes per (row, group)
    const int lane = threadIdx.x & 63;
    const int team = lane >> 3;
    const int u = lane & 7;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t row = (w / quads) * 8 + team;
    const int64_t g0 = (w % quads) * 4;
    const bool row_ok = row < M;
    const uint16_t* xr = x + (row_ok ? row : 0) * ldx + u * 8;

    uint4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t g = g0 + j;
        v[j] = (row_ok && g < G) ? *reinterpret_cast<const uint4*>(xr + g * 64)
                                 : make_uint4(0, 0, 0, 0);
    }

#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t d[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
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
        const float alpha = __uint_as_float(team8_max(__float_as_uint(amax)));

        const float s_f = alpha / 127.0f;
        const uint32_t s16 = f16_bits_rne_sat(s_f);
        const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)s16);
        const float r = (s == 0.0f) ? 0.0f : 1.0f / s;

        uint32_t b[8];
        uint32_t mor = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float prod = fabsf(f[i]) * r;
            b[i] = min(__float_as_uint(prod + kMagic), kMagicBits + 127u);
            mor |= b[i];
        }
        mor = subgroup_or<GS>(mor & 0x7Fu);
        const int fl = max(29 - (int)__builtin_clz(mor | 1u), 0);

        // magnitudes t = |q| >> FLAG at nibble (i/2) + 4 (i%2)
        uint32_t T = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            T |= __builtin_amdgcn_ubfe(b[i], (uint32_t)fl, 3u) << (4 * ((i >> 1) + 4 * (i & 1)));
        // sign bits of x moved to bit 3 of each nibble
        uint32_t S = 0;
#pragma unroll
        for (int p = 0; p < 4; ++p)
            S |= (d[p] & 0x80008000u) >> (12 - 4 * p);
        // keep a sign only where the magnitude is non-zero: t + 7 sets bit 3 iff t >= 1
        const uint32_t word = T | (S & (T + 0x77777777u));

        const int64_t g = g0 + j;
        if (row_ok && g < G) {
            const int64_t rg = g * M + row;          // (group, row) in K-group-major order
            reinterpret_cast<uint32_t*>(codes)[rg * 8 + u] = word;
            if constexpr (GS == 8) {
                flags[rg * FB + u] = (uint8_t)fl;
            } else if constexpr (GS == 16) {
                if ((u & 1) == 0)
                    flags[rg * FB + (u >> 1)] = (uint8_t)fl;
            } else if constexpr (GS == 32) {
                if ((u & 3) == 0)
                    flags[rg * FB + (u >> 2)] = (uint8_t)fl;
            } else {
                if (u == 0)
                    flags[rg] = (uint8_t)fl;
            }
            if (u == 0) {
                scales[rg] = (uint16_t)s16;
                if (zeros)
                    zeros[rg] = 0;
            }
        }
    }
}

template <int GS>
hipError_t launch_gs(const uint16_t* x, int64_t M, int64_t K, int64_t ldx, uint8_t* codes,
                     uint8_t* flags, uint16_t* scales, int8_t* zeros, hipStream_t stream)
{
    const int64_t G = K / 64;
    const int64_t quads = (G + 3) / 4;
    const int64_t waves = (M + 7) / 8 * quads;
    const int64_t blocks = (waves + 3) / 4;
    quantize_act_kernel<GS><<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(
        x, M, G, ldx, quads, codes, flags, scales, zeros);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize_act(const uint16_t* x, int64_t M, int64_t K, int64_t ldx,
                               int lzs_group, uint8_t* codes, uint8_t* flags,
                               uint16_t* scales, int8_t* zeros, hipStream_t stream)
{
    switch (lzs_group) {
    case 8:
        return launch_gs<8>(x, M, K, ldx, codes, flags, scales, zeros, stream);
    case 16:
        return launch_gs<16>(x, M, K, ldx, codes, flags, scales, zeros, stream);
    case 32:
        return launch_gs<32>(x, M, K, ldx, codes, flags, scales, zeros, stream);
    default:
        return launch_gs<64>(x, M, K, ldx, codes, flags, scales, zeros, stream);
    }
}

}  // namespace quartz
