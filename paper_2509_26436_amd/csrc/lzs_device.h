// Device arithmetic of the activation quantizer (internal), shared by the
// standalone quantizer and the GEMM epilogue that quantizes its own output
// for the next layer.
//
// Stage 1 (Eq. 1, symmetric reading) of a 64-element group with max |x| =
// alpha:  s = fp16_rne_sat(alpha / 127), r = 1/s, |q| = min(rne(fp32(|x| r)), 127)
// Stage 2 (Eq. 2 and the right shift of Section 3) of a subgroup:
//         FLAG = max(29 - clz(OR |q|), 0), c = sgn * (|q| >> FLAG)
// Two exact shortcuts, both checked over their whole input domain:
//  - fp16_rne(alpha * fp32(1/127)) equals fp16_rne(fp32(alpha / 127)) for every
//    finite bf16 alpha (alpha / 127 is never within an fp32 ulp of an fp16
//    rounding boundary);
//  - one Newton step on the hardware reciprocal, r0 + r0 * (1 - s * r0) with
//    fused multiply-adds, equals the IEEE quotient 1/s for every finite fp16 s.
// rne(p) for 0 <= p < 2^22 is read from the low bits of fp32(p + 1.5 * 2^23):
// that sum has an ulp of 1, so its rounding is round-half-even of p.
//
// Values travel as bf16 pairs: dword d holds element 2i in its low half and
// element 2i + 1 in its high half (the memory order of a bf16 row).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace quartz {

constexpr float kMagic = 12582912.0f;          // 1.5 * 2^23
constexpr uint32_t kMagicBits = 0x4B400000u;
constexpr float kInv127 = 1.0f / 127.0f;       // fp32(1/127)

typedef unsigned short lzs_us2 __attribute__((ext_vector_type(2)));

struct GroupScale {
    uint32_t s16;    // fp16 bits of s
    float r;         // 1/s (0 when s = 0)
    bool clamp;      // the clamp to 127 can bind (subnormal or saturated s)
};

// alpha >= 0: the only overflow is +inf (0x7C00), saturated to 65504
__device__ __forceinline__ GroupScale group_scale(float alpha)
{
    GroupScale g;
    const _Float16 h = (_Float16)(alpha * kInv127);
    g.s16 = min((uint32_t)__builtin_bit_cast(uint16_t, h), 0x7BFFu);
    const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)g.s16);
    const float r0 = __builtin_amdgcn_rcpf(s);
    const float e = __builtin_fmaf(-s, r0, 1.0f);
    g.r = g.s16 == 0 ? 0.0f : __builtin_fmaf(r0, e, r0);
    // rne(|x| * r) <= 127 whenever s is a normal, unsaturated fp16 value
    // (checked for every bf16 alpha); only a subnormal or saturated s needs
    // the clamp
    g.clamp = (g.s16 - 1u) < 0x3FFu || g.s16 == 0x7BFFu;
    return g;
}

// |q| of the 8 values in d[0..3], as 4 pairs: pair k holds |q| of elements
// 2k and 2k + 1 in its two 16-bit halves.  `clamp` (wave-uniform) selects
// the clamped form.
template <bool CLAMP>
__device__ __forceinline__ void mag_pairs8_t(const uint32_t (&d)[4], float r, uint32_t (&p)[4])
{
    float f[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        f[2 * k] = __uint_as_float(d[k] << 16);
        f[2 * k + 1] = __uint_as_float(d[k] & 0xFFFF0000u);
    }
    uint32_t b[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        b[i] = __float_as_uint(fabsf(f[i]) * r + kMagic);
        if constexpr (CLAMP)
            b[i] = min(b[i], kMagicBits + 127u);
    }
    // the low byte of each sum is |q| (at most 127); two of them per pair
#pragma unroll
    for (int k = 0; k < 4; ++k)
        p[k] = __builtin_amdgcn_perm(b[2 * k + 1], b[2 * k], 0x0C040C00u);
}

__device__ __forceinline__ void mag_pairs8(const uint32_t (&d)[4], float r, bool clamp,
                                           uint32_t (&p)[4])
{
    if (clamp)
        mag_pairs8_t<true>(d, r, p);
    else
        mag_pairs8_t<false>(d, r, p);
}

// OR of the 8 magnitudes of mag_pairs8
__device__ __forceinline__ uint32_t pairs_or(const uint32_t (&p)[4])
{
    const uint32_t o = p[0] | p[1] | p[2] | p[3];
    return (o | (o >> 16)) & 0x7Fu;
}

// Eq. 2: the smallest shift that leaves at most 3 magnitude bits
__device__ __forceinline__ int lzs_flag(uint32_t mor)
{
    return max(29 - (int)__builtin_clz(mor | 1u), 0);
}

// sign bits of the 8 values moved to bit 3 of their nibbles (element 8j+i at
// nibble (i/2) + 4 (i%2))
__device__ __forceinline__ uint32_t sign_nibbles(const uint32_t (&d)[4])
{
    uint32_t S = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k)
        S |= (d[k] & 0x80008000u) >> (12 - 4 * k);
    return S;
}

// The nibble word of 8 codes: magnitudes t = |q| >> FLAG (at most 7, so no
// mask is needed; both halves of a pair are shifted at once and pair k lands
// at nibble k of each half), with a sign only where t is non-zero (t + 7 sets
// bit 3 iff t >= 1).
__device__ __forceinline__ uint32_t lzs_word(const uint32_t (&p)[4], uint32_t S, int fl)
{
    const lzs_us2 sh = {(unsigned short)fl, (unsigned short)fl};
    uint32_t T = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const lzs_us2 t = __builtin_bit_cast(lzs_us2, p[k]) >> sh;
        T |= __builtin_bit_cast(uint32_t, t) << (4 * k);
    }
    return T | (S & (T + 0x77777777u));
}

}  // namespace quartz
