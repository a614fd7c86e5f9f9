// Fused activation quantizer: Stage 1 (Eq. 1, symmetric reading) and Stage 2
// (Eq. 2 leading-zero suppression + right shift, Section 3) in one pass.
//
// One 64-element group is handled by a team of 8 lanes, each lane owning 8
// consecutive bf16 values (one 16-byte load).  A work item is 8 consecutive
// rows (one per team) x 2 consecutive groups: every load instruction reads
// one full 128-byte line per row, and since the outputs are stored
// K-group-major (codes [K/64][M][32], flags [K/64][M][64/G_s], scales
// [K/64][M]) every code store of a wave writes 256 contiguous bytes.  Waves
// walk the items with a grid stride and load the next item before working on
// the current one, so loads and arithmetic overlap.  Addresses are a
// wave-uniform base (scalar registers, one buffer resource per item) plus a
// small per-lane offset; rows past M fall outside the resource range, so
// their loads read zero and their stores are dropped.
//
// Per group:  alpha = max|x| (exact, 8-lane DPP max)
//             s = fp16_rne_sat(alpha * fp32(1/127)), r = 1/s
//             |q| = min(rne(fp32(|x| * r)), 127)     (sign kept aside;
//                   the clamp only binds for subnormal or saturated s)
// Per subgroup of G_s: FLAG = max(29 - clz(OR |q|), 0)   (DPP OR across lanes)
//                      c = sgn * (|q| >> FLAG)           (truncation toward 0)
// Two exact shortcuts, both checked over their whole input domain:
//  - fp16_rne(alpha * fp32(1/127)) equals fp16_rne(fp32(alpha / 127)) for every
//    finite bf16 alpha (alpha / 127 is never within an fp32 ulp of an fp16
//    rounding boundary);
//  - one Newton step on the hardware reciprocal, r0 + r0 * (1 - s * r0) with
//    fused multiply-adds, equals the IEEE quotient 1/s for every finite fp16 s.
// rne(p) for 0 <= p < 2^22 is read from the low bits of fp32(p + 1.5 * 2^23):
// that sum has an ulp of 1, so its rounding is round-half-even of p.
#include "quartz_internal.h"

namespace quartz {
namespace {

typedef __amdgpu_buffer_rsrc_t Rsrc;
typedef unsigned short us2 __attribute__((ext_vector_type(2)));

constexpr float kMagic = 12582912.0f;          // 1.5 * 2^23
constexpr uint32_t kMagicBits = 0x4B400000u;
constexpr float kInv127 = 1.0f / 127.0f;       // fp32(1/127)
constexpr int kRsrcWord3 = 0x00020000;         // raw buffer, out-of-range reads zero
constexpr int kNonTemporal = 2;                // cache policy: x is streamed once
constexpr int kGroupsPerItem = 2;
constexpr int kWavesPerBlock = 4;

// DPP controls (gfx9 encoding).
constexpr int kQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141;  // row_half_mirror: lane i <-> 7 - i within 8

__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

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

// One group of one lane: 8 bf16 values (a 16-byte load) -> the nibble word,
// the lane's FLAG and the group's fp16 scale.
template <int GS>
__device__ __forceinline__ void quantize_group(uint4 v, uint32_t& word, int& fl, uint32_t& s16)
{
    const uint32_t d[4] = {v.x, v.y, v.z, v.w};
    float f[8];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        f[2 * p] = __uint_as_float(d[p] << 16);
        f[2 * p + 1] = __uint_as_float(d[p] & 0xFFFF0000u);
    }
    float amax = fabsf(f[0]);
#pragma unroll
    for (int i = 1; i < 8; ++i)
        amax = fmaxf(amax, fabsf(f[i]));
    const float alpha = __uint_as_float(team8_max(__float_as_uint(amax)));

    // alpha >= 0: the only overflow is +inf (0x7C00), saturated to 65504
    const _Float16 h = (_Float16)(alpha * kInv127);
    s16 = min((uint32_t)__builtin_bit_cast(uint16_t, h), 0x7BFFu);
    const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)s16);
    const float r0 = __builtin_amdgcn_rcpf(s);
    const float e = __builtin_fmaf(-s, r0, 1.0f);
    const float r = s16 == 0 ? 0.0f : __builtin_fmaf(r0, e, r0);

    // rne(|x| * r) <= 127 whenever s is a normal, unsaturated fp16 value (checked
    // for every bf16 alpha); only groups with a subnormal or saturated scale
    // need the clamp, and the wave takes that path only if one of its groups does
    uint32_t b[8];
    const bool clamp = (s16 - 1u) < 0x3FFu || s16 == 0x7BFFu;
    if (__builtin_amdgcn_ballot_w64(clamp)) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            b[i] = min(__float_as_uint(fabsf(f[i]) * r + kMagic), kMagicBits + 127u);
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            b[i] = __float_as_uint(fabsf(f[i]) * r + kMagic);
    }
    const uint32_t mor = subgroup_or<GS>((b[0] | b[1] | b[2] | b[3] | b[4] | b[5] | b[6] | b[7]) & 0x7Fu);
    fl = max(29 - (int)__builtin_clz(mor | 1u), 0);

    // magnitudes t = |q| >> FLAG (at most 7, so no mask is needed): element
    // pair (2k, 2k+1) goes to the two 16-bit halves of one word (low bytes of
    // b), both halves are shifted at once, and pair k lands at nibble k of
    // each half, i.e. element 8j+i at nibble (i/2) + 4 (i%2)
    const us2 sh = {(unsigned short)fl, (unsigned short)fl};
    uint32_t T = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t pair = __builtin_amdgcn_perm(b[2 * k + 1], b[2 * k], 0x0C040C00u);
        const us2 t = __builtin_bit_cast(us2, pair) >> sh;
        T |= __builtin_bit_cast(uint32_t, t) << (4 * k);
    }
    // sign bits of x moved to bit 3 of each nibble
    uint32_t S = 0;
#pragma unroll
    for (int p = 0; p < 4; ++p)
        S |= (d[p] & 0x80008000u) >> (12 - 4 * p);
    // keep a sign only where the magnitude is non-zero: t + 7 sets bit 3 iff t >= 1
    word = T | (S & (T + 0x77777777u));
}

template <int GS>
__global__ __launch_bounds__(64 * kWavesPerBlock) void quantize_act_kernel(
    const uint16_t* __restrict__ x, int64_t M, int64_t G, int64_t ldx, int64_t quads,
    int64_t items, uint8_t* __restrict__ codes, uint8_t* __restrict__ flags,
    uint16_t* __restrict__ scales, int8_t* __restrict__ zeros)
{
    constexpr int FB = 64 / GS;     // flag bytes per (row, group)
    const int lane = threadIdx.x & 63;
    const int team = lane >> 3;
    const int u = lane & 7;
    // item indices are wave-uniform (scalar registers) and below 2^31: the
    // caller bounds M * K / 64 by 2^28
    const uint32_t stride = gridDim.x * kWavesPerBlock;
    const uint32_t nitems = (uint32_t)items;
    const uint32_t nquads = (uint32_t)quads;
    const uint32_t x_off = (uint32_t)((team * ldx + u * 8) * 2);

    struct Item {
        int64_t row0, g0;
        int rows, ng;       // valid rows (<= 8) and groups (<= kGroupsPerItem)
    };
    auto item_of = [&](uint32_t it) {
        Item t;
        t.row0 = (int64_t)(it / nquads) * 8;
        t.g0 = (int64_t)(it % nquads) * kGroupsPerItem;
        t.rows = (int)min(M - t.row0, (int64_t)8);
        t.ng = (int)min(G - t.g0, (int64_t)kGroupsPerItem);
        return t;
    };
    auto load = [&](const Item& t, uint4 (&v)[kGroupsPerItem]) {
        // bytes from the item's base to the end of its last valid row's K elements
        const Rsrc rx = make_rsrc(x + t.row0 * ldx + t.g0 * 64,
                                  (uint32_t)(((t.rows - 1) * ldx + (G - t.g0) * 64) * 2));
#pragma unroll
        for (int j = 0; j < kGroupsPerItem; ++j)
            v[j] = j < t.ng ? __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                                          rx, (int)(x_off + j * 128), 0, kNonTemporal))
                            : make_uint4(0, 0, 0, 0);
    };
    auto work = [&](const Item& t, const uint4 (&v)[kGroupsPerItem]) {
#pragma unroll
        for (int j = 0; j < kGroupsPerItem; ++j) {
            if (j >= t.ng)
                break;
            uint32_t word, s16;
            int fl;
            quantize_group<GS>(v[j], word, fl, s16);
            const int64_t rg0 = (t.g0 + j) * M + t.row0;     // (group, first row), K-group-major
            const Rsrc rc = make_rsrc(codes + rg0 * 32, (uint32_t)(t.rows * 32));
            __builtin_amdgcn_raw_buffer_store_b32(word, rc, team * 32 + u * 4, 0, 0);
            const Rsrc rf = make_rsrc(flags + rg0 * FB, (uint32_t)(t.rows * FB));
            if ((u & (GS / 8 - 1)) == 0)
                __builtin_amdgcn_raw_buffer_store_b8((uint8_t)fl, rf, team * FB + u / (GS / 8), 0, 0);
            if (u == 0) {
                const Rsrc rs = make_rsrc(scales + rg0, (uint32_t)(t.rows * 2));
                __builtin_amdgcn_raw_buffer_store_b16((uint16_t)s16, rs, team * 2, 0, 0);
                if (zeros) {
                    const Rsrc rz = make_rsrc(zeros + rg0, (uint32_t)t.rows);
                    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)0, rz, team, 0, 0);
                }
            }
        }
    };

    // two register sets: the item being worked on and the one being loaded
    uint4 va[kGroupsPerItem], vb[kGroupsPerItem];
    uint32_t it = blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (it >= nitems)
        return;
    Item ta = item_of(it), tb = ta;
    load(ta, va);
    while (true) {
        const uint32_t nb = it + stride;
        if (nb < nitems) {
            tb = item_of(nb);
            load(tb, vb);
        }
        work(ta, va);
        if (nb >= nitems)
            break;
        it = nb + stride;
        if (it < nitems) {
            ta = item_of(it);
            load(ta, va);
        }
        work(tb, vb);
        if (it >= nitems)
            break;
    }
}

template <int GS>
hipError_t launch_gs(const uint16_t* x, int64_t M, int64_t K, int64_t ldx, uint8_t* codes,
                     uint8_t* flags, uint16_t* scales, int8_t* zeros, hipStream_t stream)
{
    const int64_t G = K / 64;
    const int64_t quads = (G + kGroupsPerItem - 1) / kGroupsPerItem;
    const int64_t items = (M + 7) / 8 * quads;
    // up to 32 waves per CU on 256 CUs, each walking the items with a grid stride
    const int64_t max_blocks = 256 * 32 / kWavesPerBlock;
    const int64_t blocks = min((items + kWavesPerBlock - 1) / kWavesPerBlock, max_blocks);
    quantize_act_kernel<GS><<<dim3((unsigned)blocks), dim3(64 * kWavesPerBlock), 0, stream>>>(
        x, M, G, ldx, quads, items, codes, flags, scales, zeros);
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
