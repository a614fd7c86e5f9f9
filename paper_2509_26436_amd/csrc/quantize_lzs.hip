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
// Per group:  alpha = max|x| (exact, 8-lane DPP max), then Stage 1 and the
// per-subgroup Stage 2 of lzs_device.h, the subgroup OR taken across the
// lanes of a subgroup with DPP.
#include "lzs_device.h"
#include "quartz_internal.h"

namespace quartz {
namespace {

typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;         // raw buffer, out-of-range reads zero
constexpr int kNonTemporal = 2;                // cache policy: x is streamed once
constexpr int kGroupsPerItem = 2;
constexpr int kWavesPerBlock = 4;

// Stage-1 modes: symmetric per group (Eq. 1, reading R1), static per tensor
// (the LDM setting), asymmetric per group (Eq. 1's zero point, repaired).
enum { kModeSym = 0, kModeStatic = 1, kModeAsym = 2 };

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

// min / max of floats over the 8 lanes of a team
__device__ __forceinline__ float team8_fmin(float v)
{
    v = fminf(v, __uint_as_float(dpp<kQuadXor1>(__float_as_uint(v))));
    v = fminf(v, __uint_as_float(dpp<kQuadXor2>(__float_as_uint(v))));
    v = fminf(v, __uint_as_float(dpp<kHalfMirror>(__float_as_uint(v))));
    return v;
}
__device__ __forceinline__ float team8_fmax(float v)
{
    v = fmaxf(v, __uint_as_float(dpp<kQuadXor1>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp<kQuadXor2>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp<kHalfMirror>(__float_as_uint(v))));
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
// the lane's FLAG and the group's fp16 scale.  kModeStatic (the LDM
// setting): the reciprocal r of the caller's per-tensor scale replaces the
// group's, values beyond 127 s clip, and there is no group scale.
// kModeAsym: the group's range [min(x_min, 0), max(x_max, 0)] spread over
// the 255 signed levels: s = fp16(span / 254), z = -127 - rne(lo r),
// q = clamp(rne(x r) + z, -127, 127), then Stage 2 on q (its sign and
// magnitude, not those of x); z8 receives z.
template <int GS, int MODE>
__device__ __forceinline__ void quantize_group(uint4 v, float r_static, uint32_t& word, int& fl,
                                               uint32_t& s16, int& z8)
{
    const uint32_t d[4] = {v.x, v.y, v.z, v.w};
    z8 = 0;
    if constexpr (MODE == kModeAsym) {
        float f[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f[2 * k] = __uint_as_float(d[k] << 16);
            f[2 * k + 1] = __uint_as_float(d[k] & 0xFFFF0000u);
        }
        float mn = 0.0f, mx = 0.0f;              // the range always includes 0
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            mn = fminf(mn, f[i]);
            mx = fmaxf(mx, f[i]);
        }
        mn = team8_fmin(mn);
        mx = team8_fmax(mx);
        const float span = mx - mn;
        const _Float16 h = (_Float16)(span / 254.0f);
        s16 = min((uint32_t)__builtin_bit_cast(uint16_t, h), 0x7BFFu);
        const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)s16);
        const float r0 = __builtin_amdgcn_rcpf(s);
        const float e = __builtin_fmaf(-s, r0, 1.0f);
        const float r = s16 == 0 ? 0.0f : __builtin_fmaf(r0, e, r0);
        // rne of a value in (-2^22, 2^22) from the low bits of fp32(v + 1.5 * 2^23)
        auto rne_int = [](float t) { return (int)(__float_as_uint(t + kMagic) - kMagicBits); };
        const int z = min(max(-127 - rne_int(mn * r), -127), 127);
        z8 = z;
        uint32_t p[4], S = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int q0 = min(max(rne_int(f[2 * k] * r) + z, -127), 127);
            const int q1 = min(max(rne_int(f[2 * k + 1] * r) + z, -127), 127);
            p[k] = (uint32_t)abs(q0) | ((uint32_t)abs(q1) << 16);
            S |= ((uint32_t)q0 >> 31) << (3 + 4 * k);
            S |= ((uint32_t)q1 >> 31) << (19 + 4 * k);
        }
        fl = lzs_flag(subgroup_or<GS>(pairs_or(p)));
        word = lzs_word(p, S, fl);
        return;
    }
    if constexpr (MODE == kModeStatic) {
        uint32_t p[4];
        mag_pairs8_t<true>(d, r_static, p);
        s16 = 0;
        fl = lzs_flag(subgroup_or<GS>(pairs_or(p)));
        word = lzs_word(p, sign_nibbles(d), fl);
        return;
    }
    // max |x| of the lane's 8 values (the fp32 values are those mag_pairs8
    // forms), then across the team (non-negative floats order as their bits)
    float f[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        f[2 * k] = __uint_as_float(d[k] << 16);
        f[2 * k + 1] = __uint_as_float(d[k] & 0xFFFF0000u);
    }
    float amax = fabsf(f[0]);
#pragma unroll
    for (int i = 1; i < 8; ++i)
        amax = fmaxf(amax, fabsf(f[i]));
    const float alpha = __uint_as_float(team8_max(__float_as_uint(amax)));

    const GroupScale gs = group_scale(alpha);
    s16 = gs.s16;
    // the wave takes the clamped path only if one of its groups needs it
    uint32_t p[4];
    mag_pairs8(d, gs.r, __builtin_amdgcn_ballot_w64(gs.clamp) != 0, p);
    fl = lzs_flag(subgroup_or<GS>(pairs_or(p)));
    word = lzs_word(p, sign_nibbles(d), fl);
}

template <int GS, int MODE>
__global__ __launch_bounds__(64 * kWavesPerBlock) void quantize_act_kernel(
    const uint16_t* __restrict__ x, int64_t M, int64_t G, int64_t ldx, int64_t quads,
    int64_t items, uint8_t* __restrict__ codes, uint8_t* __restrict__ flags,
    uint16_t* __restrict__ scales, int8_t* __restrict__ zeros, float r_static)
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
            int fl, z8;
            quantize_group<GS, MODE>(v[j], r_static, word, fl, s16, z8);
            const int64_t rg0 = (t.g0 + j) * M + t.row0;     // (group, first row), K-group-major
            const Rsrc rc = make_rsrc(codes + rg0 * 32, (uint32_t)(t.rows * 32));
            __builtin_amdgcn_raw_buffer_store_b32(word, rc, team * 32 + u * 4, 0, 0);
            const Rsrc rf = make_rsrc(flags + rg0 * FB, (uint32_t)(t.rows * FB));
            if ((u & (GS / 8 - 1)) == 0)
                __builtin_amdgcn_raw_buffer_store_b8((uint8_t)fl, rf, team * FB + u / (GS / 8), 0, 0);
            if (MODE != kModeStatic && u == 0) {
                const Rsrc rs = make_rsrc(scales + rg0, (uint32_t)(t.rows * 2));
                __builtin_amdgcn_raw_buffer_store_b16((uint16_t)s16, rs, team * 2, 0, 0);
                if (zeros) {
                    const Rsrc rz = make_rsrc(zeros + rg0, (uint32_t)t.rows);
                    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)z8, rz, team, 0, 0);
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

template <int GS, int MODE>
hipError_t launch_gs(const uint16_t* x, int64_t M, int64_t K, int64_t ldx, uint8_t* codes,
                     uint8_t* flags, uint16_t* scales, int8_t* zeros, float r_static,
                     hipStream_t stream)
{
    const int64_t G = K / 64;
    const int64_t quads = (G + kGroupsPerItem - 1) / kGroupsPerItem;
    const int64_t items = (M + 7) / 8 * quads;
    // up to 32 waves per compute unit, each walking the items with a grid stride
    const int64_t max_blocks = (int64_t)device_compute_units() * 32 / kWavesPerBlock;
    const int64_t blocks = min((items + kWavesPerBlock - 1) / kWavesPerBlock, max_blocks);
    quantize_act_kernel<GS, MODE><<<dim3((unsigned)blocks), dim3(64 * kWavesPerBlock), 0, stream>>>(
        x, M, G, ldx, quads, items, codes, flags, scales, zeros, r_static);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_any(const uint16_t* x, int64_t M, int64_t K, int64_t ldx, int lzs_group,
                      uint8_t* codes, uint8_t* flags, uint16_t* scales, int8_t* zeros,
                      float r_static, hipStream_t stream)
{
    switch (lzs_group) {
    case 8:
        return launch_gs<8, MODE>(x, M, K, ldx, codes, flags, scales, zeros, r_static, stream);
    case 16:
        return launch_gs<16, MODE>(x, M, K, ldx, codes, flags, scales, zeros, r_static, stream);
    case 32:
        return launch_gs<32, MODE>(x, M, K, ldx, codes, flags, scales, zeros, r_static, stream);
    default:
        return launch_gs<64, MODE>(x, M, K, ldx, codes, flags, scales, zeros, r_static, stream);
    }
}

}  // namespace

hipError_t launch_quantize_act(const uint16_t* x, int64_t M, int64_t K, int64_t ldx,
                               int lzs_group, uint8_t* codes, uint8_t* flags,
                               uint16_t* scales, int8_t* zeros, bool asymmetric,
                               hipStream_t stream)
{
    if (asymmetric)
        return launch_any<kModeAsym>(x, M, K, ldx, lzs_group, codes, flags, scales, zeros, 0.0f,
                                     stream);
    return launch_any<kModeSym>(x, M, K, ldx, lzs_group, codes, flags, scales, zeros, 0.0f,
                                stream);
}

hipError_t launch_quantize_act_static(const uint16_t* x, int64_t M, int64_t K, int64_t ldx,
                                      float scale, int lzs_group, uint8_t* codes,
                                      uint8_t* flags, hipStream_t stream)
{
    // r = 1/s, the IEEE quotient (host division)
    return launch_any<kModeStatic>(x, M, K, ldx, lzs_group, codes, flags, nullptr, nullptr, 1.0f / scale,
                            stream);
}

}  // namespace quartz
