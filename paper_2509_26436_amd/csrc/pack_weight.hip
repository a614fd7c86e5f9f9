// Weight pre-pack: symmetric round-to-nearest int4 per 64-element group along
// K with an fp16 group scale (the weight setting of Appendix C), written in
// the GEMM's panel layout (see quartz_internal.h), plus the debug unpack.
// The per-channel variant (the LDM setting of the experimental-details
// appendix) first reduces each output channel's max |w| over all of K to one
// fp16 scale, then packs with it; the scale is stored in every group's scale
// slot, so the layout is the same.
//
// A team of 8 lanes owns one (column n, group g): each lane loads 8 bf16,
// the team reduces max|w| with DPP, every lane computes
//   s_w = fp16_rne_sat(max|w| / 7),  r = 1/s_w,  |wq| = min(rne(|w| * r), 7)
// and stores one 32-bit word of 8 sign-magnitude codes: the nibble word of the
// activation codes' order with its sign bits moved (weight_word_store), so the
// GEMM turns it into fp8 operands with a mask and a rotation.
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

typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;     // raw buffer, out-of-range reads zero
constexpr int kNonTemporal = 2;            // cache policy: w is streamed once
constexpr int kWavesPerBlock = 4;
constexpr int kGroupsPerItem = 2;

__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

// One column-group of one lane: 8 bf16 weights -> the nibble word; the team's
// fp16 scale.  r = 1/s is one Newton step on the hardware reciprocal, equal to
// the IEEE quotient for every finite fp16 s; the scale itself keeps the IEEE
// division (fp16(beta * fp32(1/7)) differs from fp16(beta / 7) for a few beta).
// PER_CHANNEL: s16 is the channel's scale on entry instead of the group's.
template <bool PER_CHANNEL>
__device__ __forceinline__ void pack_group(uint4 v, uint32_t& word, uint32_t& s16)
{
    const uint32_t d[4] = {v.x, v.y, v.z, v.w};
    float f[8];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        f[2 * p] = __uint_as_float(d[p] << 16);
        f[2 * p + 1] = __uint_as_float(d[p] & 0xFFFF0000u);
    }
    if constexpr (!PER_CHANNEL) {
        float amax = fabsf(f[0]);
#pragma unroll
        for (int i = 1; i < 8; ++i)
            amax = fmaxf(amax, fabsf(f[i]));
        uint32_t ab = __float_as_uint(amax);
        ab = max(ab, dpp_xor1(ab));
        ab = max(ab, dpp_xor2(ab));
        ab = max(ab, dpp_half_mirror(ab));
        const float beta = __uint_as_float(ab);
        s16 = f16_bits_rne_sat(beta / 7.0f);
    }
    const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)s16);
    const float r0 = __builtin_amdgcn_rcpf(s);
    const float e = __builtin_fmaf(-s, r0, 1.0f);
    const float r = s16 == 0 ? 0.0f : __builtin_fmaf(r0, e, r0);

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
    word = weight_word_store(T | (S & (T + 0x77777777u)));
}

// A work item is 8 consecutive columns of one panel (one team of 8 lanes per
// column, each lane 8 weights) x kGroupsPerItem groups.  Waves walk the items
// with a grid stride and load the next item before packing the current one.
// Columns past N read as zero (outside the buffer range) and pack to zero
// codes and scales, as the padded panel layout requires.
template <bool PER_CHANNEL>
__global__ __launch_bounds__(64 * kWavesPerBlock) void pack_weight_kernel(
    const uint16_t* __restrict__ w, int64_t N, int64_t K, int64_t panels,
    uint8_t* __restrict__ w_packed, uint16_t* __restrict__ w_scales)
{
    const int lane = threadIdx.x & 63;
    const int team = lane >> 3;            // column within the item
    const int u = lane & 7;
    const int64_t G = K / 64;
    // item indices are wave-uniform and below 2^31 (N * K / 64 <= 2^28)
    const uint32_t gpairs = (uint32_t)((G + kGroupsPerItem - 1) / kGroupsPerItem);
    const uint32_t nitems = (uint32_t)(panels * (kPanel / 8)) * gpairs;
    const uint32_t stride = gridDim.x * kWavesPerBlock;
    const uint32_t w_off = (uint32_t)((team * K + u * 8) * 2);

    struct Item {
        int64_t panel, n0, g0;   // first column n0 = panel * 64 + 8 c8
        int c8, ng;
    };
    auto item_of = [&](uint32_t it) {
        Item t;
        const uint32_t pc = it / gpairs;           // (panel, 8-column block)
        t.g0 = (int64_t)(it % gpairs) * kGroupsPerItem;
        t.panel = pc / (kPanel / 8);
        t.c8 = (int)(pc % (kPanel / 8));
        t.n0 = t.panel * kPanel + t.c8 * 8;
        t.ng = (int)min(G - t.g0, (int64_t)kGroupsPerItem);
        return t;
    };
    auto load = [&](const Item& t, uint4 (&v)[kGroupsPerItem]) {
        // bytes from the item's base to the end of its last real column's K weights
        const int64_t cols = min(N - t.n0, (int64_t)8);
        const uint32_t bytes =
            cols > 0 ? (uint32_t)(((cols - 1) * K + (G - t.g0) * 64) * 2) : 0u;
        const Rsrc rw = make_rsrc(w + (cols > 0 ? t.n0 * K + t.g0 * 64 : 0), bytes);
#pragma unroll
        for (int j = 0; j < kGroupsPerItem; ++j)
            v[j] = j < t.ng ? __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                                          rw, (int)(w_off + j * 128), 0, kNonTemporal))
                            : make_uint4(0, 0, 0, 0);
    };
    auto work = [&](const Item& t, const uint4 (&v)[kGroupsPerItem]) {
        const int cpan = t.c8 * 8 + team;
        const int64_t n = t.n0 + team;
#pragma unroll
        for (int j = 0; j < kGroupsPerItem; ++j) {
            if (j >= t.ng)
                break;
            uint32_t word, s16 = 0;
            const int64_t g = t.g0 + j;
            if constexpr (PER_CHANNEL)      // written to group 0's slot by row_scale_kernel
                s16 = reinterpret_cast<const uint16_t*>(
                    w_packed + t.panel * G * kChunkBytes + kChunkCodeBytes)[cpan];
            pack_group<PER_CHANNEL>(v[j], word, s16);
            uint8_t* chunk = w_packed + (t.panel * G + g) * kChunkBytes;
            reinterpret_cast<uint32_t*>(chunk + cpan * 32)[u] = word;
            if (u == 0 && (!PER_CHANNEL || g > 0)) {
                reinterpret_cast<uint16_t*>(chunk + kChunkCodeBytes)[cpan] = (uint16_t)s16;
                if (!PER_CHANNEL && n < N && w_scales)
                    w_scales[n * G + g] = (uint16_t)s16;
            }
        }
    };

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

// One wave per column n of the padded panels: s_w[n] = fp16_rne_sat(max over
// all of K of |w[n,k]| / 7), written to the scale slot of group 0 of its
// panel (0 for the padding columns) and to w_scales[n] if given.
__global__ __launch_bounds__(64 * kWavesPerBlock) void row_scale_kernel(
    const uint16_t* __restrict__ w, int64_t N, int64_t K, int64_t cols,
    uint8_t* __restrict__ w_packed, uint16_t* __restrict__ w_scales)
{
    const int64_t n = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (n >= cols)
        return;
    uint32_t ab = 0;           // max |w| as fp32 bits (non-negative floats order as their bits)
    if (n < N) {
        const Rsrc rw = make_rsrc(w + n * K, (uint32_t)(K * 2));
        for (int64_t k = (int64_t)lane * 8; k < K; k += 64 * 8) {
            const uint4 v = __builtin_bit_cast(
                uint4, __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(k * 2), 0, kNonTemporal));
            const uint32_t d[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int p = 0; p < 4; ++p)
                ab = max(ab, max((d[p] << 16) & 0x7FFFFFFFu, d[p] & 0x7FFF0000u));
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        ab = max(ab, (uint32_t)__shfl_xor((int)ab, off));
    if (lane == 0) {
        const uint32_t s16 = f16_bits_rne_sat(__uint_as_float(ab) / 7.0f);
        const int64_t G = K / 64;
        reinterpret_cast<uint16_t*>(w_packed + (n / kPanel) * G * kChunkBytes +
                                    kChunkCodeBytes)[n % kPanel] = (uint16_t)s16;
        if (n < N && w_scales)
            w_scales[n] = (uint16_t)s16;
    }
}

// One thread per (group g, column n): the sum of the 64 int4 weight codes of
// that group, int16 [K/64][N] (the weight group sums of the asymmetric mode).
__global__ __launch_bounds__(256) void weight_sums_kernel(const uint8_t* __restrict__ w_packed,
                                                          int64_t N, int64_t K,
                                                          int16_t* __restrict__ sums)
{
    const int64_t G = K / 64;
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= G * N)
        return;
    const int64_t g = t / N;
    const int64_t n = t - g * N;
    const uint4* src = reinterpret_cast<const uint4*>(
        w_packed + ((n / kPanel) * G + g) * kChunkBytes + (n % kPanel) * 32);
    int total = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint4 v = src[h];
        const uint32_t words[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int w = 0; w < 4; ++w)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint32_t nib = (weight_word_nibbles(words[w]) >> (4 * i)) & 0xFu;
                const int mag = (int)(nib & 7u);
                total += (nib & 8u) ? -mag : mag;
            }
    }
    sums[g * N + n] = (int16_t)total;
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
    const uint32_t word = weight_word_nibbles(reinterpret_cast<const uint32_t*>(
        w_packed + (panel * G + g) * kChunkBytes + cpan * 32)[j % 8]);
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

template <bool PER_CHANNEL>
hipError_t launch_pack(const uint16_t* w, int64_t N, int64_t K, uint8_t* w_packed,
                       uint16_t* w_scales, hipStream_t stream)
{
    const int64_t panels = (N + kPanel - 1) / kPanel;
    const int64_t gpairs = (K / 64 + kGroupsPerItem - 1) / kGroupsPerItem;
    const int64_t items = panels * (kPanel / 8) * gpairs;
    // up to 32 waves per compute unit, each walking the items with a grid stride
    const int64_t blocks = min((items + kWavesPerBlock - 1) / kWavesPerBlock,
                               (int64_t)device_compute_units() * 32 / kWavesPerBlock);
    pack_weight_kernel<PER_CHANNEL><<<dim3((unsigned)blocks), dim3(64 * kWavesPerBlock), 0, stream>>>(
        w, N, K, panels, w_packed, w_scales);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_pack_weight(const uint16_t* w, int64_t N, int64_t K, uint8_t* w_packed,
                              uint16_t* w_scales, hipStream_t stream)
{
    return launch_pack<false>(w, N, K, w_packed, w_scales, stream);
}

hipError_t launch_pack_weight_per_channel(const uint16_t* w, int64_t N, int64_t K,
                                          uint8_t* w_packed, uint16_t* w_scales,
                                          hipStream_t stream)
{
    const int64_t cols = (N + kPanel - 1) / kPanel * kPanel;
    const int64_t blocks = (cols + kWavesPerBlock - 1) / kWavesPerBlock;
    row_scale_kernel<<<dim3((unsigned)blocks), dim3(64 * kWavesPerBlock), 0, stream>>>(
        w, N, K, cols, w_packed, w_scales);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    return launch_pack<true>(w, N, K, w_packed, nullptr, stream);
}

hipError_t launch_weight_group_sums(const uint8_t* w_packed, int64_t N, int64_t K,
                                    int16_t* sums, hipStream_t stream)
{
    const int64_t threads = N * (K / 64);
    const int64_t blocks = (threads + 255) / 256;
    weight_sums_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(w_packed, N, K, sums);
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
