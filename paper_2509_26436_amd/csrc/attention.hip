// LZS attention (the attention setting of the paper's hardware appendix,
// Table 8): per head O = softmax(Q K^T / sqrt(d)) V, with every operand of
// both products an activation quantized by Eq. 1 and Eq. 2 (Q and K per
// token along d, V^T per channel along the keys, the binary32 softmax output
// per query row in 64-key groups), and both products exact per-group integer
// products on the matrix cores with the fp16 group scales applied in fp32.
//
// Kernels here:
//  * quantize_vt_kernel: V [rows][ldv] (rows = head * L + key) quantized along
//    the keys, i.e. the activation quantizer on V^T, through an LDS transpose
//    of 64 keys x 32 channels;
//  * softmax_quantize_kernel: one wave per score row: the row's max and sum
//    (online, then across the wave), P = exp(S - max) / sum in binary32, and
//    the activation quantizer on P per 64-key group (a team of 8 lanes per
//    group, as the standalone quantizer);
//  * the GEMM kernel template's ATTN instantiations for the scores (fp32
//    output) and the PV product (bf16 output).
#include <cmath>

#include "lzs_device.h"
#include "w4a4_gemm_kernel.h"

namespace quartz {

hipError_t launch_gemm_attn_scores(const GemmLaunch& a, hipStream_t stream)
{
    return launch_mode<false, false, false, true, true>(a, stream);
}

hipError_t launch_gemm_attn_pv(const GemmLaunch& a, hipStream_t stream)
{
    return launch_mode<false, false, false, true, false>(a, stream);
}

namespace {

constexpr int kDppQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror: lane i <-> 7 - i within 8

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// max over the 8 lanes of a team (non-negative floats order as their bits)
__device__ __forceinline__ uint32_t team_max(uint32_t v)
{
    v = max(v, dpp_u<kDppQuadXor1>(v));
    v = max(v, dpp_u<kDppQuadXor2>(v));
    v = max(v, dpp_u<kDppHalfMirror>(v));
    return v;
}

template <int GS>
__device__ __forceinline__ uint32_t team_subgroup_or(uint32_t v)
{
    if constexpr (GS >= 16)
        v |= dpp_u<kDppQuadXor1>(v);
    if constexpr (GS >= 32)
        v |= dpp_u<kDppQuadXor2>(v);
    if constexpr (GS >= 64)
        v |= dpp_u<kDppHalfMirror>(v);
    return v;
}

// Stores of one team's group (lane u of the team holds code word u): the
// group's 32 code bytes, its FLAG bytes and its fp16 scale, K-group-major
// (plane g, row `row` of `rows`).
template <int GS>
__device__ __forceinline__ void store_group(uint8_t* codes, uint8_t* flags, uint16_t* scales,
                                            int64_t rows, int64_t g, int64_t row, int u,
                                            uint32_t word, int fl, uint32_t s16)
{
    constexpr int FB = 64 / GS;
    const int64_t rg = g * rows + row;
    reinterpret_cast<uint32_t*>(codes + rg * 32)[u] = word;
    if ((u & (GS / 8 - 1)) == 0)
        flags[rg * FB + u / (GS / 8)] = (uint8_t)fl;
    if (u == 0)
        scales[rg] = (uint16_t)s16;
}

// ---------------------------------------------------------------- V^T
// Block: one head, one 64-key group g, 32 channels c0 .. c0 + 31 (256
// threads).  Thread t loads 8 channels of key t / 4 (16 bytes) and writes
// them transposed into LDS; team j (8 lanes) then quantizes channel c0 + j's
// 64 keys, lane u holding keys 8u .. 8u + 7 as one 16-byte LDS read.
template <int GS>
__global__ __launch_bounds__(256) void quantize_vt_kernel(
    const uint16_t* __restrict__ v, int64_t L, int64_t d, int64_t ldv, int64_t heads,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ flags, uint16_t* __restrict__ scales)
{
    __shared__ __attribute__((aligned(16))) uint16_t tile[32][64 + 8];
    const int64_t cblocks = d / 32;
    const int64_t gblocks = L / 64;
    const int64_t b = blockIdx.x;
    const int64_t h = b / (gblocks * cblocks);
    const int64_t g = (b / cblocks) % gblocks;
    const int64_t c0 = (b % cblocks) * 32;
    const int t = threadIdx.x;
    {
        const int key = t >> 2, cq = (t & 3) * 8;
        const uint4 x = *reinterpret_cast<const uint4*>(v + (h * L + g * 64 + key) * ldv + c0 + cq);
        const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            tile[cq + 2 * i][key] = (uint16_t)w[i];
            tile[cq + 2 * i + 1][key] = (uint16_t)(w[i] >> 16);
        }
    }
    __syncthreads();
    const int team = t >> 3, u = t & 7;
    const uint4 x = *reinterpret_cast<const uint4*>(&tile[team][8 * u]);
    const uint32_t dw[4] = {x.x, x.y, x.z, x.w};
    float amax = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        amax = fmaxf(amax, fabsf(__uint_as_float(dw[k] << 16)));
        amax = fmaxf(amax, fabsf(__uint_as_float(dw[k] & 0xFFFF0000u)));
    }
    const float alpha = __uint_as_float(team_max(__float_as_uint(amax)));
    const GroupScale gsc = group_scale(alpha);
    uint32_t p[4];
    mag_pairs8(dw, gsc.r, __builtin_amdgcn_ballot_w64(gsc.clamp) != 0, p);
    const int fl = lzs_flag(team_subgroup_or<GS>(pairs_or(p)));
    const uint32_t word = lzs_word(p, sign_nibbles(dw), fl);
    store_group<GS>(codes, flags, scales, heads * d, g, h * d + c0 + team, u, word, fl, gsc.s16);
}

// -------------------------------------------------------- softmax + quantize
// One wave per row of S (N scores, N % 64 == 0).  Lane l covers, for chunk i,
// group 8 i + l / 8 and its elements 8 (l % 8) .. + 7 (32 contiguous bytes).
// Pass 1: per lane the running (max, sum of exp) over its chunks, combined
// across the wave; pass 2: P = exp(S - max) * (1 / sum), then per group the
// activation quantizer on binary32 values: alpha = max P (team max),
// s = fp16(alpha / 127) (IEEE quotient, RNE), r = 1 / s, q = min(rne(P r), 127)
// (P >= 0, so no signs), FLAG per subgroup, c = q >> FLAG.
template <int GS>
__global__ __launch_bounds__(256) void softmax_quantize_kernel(
    const float* __restrict__ S, int64_t M, int64_t N, int64_t lds, uint8_t* __restrict__ codes,
    uint8_t* __restrict__ flags, uint16_t* __restrict__ scales)
{
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= M)
        return;                                   // wave-uniform
    const int lane = threadIdx.x & 63;
    const int64_t G = N / 64;
    const int chunks = (int)((G + 7) / 8);
    const float* srow = S + row * lds;
    auto load8 = [&](int i, float (&x)[8]) {
        const int64_t g = 8 * (int64_t)i + (lane >> 3);
        if (g < G) {
            const float4* p = reinterpret_cast<const float4*>(srow + g * 64 + 8 * (lane & 7));
            const float4 a = p[0], b = p[1];
            x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
            x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
        } else {
#pragma unroll
            for (int k = 0; k < 8; ++k)
                x[k] = -INFINITY;
        }
    };
    // pass 1: running max and sum of exp per lane
    float m = -INFINITY, s = 0.0f;
    for (int i = 0; i < chunks; ++i) {
        float x[8];
        load8(i, x);
        float cm = x[0];
#pragma unroll
        for (int k = 1; k < 8; ++k)
            cm = fmaxf(cm, x[k]);
        if (cm == -INFINITY)
            continue;
        const float mn = fmaxf(m, cm);
        float cs = 0.0f;
#pragma unroll
        for (int k = 0; k < 8; ++k)
            cs += expf(x[k] - mn);
        s = s * expf(m - mn) + cs;
        m = mn;
    }
    // across the wave: (m, s) pairs combined by max and rescaled sum
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float mo = __shfl_xor(m, off, 64);
        const float so = __shfl_xor(s, off, 64);
        const float mn = fmaxf(m, mo);
        s = (m == -INFINITY ? 0.0f : s * expf(m - mn)) + (mo == -INFINITY ? 0.0f : so * expf(mo - mn));
        m = mn;
    }
    const float inv = 1.0f / s;
    // pass 2: probabilities and their quantization
    const int u = lane & 7;
    for (int i = 0; i < chunks; ++i) {
        const int64_t g = 8 * (int64_t)i + (lane >> 3);
        float x[8];
        load8(i, x);
        float pv[8], amax = 0.0f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            pv[k] = expf(x[k] - m) * inv;
            amax = fmaxf(amax, pv[k]);
        }
        const float alpha = __uint_as_float(team_max(__float_as_uint(amax)));
        const _Float16 h = (_Float16)(alpha / 127.0f);
        const uint32_t s16 = __builtin_bit_cast(uint16_t, h);
        const float sc = (float)h;
        const float r = s16 == 0 ? 0.0f : 1.0f / sc;
        uint32_t q[8], mor = 0;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            q[k] = (uint32_t)min(__builtin_rintf(pv[k] * r), 127.0f);
            mor |= q[k];
        }
        const int fl = lzs_flag(team_subgroup_or<GS>(mor));
        // element 8 u + k of the group is nibble (k / 2) + 4 (k % 2) of word u
        uint32_t word = 0;
#pragma unroll
        for (int k = 0; k < 8; ++k)
            word |= (q[k] >> fl) << (4 * ((k >> 1) + 4 * (k & 1)));
        if (g < G)
            store_group<GS>(codes, flags, scales, M, g, row, u, word, fl, s16);
    }
}

}  // namespace

hipError_t launch_quantize_vt(const uint16_t* v, int64_t heads, int64_t L, int64_t d, int64_t ldv,
                              int lzs_group, uint8_t* codes, uint8_t* flags, uint16_t* scales,
                              hipStream_t stream)
{
    const int64_t blocks = heads * (L / 64) * (d / 32);
    const dim3 grid((unsigned)blocks), block(256);
    switch (lzs_group) {
    case 8:
        quantize_vt_kernel<8><<<grid, block, 0, stream>>>(v, L, d, ldv, heads, codes, flags, scales);
        break;
    case 16:
        quantize_vt_kernel<16><<<grid, block, 0, stream>>>(v, L, d, ldv, heads, codes, flags, scales);
        break;
    case 32:
        quantize_vt_kernel<32><<<grid, block, 0, stream>>>(v, L, d, ldv, heads, codes, flags, scales);
        break;
    default:
        quantize_vt_kernel<64><<<grid, block, 0, stream>>>(v, L, d, ldv, heads, codes, flags, scales);
        break;
    }
    return hipGetLastError();
}

hipError_t launch_softmax_quantize(const float* S, int64_t M, int64_t N, int64_t lds, int lzs_group,
                                   uint8_t* codes, uint8_t* flags, uint16_t* scales,
                                   hipStream_t stream)
{
    const dim3 grid((unsigned)((M + 3) / 4)), block(256);
    switch (lzs_group) {
    case 8:
        softmax_quantize_kernel<8><<<grid, block, 0, stream>>>(S, M, N, lds, codes, flags, scales);
        break;
    case 16:
        softmax_quantize_kernel<16><<<grid, block, 0, stream>>>(S, M, N, lds, codes, flags, scales);
        break;
    case 32:
        softmax_quantize_kernel<32><<<grid, block, 0, stream>>>(S, M, N, lds, codes, flags, scales);
        break;
    default:
        softmax_quantize_kernel<64><<<grid, block, 0, stream>>>(S, M, N, lds, codes, flags, scales);
        break;
    }
    return hipGetLastError();
}

}  // namespace quartz
