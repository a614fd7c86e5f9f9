// Fused LZS attention (the attention setting of the hardware appendix,
// Table 8) for head dimensions 64 and 128: the scores never leave registers.
//
// Per head, O = softmax(S) V with S = Q~ K~^T / sqrt(d); Q~, K~ quantized per
// token along d, V~^T per channel along the keys and the binary32 softmax
// output P per query row in 64-key groups, all by Eq. 1 and Eq. 2, and both
// products exact per-group integer products with the fp16 group scales
// applied in fp32 (the same quantities the unfused path materializes).
//
// The quantized P of a 64-key group needs the row's final max and sum (its
// group scale is fp16(max P / 127) of the normalized values), so each query
// row is swept twice:
//   pass 1  S of every 64-key chunk, the running max and sum of exp;
//   pass 2  S again, P = exp(S - max) / sum in binary32, the group scale,
//           Stage-1 codes, FLAG per subgroup and the truncated LZS values
//           d = c 2^FLAG, which go straight into the PV matrix product.
// The codes are rne(e R) with e = exp(S - max) and R = (1 / sum) (1 / s):
// one binary32 rounding fewer than rne(P r) with P rounded first, so a code
// can differ from the unfused path's only where P r lies within an ulp of a
// rounding boundary.
// One wave owns 32 queries of one head and streams every key chunk through
// registers: no LDS, no barriers.  The operands come from HBM / L2 already
// decoded to fp8 e4m3 (expand_fp8_kernel: every d = c 2^FLAG is exact in
// e4m3), since every chunk of K~ and V~^T is read by all L / 32 query waves of
// its head and decoding it once is cheaper than decoding it L / 32 times.
//
// Layout of the score tiles.  The product runs as S^T = K~ Q~^T on
// v_mfma_f32_32x32x64_f8f6f4 (rows: keys, columns: queries), so lane l holds
// query l % 32 and 16 keys per 32-key tile.  Row rho of key tile t is fed
// with key 32 ((rho >> 2) & 1) + 16 t + 4 (rho >> 3) + (rho & 3) of the
// chunk, which puts keys 32 h + 16 t + r (register r, h = l / 32) in lane l:
// each half-wave holds 32 consecutive keys of every query, so row maxima,
// group maxima and the FLAG subgroups (G_s <= 32) are in-lane reductions and
// a 64-key group takes one exchange between the two half-waves.  The same
// registers, converted to e4m3 and packed in the byte order the fp8 expansion
// gives V~^T's keys, are the k-slice of the PV product O^T = V~^T P~^T.
#include <algorithm>
#include <cmath>

#include "lzs_device.h"
#include "w4a4_gemm_kernel.h"

namespace quartz {

namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));


// ------------------------------------------------------------ fp8 expansion
// One (group, row) of a K-group-major LZS activation per thread: its 32 code
// bytes decoded to 64 e4m3 bytes at out[row][64 g ..] (word w of the group
// gives bytes 8 w .. 8 w + 7 in the order decode_nibbles_fp8 writes them).
template <int GS>
__global__ __launch_bounds__(256) void expand_fp8_kernel(const uint8_t* __restrict__ codes,
                                                         const uint8_t* __restrict__ flags,
                                                         int64_t rows, int64_t G,
                                                         uint8_t* __restrict__ out)
{
    constexpr int FB = 64 / GS;
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= rows * G)
        return;
    const int64_t g = t / rows, row = t % rows;
    const uint4 c0 = reinterpret_cast<const uint4*>(codes + t * 32)[0];
    const uint4 c1 = reinterpret_cast<const uint4*>(codes + t * 32)[1];
    const uint32_t w[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
    FlagRaw<GS> raw;
    if constexpr (FB == 8)
        raw = *reinterpret_cast<const uint2*>(flags + t * FB);
    else if constexpr (FB == 4)
        raw = *reinterpret_cast<const uint32_t*>(flags + t * FB);
    else if constexpr (FB == 2)
        raw = *reinterpret_cast<const uint16_t*>(flags + t * FB);
    else
        raw = flags[t];
    const uint2 f = flags_dwords<GS>(raw);
    uint32_t o[16];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        Fp8Table tb;
        switch (i / (GS / 8)) {
        case 0: tb = fp8_table_raw<0>(f.x, f.y); break;
        case 1: tb = fp8_table_raw<1>(f.x, f.y); break;
        case 2: tb = fp8_table_raw<2>(f.x, f.y); break;
        case 3: tb = fp8_table_raw<3>(f.x, f.y); break;
        case 4: tb = fp8_table_raw<4>(f.x, f.y); break;
        case 5: tb = fp8_table_raw<5>(f.x, f.y); break;
        case 6: tb = fp8_table_raw<6>(f.x, f.y); break;
        default: tb = fp8_table_raw<7>(f.x, f.y); break;
        }
        const uint2 d = decode_nibbles_fp8(w[i], tb);
        o[2 * i] = d.x;
        o[2 * i + 1] = d.y;
    }
    uint4* dst = reinterpret_cast<uint4*>(out + row * (64 * G) + 64 * g);
#pragma unroll
    for (int k = 0; k < 4; ++k)
        dst[k] = make_uint4(o[4 * k], o[4 * k + 1], o[4 * k + 2], o[4 * k + 3]);
}

__device__ __forceinline__ v8i load32(const uint8_t* p)
{
    const uint4 a = reinterpret_cast<const uint4*>(p)[0];
    const uint4 b = reinterpret_cast<const uint4*>(p)[1];
    return v8i{(int)a.x, (int)a.y, (int)a.z, (int)a.w, (int)b.x, (int)b.y, (int)b.z, (int)b.w};
}

// operand of the scale outer product (fp16 32x32x16, only k = 0 non-zero):
// the lower half-wave supplies k = 0 .. 7, the upper one k = 8 .. 15
__device__ __forceinline__ v8h scale_operand(uint16_t bits, int h)
{
    v8h v = {};
    v[0] = h ? (_Float16)0.0f : __builtin_bit_cast(_Float16, bits);
    return v;
}

__device__ __forceinline__ v16f mfma_fp8(const v8i& a, const v8i& b)
{
    const v16f zero = {};
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, zero, 0, 0, 0, 0, 0, 0);
}

__device__ __forceinline__ v16f mfma_outer(const v8h& a, const v8h& b)
{
    const v16f zero = {};
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, zero, 0, 0, 0);
}

__device__ __forceinline__ float xhalf(float v)       // value of lane l ^ 32
{
    return __shfl_xor(v, 32, 64);
}

// LDS staging of one 64-key chunk, in the order the MFMA lanes read it, so
// that every operand read is one conflict-free ds_read_b128 per 16 bytes:
//   K~   [t][g][j][lane][16 B]: lane (rho, h) of key tile t holds bytes
//        64 g + 32 h + 16 j .. of key kappa(t, rho) (see krow below);
//   V~^T [i][j][lane][16 B]: lane (n, h) holds bytes 32 h + 16 j .. of the
//        chunk's 64 keys of channel 32 i + n;
//   the key scales [t][g][rho] and the channel scales [D] (fp16).
template <int G, int W>
struct AttnStage {
    static constexpr int D = 64 * G;
    static constexpr int kK = 64 * D;               // K~ bytes
    static constexpr int kV = D * 64;               // V~^T bytes
    static constexpr int kSk = 64 * G * 2;
    static constexpr int kSv = D * 2;
    static constexpr int kBytes = kK + kV + kSk + kSv;
    static constexpr int kThreads = 64 * W;
    static constexpr int kKPieces = kK / 16, kVPieces = kV / 16;   // 16-byte pieces
    static constexpr int kKItems = (kKPieces + kThreads - 1) / kThreads;   // per thread
    static constexpr int kVItems = (kVPieces + kThreads - 1) / kThreads;
};

// One block: 4 waves, queries qb * 128 + 32 w .. + 31 of head `head`, which
// share the staged chunks.  qx / kx: [heads L][64 G] e4m3, qs / ks:
// [G][heads L] fp16; vx: [heads d][L] e4m3 (V^T), vs: [L / 64][heads d] fp16;
// o: bf16 [L][ldo], head h at columns h d ...
template <int GS, int G, int W>
__global__ __launch_bounds__(64 * W, 8 / W) void lzs_attention_fused_kernel(
    const uint8_t* __restrict__ qx, const uint16_t* __restrict__ qs,
    const uint8_t* __restrict__ kx, const uint16_t* __restrict__ ks,
    const uint8_t* __restrict__ vx, const uint16_t* __restrict__ vs, int64_t heads, int64_t L,
    float kexp, uint16_t* __restrict__ o, int64_t ldo, int64_t qblocks)
{
    using St = AttnStage<G, W>;
    constexpr int D = St::D;
    constexpr int TV = D / 32;                 // channel tiles of the PV product
    __shared__ __attribute__((aligned(16))) uint8_t smem[2][St::kBytes];
    // each wave's Q~ operand, [g][j][lane][16 B] (written and read by that wave only)
    __shared__ __attribute__((aligned(16))) uint8_t qsm[W][G * 2048];

    // blocks of one head on one XCD (consecutive block ids go round robin
    // over the 8 XCDs), so its K~ / V~^T chunks are shared in that L2
    const int64_t total = heads * qblocks;
    const int64_t bid = blockIdx.x;
    const int64_t logical = total % 8 == 0 ? (bid % 8) * (total / 8) + bid / 8 : bid;
    const int64_t head = logical / qblocks;
    const int tid = threadIdx.x;
    const int64_t q0 = (logical % qblocks) * (32 * W) + (tid >> 6) * 32;
    // a wave past the end of a ragged last block still loads and waits at
    // the barriers, and computes nothing (wave-uniform)
    const bool active = q0 < L;
    const int lane = tid & 63;
    const int n = lane & 31, h = lane >> 5;
    const int64_t rows = heads * L;
    const int64_t chunks = L / 64;

    // ---- cooperative staging: thread tid moves pieces tid + 256 p
    // K~ piece u: key u / (D / 16), bytes 16 (u % (D / 16)) of its row
    auto k_lds_off = [](int u) {
        const int key = u / (D / 16), part = u % (D / 16);
        const int g = part >> 2, hh = (part >> 1) & 1, j = part & 1;
        const int t = (key >> 4) & 1;
        const int rho = 8 * ((key >> 2) & 3) + 4 * (key >> 5) + (key & 3);
        return (((t * G + g) * 2 + j) * 64 + rho + 32 * hh) * 16;
    };
    // V~^T piece u: channel u / 4, bytes 16 (u % 4) of its 64-key row
    auto v_lds_off = [](int u) {
        const int ch = u >> 2, part = u & 3;
        const int i = ch >> 5, nn = ch & 31, hh = part >> 1, j = part & 1;
        return St::kK + ((i * 2 + j) * 64 + nn + 32 * hh) * 16;
    };
    // key scale of key `key`, group g -> [t][g][rho]
    auto sk_lds_off = [](int key, int g) {
        const int t = (key >> 4) & 1;
        const int rho = 8 * ((key >> 2) & 3) + 4 * (key >> 5) + (key & 3);
        return St::kK + St::kV + ((t * G + g) * 32 + rho) * 2;
    };
    v4u kr[St::kKItems], vr[St::kVItems];     // native vectors: kept in registers
    uint16_t skr = 0, svr = 0;
    auto load_chunk = [&](int64_t c, bool with_v) {
        const uint8_t* kc = kx + (head * L + 64 * c) * D;
#pragma unroll
        for (int p = 0; p < St::kKItems; ++p)
            if (tid + St::kThreads * p < St::kKPieces)
                kr[p] = reinterpret_cast<const v4u*>(kc)[tid + St::kThreads * p];
        if (tid < 64 * G)
            skr = ks[(tid >> 6) * rows + head * L + 64 * c + (tid & 63)];
        if (with_v) {
#pragma unroll
            for (int p = 0; p < St::kVItems; ++p) {
                const int u = tid + St::kThreads * p;
                if (u < St::kVPieces)
                    vr[p] = *reinterpret_cast<const v4u*>(vx + (head * D + (u >> 2)) * L + 64 * c + 16 * (u & 3));
            }
            if (tid < D)
                svr = vs[c * heads * D + head * D + tid];
        }
    };
    auto store_chunk = [&](int b, bool with_v) {
        uint8_t* s = smem[b];
#pragma unroll
        for (int p = 0; p < St::kKItems; ++p)
            if (tid + St::kThreads * p < St::kKPieces)
                *reinterpret_cast<v4u*>(s + k_lds_off(tid + St::kThreads * p)) = kr[p];
        if (tid < 64 * G)
            *reinterpret_cast<uint16_t*>(s + sk_lds_off(tid & 63, tid >> 6)) = skr;
        if (with_v) {
#pragma unroll
            for (int p = 0; p < St::kVItems; ++p)
                if (tid + St::kThreads * p < St::kVPieces)
                    *reinterpret_cast<v4u*>(s + v_lds_off(tid + St::kThreads * p)) = vr[p];
            if (tid < D)
                *reinterpret_cast<uint16_t*>(s + St::kK + St::kV + St::kSk + 2 * tid) = svr;
        }
    };
    auto lds32 = [&](const uint8_t* s) {
        const uint4 a = *reinterpret_cast<const uint4*>(s);
        const uint4 b = *reinterpret_cast<const uint4*>(s + 1024);
        return v8i{(int)a.x, (int)a.y, (int)a.z, (int)a.w, (int)b.x, (int)b.y, (int)b.z, (int)b.w};
    };

    uint8_t* const qw = qsm[tid >> 6];
    v8h sqop[G];
    if (active) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const uint4* src = reinterpret_cast<const uint4*>(qx + (head * L + q0 + n) * D + 64 * g + 32 * h);
            *reinterpret_cast<uint4*>(qw + g * 2048 + lane * 16) = src[0];
            *reinterpret_cast<uint4*>(qw + g * 2048 + 1024 + lane * 16) = src[1];
            sqop[g] = scale_operand(qs[g * rows + head * L + q0 + n], h);
        }
    }

    // x (the scores before the 1 / sqrt(d)) of the chunk in stage s: x[t][r]
    // belongs to key 32 h + 16 t + r of the chunk and query q0 + n
    auto scores = [&](const uint8_t* s, v16f (&x)[2]) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const v8i kop = lds32(s + (t * G + g) * 2048 + lane * 16);
                const uint16_t skb =
                    *reinterpret_cast<const uint16_t*>(s + St::kK + St::kV + ((t * G + g) * 32 + n) * 2);
                const v16f sc = mfma_outer(scale_operand(skb, h), sqop[g]);
                const v16f p = mfma_fp8(kop, lds32(qw + g * 2048 + lane * 16));
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    x[t][r] = g == 0 ? p[r] * sc[r] : fmaf(p[r], sc[r], x[t][r]);
            }
        }
    };

    // pass 1: per lane the running max and sum of exp over its 32 keys of
    // every chunk, in the base-2 domain: exp(S - m) = 2^((x - m_x) kexp)
    float m = -INFINITY, l = 0.0f;
    load_chunk(0, false);
    store_chunk(0, false);
    __syncthreads();
    for (int64_t c = 0; c < chunks; ++c) {
        if (c + 1 < chunks)
            load_chunk(c + 1, false);
        if (active) {
            v16f x[2];
            scores(smem[c & 1], x);
            // four independent chains per reduction (a lone chain of 32
            // dependent instructions leaves the SIMD idle between them)
            float cm4[4] = {x[0][0], x[0][8], x[1][0], x[1][8]};
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    cm4[2 * t + r / 8] = fmaxf(cm4[2 * t + r / 8], x[t][r]);
            const float mn = fmaxf(m, fmaxf(fmaxf(cm4[0], cm4[1]), fmaxf(cm4[2], cm4[3])));
            const float nmk = -mn * kexp;
            float cs4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    cs4[2 * t + r / 8] += __builtin_amdgcn_exp2f(fmaf(x[t][r], kexp, nmk));
            l = l * __builtin_amdgcn_exp2f((m - mn) * kexp) + ((cs4[0] + cs4[1]) + (cs4[2] + cs4[3]));
            m = mn;
        }
        if (c + 1 < chunks)
            store_chunk((c + 1) & 1, false);
        __syncthreads();
    }
    {
        // the two half-waves' keys of the same query (identical result in both)
        const float mo = xhalf(m), lo = xhalf(l);
        const float mf = fmaxf(m, mo);
        l = l * __builtin_amdgcn_exp2f((m - mf) * kexp) + lo * __builtin_amdgcn_exp2f((mo - mf) * kexp);
        m = mf;
    }
    const float inv_l = 1.0f / l;
    const float nmk = -m * kexp;

    v16f acc[TV];
#pragma unroll
    for (int i = 0; i < TV; ++i)
        acc[i] = v16f{};
    // pass 2
    load_chunk(0, true);
    store_chunk(0, true);
    __syncthreads();
    for (int64_t c = 0; c < chunks; ++c) {
        if (c + 1 < chunks)
            load_chunk(c + 1, true);
        if (active) {
            const uint8_t* s = smem[c & 1];
            v16f x[2];
            scores(s, x);
            // e = exp(S - max) and its maximum over each 8 consecutive keys
            float e8[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    #pragma unroll
            for (int t = 0; t < 2; ++t)
    #pragma unroll
                for (int r = 0; r < 16; ++r) {
                    x[t][r] = __builtin_amdgcn_exp2f(fmaf(x[t][r], kexp, nmk));
                    e8[2 * t + r / 8] = fmaxf(e8[2 * t + r / 8], x[t][r]);
                }
            // alpha = max of P = e / sum over the 64-key group (binary32 rounding
            // of e * inv_l is monotone, so max(e) * inv_l is that maximum), the
            // fp16 scale and r = 1 / s.  The code multiplier R = inv_l r takes
            // P r in one rounding instead of two.
            float emax = fmaxf(fmaxf(e8[0], e8[1]), fmaxf(e8[2], e8[3]));
            emax = fmaxf(emax, xhalf(emax));
            const float alpha = emax * inv_l;
            const _Float16 s16 = (_Float16)(alpha / 127.0f);
            const uint16_t sbits = __builtin_bit_cast(uint16_t, s16);
            const float R = sbits == 0 ? 0.0f : inv_l * (1.0f / (float)s16);
            // FLAG of each subgroup from its largest code (q = min(rne(e R), 127)
            // is monotone in e), as the e4m3 table of c 2^FLAG, c = 0 .. 7: the
            // base table with FLAG added to the exponent field of entries 1 .. 7
            auto flag_of = [&](float emx) {
                return lzs_flag((uint32_t)fminf(__builtin_rintf(emx * R), 127.0f));
            };
            int fl[4];
            if constexpr (GS == 8) {
    #pragma unroll
                for (int k = 0; k < 4; ++k)
                    fl[k] = flag_of(e8[k]);
            } else if constexpr (GS == 16) {
    #pragma unroll
                for (int t = 0; t < 2; ++t)
                    fl[2 * t] = fl[2 * t + 1] = flag_of(fmaxf(e8[2 * t], e8[2 * t + 1]));
            } else {
                float e4 = fmaxf(fmaxf(e8[0], e8[1]), fmaxf(e8[2], e8[3]));
                if constexpr (GS == 64)
                    e4 = emax;
                fl[0] = fl[1] = fl[2] = fl[3] = flag_of(e4);
            }
            Fp8Table tab[4];
    #pragma unroll
            for (int k = 0; k < 4; ++k) {
                tab[k].lo = kTabLo + (uint32_t)fl[k] * 0x08080800u;
                tab[k].hi = kTabHi + (uint32_t)fl[k] * 0x08080808u;
            }
            // The k-slice of P~^T: dword k of the operand holds keys (relative to
            // the half-wave) 8 (k / 2) + {0, 4, 1, 5} (k even) or {2, 6, 3, 7}
            // (k odd), the byte order of the expanded V~^T rows.  Per dword the
            // four Stage-1 codes q = min(rne(e R), 127) as bytes (v_cvt_pk_u8_f32
            // rounds to nearest even), c = q >> FLAG per byte, and the e4m3 value
            // of c 2^FLAG by table lookup.
            v8i pop;
    #pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int t = k >> 2, base = 8 * ((k >> 1) & 1) + 2 * (k & 1);
                const int sub = k >> 1;
                uint32_t w = __builtin_amdgcn_cvt_pk_u8_f32(fminf(x[t][base] * R, 127.0f), 0u, 0u);
                w = __builtin_amdgcn_cvt_pk_u8_f32(fminf(x[t][base + 4] * R, 127.0f), 1u, w);
                w = __builtin_amdgcn_cvt_pk_u8_f32(fminf(x[t][base + 1] * R, 127.0f), 2u, w);
                w = __builtin_amdgcn_cvt_pk_u8_f32(fminf(x[t][base + 5] * R, 127.0f), 3u, w);
                const uint32_t cb = (w >> fl[sub]) & 0x07070707u;
                pop[k] = (int)__builtin_amdgcn_perm(tab[sub].hi, tab[sub].lo, cb);
            }
            const v8h spop = scale_operand(sbits, h);
#pragma unroll
            for (int i = 0; i < TV; ++i) {
                const v8i vop = lds32(s + St::kK + i * 2048 + lane * 16);
                const uint16_t svb = *reinterpret_cast<const uint16_t*>(
                    s + St::kK + St::kV + St::kSk + (32 * i + n) * 2);
                const v16f sc = mfma_outer(scale_operand(svb, h), spop);
                const v16f p = mfma_fp8(vop, pop);
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc[i][r] = fmaf(p[r], sc[r], acc[i][r]);
            }
        }
        if (c + 1 < chunks)
            store_chunk((c + 1) & 1, true);
        __syncthreads();
    }
    if (!active)
        return;
    // O^T tile i, register r: channel 32 i + 8 (r / 4) + 4 h + r % 4 of query
    // q0 + n; four consecutive channels per 8-byte store
    typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
    typedef float f2 __attribute__((ext_vector_type(2)));
    uint16_t* orow = o + (q0 + n) * ldo + head * D;
#pragma unroll
    for (int i = 0; i < TV; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const f2 a = {acc[i][4 * j], acc[i][4 * j + 1]};
            const f2 b = {acc[i][4 * j + 2], acc[i][4 * j + 3]};
            const uint2 v = {__builtin_bit_cast(uint32_t, __builtin_convertvector(a, bf2)),
                             __builtin_bit_cast(uint32_t, __builtin_convertvector(b, bf2))};
            *reinterpret_cast<uint2*>(orow + 32 * i + 8 * j + 4 * h) = v;
        }
}

template <int GS, int W>
void launch_fused_w(const uint8_t* qx, const uint16_t* qs, const uint8_t* kx, const uint16_t* ks,
                    const uint8_t* vx, const uint16_t* vs, int64_t heads, int64_t L, int64_t d,
                    uint16_t* o, int64_t ldo, hipStream_t stream)
{
    const int64_t qblocks = (L + 32 * W - 1) / (32 * W);
    const dim3 grid((unsigned)(heads * qblocks)), block(64 * W);
    const float kexp = (float)(1.4426950408889634 / std::sqrt((double)d));
    if (d == 64)
        lzs_attention_fused_kernel<GS, 1, W><<<grid, block, 0, stream>>>(qx, qs, kx, ks, vx, vs, heads, L,
                                                                          kexp, o, ldo, qblocks);
    else
        lzs_attention_fused_kernel<GS, 2, W><<<grid, block, 0, stream>>>(qx, qs, kx, ks, vx, vs, heads, L,
                                                                          kexp, o, ldo, qblocks);
}

// Block shape: 8 query waves per block share each staged chunk among twice
// the queries of 4 and cost ~8.5 % less per wave, but run one block per CU,
// so a launch takes whole rounds of 8-wave blocks; with 4-wave blocks (two
// per CU) a partial last round is spread one block per CU and runs faster
// per block, so the time grows about linearly with the block count.  Take 8
// waves only when the last round of 8-wave blocks is nearly full (measured
// at L = 4608: 40 heads, 2.81 rounds, 0.88 against 0.93 ms; 32 and 64 heads,
// 2.25 and 4.5 rounds, favour 4 waves).
template <int GS>
hipError_t launch_fused_gs(const uint8_t* qx, const uint16_t* qs, const uint8_t* kx,
                           const uint16_t* ks, const uint8_t* vx, const uint16_t* vs,
                           int64_t heads, int64_t L, int64_t d, uint16_t* o, int64_t ldo,
                           hipStream_t stream)
{
    const int64_t cus = std::max<int64_t>(1, device_compute_units());
    const int64_t blocks8 = heads * ((L + 255) / 256);
    const int64_t rounds8 = (blocks8 + cus - 1) / cus;
    if (rounds8 * cus * 100 <= blocks8 * 109)
        launch_fused_w<GS, 8>(qx, qs, kx, ks, vx, vs, heads, L, d, o, ldo, stream);
    else
        launch_fused_w<GS, 4>(qx, qs, kx, ks, vx, vs, heads, L, d, o, ldo, stream);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_expand_fp8(const uint8_t* codes, const uint8_t* flags, int64_t rows, int64_t K,
                             int lzs_group, uint8_t* out, hipStream_t stream)
{
    const int64_t G = K / 64;
    const dim3 grid((unsigned)((rows * G + 255) / 256)), block(256);
    switch (lzs_group) {
    case 8: expand_fp8_kernel<8><<<grid, block, 0, stream>>>(codes, flags, rows, G, out); break;
    case 16: expand_fp8_kernel<16><<<grid, block, 0, stream>>>(codes, flags, rows, G, out); break;
    case 32: expand_fp8_kernel<32><<<grid, block, 0, stream>>>(codes, flags, rows, G, out); break;
    default: expand_fp8_kernel<64><<<grid, block, 0, stream>>>(codes, flags, rows, G, out); break;
    }
    return hipGetLastError();
}

hipError_t launch_attention_fused(const uint8_t* qx, const uint16_t* qs, const uint8_t* kx,
                                  const uint16_t* ks, const uint8_t* vx, const uint16_t* vs,
                                  int64_t heads, int64_t L, int64_t d, int lzs_group, uint16_t* o,
                                  int64_t ldo, hipStream_t stream)
{
    switch (lzs_group) {
    case 8: return launch_fused_gs<8>(qx, qs, kx, ks, vx, vs, heads, L, d, o, ldo, stream);
    case 16: return launch_fused_gs<16>(qx, qs, kx, ks, vx, vs, heads, L, d, o, ldo, stream);
    case 32: return launch_fused_gs<32>(qx, qs, kx, ks, vx, vs, heads, L, d, o, ldo, stream);
    default: return launch_fused_gs<64>(qx, qs, kx, ks, vx, vs, heads, L, d, o, ldo, stream);
    }
}

}  // namespace quartz
