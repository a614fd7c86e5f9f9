// The per-group W4A4 linear layer with a bf16 output (quartz_w4a4_linear and
// its workspace and scratch variants): the kernel of the headline path.
//
// Same arithmetic as the kernel template of w4a4_gemm_kernel.h -- per 64-group
// g the fp8 MFMA gives the exact integer product P_g, one fp16 MFMA the tile of
// scale products s_a[m,g] s_w[n,g], and one FMA per output folds
// P_g * (s_a s_w) into fp32 -- with the data paths arranged for the cost of
// each operand:
//
//  * Tile 128 x 256 (M x N), 8 math waves as 2 (M) x 4 (N), 64 x 64 each, and
//    4 decode waves.  The activation decode (a table lookup per FLAG, ~8
//    instructions per 8 codes) is done once per tile row by the decode waves
//    and shared through LDS; per output it costs half of what a 256-row tile
//    with 128 columns costs.
//  * The weights pass through LDS as stored (4 bits each, 8 KB per group) and
//    each math wave turns the words of its own 64 columns into fp8 operands
//    itself: a stored weight word becomes fp8 with one mask, or a rotation
//    and a mask (weight_word_store), so the 2-fold redundancy (two math waves
//    share each column) costs less than staging decoded bytes would.  LDS
//    traffic per 128 x 256 x 64 step: 16 KB written, 48 KB read, against 24
//    KB and 64 KB for the template's 256 x 128 step (decoded operands).
//  * The decoded activations (8 KB per group), the raw weight words and both
//    groups of scales pass through LDS in three stages.
//
// The persistent schedule, the stream-K split with its partial-sum finisher
// and the output code are those of the template (gemm_schedule.h), for this
// tile shape.
#pragma once

#include "w4a4_gemm_kernel.h"

namespace quartz {
namespace {

constexpr int LBM = 128;                    // tile rows (M)
constexpr int LBN = 256;                    // tile columns (N)
constexpr int kLinMathWaves = 8;            // 2 (M) x 4 (N), 64 x 64 each
constexpr int kLinDecodeWaves = 4;
constexpr int kLinThreads = 64 * (kLinMathWaves + kLinDecodeWaves);
constexpr int kLinWavesN = 4;
constexpr int kLinStages = 3;
constexpr int kLinPanels = LBN / kPanel;    // weight panels per tile
static_assert(kLinStages == kPipelineStages, "segments are padded to whole rounds of the stages");
static_assert(64 * kLinDecodeWaves == 2 * LBM && 64 * kLinDecodeWaves == LBN, "decode roles");

// STATIC: the LDM setting (one per-tensor activation scale, per-channel
// weight scales): no per-group scales, so the fp8 MFMAs accumulate the exact
// integer sum in place and the output code applies act_scale * s_w[n].  With
// no dequantization pipeline the math waves have the registers to take their
// weight words straight from global memory (a ring three groups deep), and
// only the decoded activations pass through LDS.
// QOUT: the output quantized for the next layer (quartz_w4a4_linear_quantize)
// instead of bf16: each math wave runs its 64 x 64 tile through the
// activation quantizer in its own LDS region (quantize_tile_out).
// ASYM: the asymmetric mode's zero points z[g][m] and weight group sums
// W[g][n]: each tile's fp8 MFMA starts from the correction -z (x) W (one more
// fp16 outer-product MFMA, exact in fp32), so it yields P_g - z W_g, the group
// product of the activations s (d - z); -z and W * 2^-9 pass through LDS as
// fp16 next to the group scales.
template <int GS, bool GELU, bool SPLIT, bool STATIC, bool QOUT, bool ASYM>
__global__ __launch_bounds__(kLinThreads) void w4a4_linear_kernel(
    const uint8_t* __restrict__ codes, const uint8_t* __restrict__ flags,
    const uint16_t* __restrict__ scales, const uint8_t* __restrict__ w_packed,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ y, int64_t M, int64_t N, int64_t K,
    int64_t ldy, GemmSchedule sch, uint32_t* __restrict__ counters, float* __restrict__ slots,
    float act_scale, QuantOut qout, const int8_t* __restrict__ zeros,
    const int16_t* __restrict__ wsums)
{
    static_assert(!ASYM || (!STATIC && !QOUT), "the asymmetric mode has per-group scales and a bf16 output");
    // One LDS array: the operand stages at the lowest addresses (so every
    // fragment address of the main loop is a lane offset plus a 16-bit
    // immediate), then the math waves' output transpose regions.
    //   As:  decoded activations, stage-major; row r's 16-byte chunk c at
    //        swz(r, c)
    //   Bs:  stored weight words of the tile's columns, k half h of column c
    //        (16 bytes) at h * LBN * 16 + c * 16: the 16 lanes of a read phase
    //        cover 256 consecutive bytes
    //   sas, sws: group scales as fp16 bits; entries LBM (LBN) stay 0: the
    //        upper half-wave's k slots of the outer-product MFMA read them
    //   szs, sWs (ASYM): -z and W * 2^-9 as fp16 bits, padded the same way
    //   Ts:  8 KB per math wave: its bf16 output tile on the way to 16-byte
    //        stores, or to the quantizer (QOUT)
    constexpr int kAsBytes = kLinStages * LBM * 64;
    constexpr int kBsBytes = kLinStages * LBN * 32;
    constexpr int kSasBytes = kLinStages * (LBM + 8) * 2;
    constexpr int kSwsBytes = kLinStages * (LBN + 8) * 2;
    constexpr int kSzsBytes = ASYM ? kSasBytes : 0;
    constexpr int kSWsBytes = ASYM ? kSwsBytes : 0;
    constexpr int kStageLds = kAsBytes + kBsBytes + kSasBytes + kSwsBytes + kSzsBytes + kSWsBytes;
    static_assert(kStageLds % 16 == 0, "transpose regions stay 16-byte aligned");
    __shared__ __attribute__((aligned(16)))
    uint8_t lds_main[kStageLds + kLinMathWaves * kTransposeBytes];
    uint8_t (*const As)[LBM * 64] = reinterpret_cast<uint8_t (*)[LBM * 64]>(lds_main);
    uint8_t (*const Bs)[LBN * 32] = reinterpret_cast<uint8_t (*)[LBN * 32]>(lds_main + kAsBytes);
    uint16_t (*const sas)[LBM + 8] =
        reinterpret_cast<uint16_t (*)[LBM + 8]>(lds_main + kAsBytes + kBsBytes);
    uint16_t (*const sws)[LBN + 8] =
        reinterpret_cast<uint16_t (*)[LBN + 8]>(lds_main + kAsBytes + kBsBytes + kSasBytes);
    uint16_t (*const szs)[LBM + 8] = reinterpret_cast<uint16_t (*)[LBM + 8]>(
        lds_main + kAsBytes + kBsBytes + kSasBytes + kSwsBytes);
    uint16_t (*const sWs)[LBN + 8] = reinterpret_cast<uint16_t (*)[LBN + 8]>(
        lds_main + kAsBytes + kBsBytes + kSasBytes + kSwsBytes + kSzsBytes);
    uint8_t* const Ts = lds_main + kStageLds;

    constexpr int FB = 64 / GS;                 // flag bytes per (group, row)
    const int tid = threadIdx.x;
    const int uwave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t blk = (int32_t)blockIdx.x;
    const int G = (int)(K / 64);
    const int64_t panels = (N + kPanel - 1) / kPanel;

    auto fresh_schedule = [&] {
        GemmSchedule s = sch;
        asm volatile("" : "+s"(s.tiles_n), "+s"(s.groups), "+s"(s.blocks), "+s"(s.sk_first),
                          "+s"(s.sk_q), "+s"(s.sk_r), "+s"(s.sk_blocks), "+s"(s.sk_tiles));
        return s;
    };
    auto fresh_tid = [&] {
        int t = tid;
        asm volatile("" : "+v"(t));
        return t;
    };

    // ------------------------------------------------------ decode waves
    // Thread d: half ah of activation row dr of the tile (16 code bytes, the
    // half's FLAGs), that row's scale (ah == 0 stores it), and the 32 code
    // bytes and the scale of tile column d.  Rows past M and columns past the
    // packed panels fall outside the buffer ranges and read as zero; they only
    // feed outputs that are never stored.
    if (uwave >= kLinMathWaves) {
        const int d = tid - kLinMathWaves * 64;
        const int dr = d >> 1, ah = d & 1;
        const uint32_t b_off = (uint32_t)((d / kPanel) * G * kChunkBytes + (d % kPanel) * 32);
        const uint32_t sw_off =
            (uint32_t)((d / kPanel) * G * kChunkBytes + kChunkCodeBytes + (d % kPanel) * 2);

        GemmCursor fc;
        int fg = 0, fend = 0;
        bool fdone = false;
        int64_t m0 = 0, panel0 = 0;
        uint32_t rows = 0, b_bytes = 0;
        auto set_ranges = [&] {
            m0 = (int64_t)fc.tm * LBM;
            panel0 = (int64_t)fc.tn * kLinPanels;
            rows = (uint32_t)min(M - m0, (int64_t)LBM);
            const int64_t blk_panels = min(panels - panel0, (int64_t)kLinPanels);
            b_bytes = (uint32_t)((blk_panels - 1) * G * kChunkBytes + kChunkBytes);
        };
        if (!cursor_begin(fresh_schedule(), blk, fc))
            return;
        fg = fc.sg.g0;
        fend = fc.sg.g0 + padded_steps(fc.sg.g1 - fc.sg.g0);
        set_ranges();

        struct Raw {
            uint4 a, b0, b1;
            uint32_t f;
            uint16_t sa, sw;
            uint32_t z, wsum;        // ASYM: the raw zero point (int8) and group sum (int16)
        };
        // as in the template: every step loads (a no-op step reloads the
        // segment's last group), so the compiler waits for exactly the ring
        // slot it decodes
        auto fetch_next = [&](Raw& r) {
            const int g = min(fg, fc.sg.g1 - 1);
            const int64_t prow = (int64_t)g * M + m0;
            const Rsrc ra = make_rsrc(codes + prow * 32, rows * 32u);
            const Rsrc rf = make_rsrc(flags + prow * FB, rows * (uint32_t)FB);
            const Rsrc rs = make_rsrc(STATIC ? nullptr : scales + prow, STATIC ? 0u : rows * 2u);
            const Rsrc rb = make_rsrc(w_packed + (panel0 * G + g) * kChunkBytes, b_bytes);
            r.a = __builtin_bit_cast(
                uint4, __builtin_amdgcn_raw_buffer_load_b128(ra, (int)((uint32_t)dr * 32u + ah * 16u), 0, 0));
            r.f = load_half_flags<GS>(rf, (uint32_t)dr * FB, ah);
            if constexpr (!STATIC) {
                r.sa = __builtin_amdgcn_raw_buffer_load_b16(rs, dr * 2, 0, 0);
                r.sw = __builtin_amdgcn_raw_buffer_load_b16(rb, (int)sw_off, 0, 0);
                r.b0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rb, (int)b_off, 0, 0));
                r.b1 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rb, (int)b_off + 16, 0, 0));
            }
            if constexpr (ASYM) {
                const Rsrc rz = make_rsrc(zeros + prow, rows);
                r.z = __builtin_amdgcn_raw_buffer_load_b8(rz, dr, 0, 0);
                const int64_t n0 = panel0 * kPanel;
                const Rsrc rw = make_rsrc(wsums + (int64_t)g * N + n0,
                                          n0 < N ? (uint32_t)((N - n0) * 2) : 0u);
                r.wsum = __builtin_amdgcn_raw_buffer_load_b16(rw, d * 2, 0, 0);
            }
            if (!fdone && ++fg == fend) {
                if (cursor_next(fresh_schedule(), blk, fc)) {
                    fg = fc.sg.g0;
                    fend = fc.sg.g0 + padded_steps(fc.sg.g1 - fc.sg.g0);
                    set_ranges();
                } else {
                    fdone = true;
                }
            }
        };
        // decode the half row into its two 16-byte chunks of LDS stage `buf`;
        // word w of the half uses FLAG w / (G_s / 8) of the half
        auto stage = [&](const Raw& r, int buf) {
            const uint32_t a[4] = {r.a.x, r.a.y, r.a.z, r.a.w};
            constexpr int kWordsPerFlag = GS / 8;
            uint2 o[4];
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                Fp8Table t;
                switch (w / kWordsPerFlag) {
                case 0: t = fp8_table_raw<0>(r.f, 0u); break;
                case 1: t = fp8_table_raw<1>(r.f, 0u); break;
                case 2: t = fp8_table_raw<2>(r.f, 0u); break;
                default: t = fp8_table_raw<3>(r.f, 0u); break;
                }
                o[w] = decode_nibbles_fp8(a[w], t);
            }
            *reinterpret_cast<uint4*>(As[buf] + swz(dr, 2 * ah)) = make_uint4(o[0].x, o[0].y, o[1].x, o[1].y);
            *reinterpret_cast<uint4*>(As[buf] + swz(dr, 2 * ah + 1)) = make_uint4(o[2].x, o[2].y, o[3].x, o[3].y);
            if constexpr (!STATIC) {
                *reinterpret_cast<uint4*>(Bs[buf] + d * 16) = r.b0;
                *reinterpret_cast<uint4*>(Bs[buf] + LBN * 16 + d * 16) = r.b1;
                if (ah == 0)
                    sas[buf][dr] = r.sa;
                sws[buf][d] = r.sw;
            }
            if constexpr (ASYM) {
                // -z and W * 2^-9 (the unit of the weight operands), both exact
                // in fp16 (|z| <= 128, |W| <= 512)
                if (ah == 0)
                    szs[buf][dr] = __builtin_bit_cast(uint16_t, (_Float16)(-(int)(int8_t)r.z));
                sWs[buf][d] = __builtin_bit_cast(
                    uint16_t, (_Float16)((float)(int)(int16_t)r.wsum * (1.0f / kWeightUnitInv)));
            }
        };

        // The decode of each group gates the math waves two steps later: these
        // waves run at raised priority, keep 2 x 3 groups of loads in flight
        // and decode two groups ahead, one workgroup barrier per step (plus
        // one before the first), as many as the math waves execute.
        constexpr int kRing = 2 * kLinStages;
        Raw ring[kRing];
        __builtin_amdgcn_s_setprio(2);
        if (!STATIC && d < 8 * kLinStages) {
            sas[d >> 3][LBM + (d & 7)] = 0;
            sws[d >> 3][LBN + (d & 7)] = 0;
            if constexpr (ASYM) {
                szs[d >> 3][LBM + (d & 7)] = 0;
                sWs[d >> 3][LBN + (d & 7)] = 0;
            }
        }
        const int steps = gemm_steps(fresh_schedule(), blk);
#pragma unroll
        for (int i = 0; i < kRing; ++i)
            fetch_next(ring[i]);
        stage(ring[0], 0);
        fetch_next(ring[0]);
        stage(ring[1], 1);
        fetch_next(ring[1]);
        lds_sync();
        auto dstep = [&](int u) {
            const int k = (u + 2) % kRing;
            stage(ring[k], (u + 2) % kLinStages);
            fetch_next(ring[k]);
            lds_sync();
        };
        int s = 0;
        for (; s + kRing <= steps; s += kRing) {
#pragma unroll
            for (int u = 0; u < kRing; ++u)
                dstep(u);
        }
#pragma unroll
        for (int u = 0; u < kRing - 1; ++u)
            if (s + u < steps)
                dstep(u);
        return;
    }

    // -------------------------------------------------------- math waves
    int lane, wm, wn, l32, khalf;
    uint32_t a_lo, a_hi, b_lo;
    auto set_fragment_indices = [&] {
        const int t = fresh_tid();
        const int w = __builtin_amdgcn_readfirstlane(t >> 6) & (kLinMathWaves - 1);
        lane = t & 63;
        wm = w / kLinWavesN;
        wn = w % kLinWavesN;
        l32 = t & 31;
        khalf = (t >> 5) & 1;
        a_lo = (uint32_t)swz(wm * WM + l32, 2 * khalf);
        a_hi = (uint32_t)swz(wm * WM + l32, 2 * khalf + 1);
        b_lo = (uint32_t)(khalf * LBN * 16 + (wn * WN + l32) * 16);
    };
    auto frag_at = [](const uint8_t* stage, uint32_t lo, uint32_t hi, int rows_off) {
        const uint4 l = *reinterpret_cast<const uint4*>(stage + lo + rows_off * 64);
        const uint4 h = *reinterpret_cast<const uint4*>(stage + hi + rows_off * 64);
        return v8i{(int)l.x, (int)l.y, (int)l.z, (int)l.w, (int)h.x, (int)h.y, (int)h.z, (int)h.w};
    };

    // ---- weight operands: the stored words of this lane's column (tile j) and
    // k half, from LDS stage buf, decoded in registers
    auto raw_w = [&](int j, int buf) {
        return *reinterpret_cast<const uint4*>(Bs[buf] + b_lo + j * 32 * 16);
    };
    auto decode_w = [](const uint4& c) {
        const uint2 w0 = decode_weight_fp8(c.x), w1 = decode_weight_fp8(c.y);
        const uint2 w2 = decode_weight_fp8(c.z), w3 = decode_weight_fp8(c.w);
        return v8i{(int)w0.x, (int)w0.y, (int)w1.x, (int)w1.y, (int)w2.x, (int)w2.y, (int)w3.x, (int)w3.y};
    };

    // ---- STATIC: the weight words straight from global memory, in a ring of
    // three groups (this lane's 16 bytes of each of the wave's two column
    // tiles) fetched by a cursor of its own that walks the same segments
    // group by group; ring0 is the group being multiplied.
    struct WRaw {
        uint4 c0, c1;
    };
    WRaw ring0, ring1, ring2;
    GemmCursor bcur;
    int bg = 0;
    bool bdone = false;
    int64_t bpanel = 0;
    auto bfetch = [&](WRaw& r) {
        const int g = min(bg, bcur.sg.g1 - 1);
        const Rsrc rb = make_rsrc(w_packed + (bpanel * G + g) * kChunkBytes,
                                  bpanel < panels ? (uint32_t)kChunkCodeBytes : 0u);
        const int off = (int)((uint32_t)l32 * 32u + (uint32_t)khalf * 16u);
        r.c0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rb, off, 0, 0));
        r.c1 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rb, off + 1024, 0, 0));
        if (!bdone && ++bg == bcur.sg.g1) {
            if (cursor_next(fresh_schedule(), blk, bcur)) {
                bg = bcur.sg.g0;
                bpanel = (int64_t)bcur.tn * kLinPanels + wn;
            } else {
                bdone = true;
            }
        }
    };

    v16f acc[TM][TN];
    v8i bf, bf1, af[TM];
    // operands of the scale outer-product MFMA (fp16 32x32x8, k = 0 the only
    // non-zero one): dword 0 holds the scale in its low half (a zero-extending
    // 16-bit LDS load; the upper half-wave, k = 4..7, reads the zero pad),
    // dword 1 is zero once and never written again, so refilling an operand
    // is one LDS load and no vector instruction
    typedef int v2i __attribute__((ext_vector_type(2)));
    v2i sa_op[TM], sw_op[TN];
    v2i za_op[TM], ws_op[TN];                // ASYM: -z and W, the same way
    uint4 wraw;
    auto load_af = [&](int i, int buf) { af[i] = frag_at(As[buf], a_lo, a_hi, i * 32); };
    auto load_a = [&](int i, int buf) {
        af[i] = frag_at(As[buf], a_lo, a_hi, i * 32);
        sa_op[i][0] = (int)sas[buf][khalf ? LBM : wm * WM + i * 32 + l32];
        if constexpr (ASYM)
            za_op[i][0] = (int)szs[buf][khalf ? LBM : wm * WM + i * 32 + l32];
    };
    auto load_sw = [&](int j, int buf) {
        sw_op[j][0] = (int)sws[buf][khalf ? LBN : wn * WN + j * 32 + l32];
        if constexpr (ASYM)
            ws_op[j][0] = (int)sWs[buf][khalf ? LBN : wn * WN + j * 32 + l32];
    };

    v16f pc, sc;                             // tile product and scale tile in flight
    const v16f zero = {};
    auto fma_rows = [&](int i, int j, const v16f& p, const v16f& sc, int r0) {
#pragma unroll
        for (int r = r0; r < r0 + 8; ++r)
            acc[i][j][r] = fmaf(p[r], sc[r], acc[i][j][r]);
        asm volatile("" : "+v"(acc[i][j]));
    };
    auto fma_tile = [&](int i, int j, const v16f& p, const v16f& sc) {
        fma_rows(i, j, p, sc, 0);
        fma_rows(i, j, p, sc, 8);
    };
    // the 32 x 32 tile of scale products: fp16 MFMA with one non-zero k
    // (32x32x8 runs at the rate of 32x32x16, 15-17 ns, with operands half as
    // wide)
    auto scale_tile = [&](int i, int j) {
        typedef _Float16 v4h __attribute__((ext_vector_type(4)));
        __builtin_amdgcn_s_setprio(3);
        const v16f sc = __builtin_amdgcn_mfma_f32_32x32x8f16(
            __builtin_bit_cast(v4h, sa_op[i]), __builtin_bit_cast(v4h, sw_op[j]), zero, 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
        return sc;
    };
    // the fp8 product of rows i with the weight operand in bf (column tile
    // j); ASYM: started from the correction tile -z (x) W, so it is P_g - z W_g
    auto mfma_p = [&](int i, int j) {
        typedef _Float16 v4h __attribute__((ext_vector_type(4)));
        __builtin_amdgcn_s_setprio(3);
        v16f c = zero;
        if constexpr (ASYM)
            c = __builtin_amdgcn_mfma_f32_32x32x8f16(__builtin_bit_cast(v4h, za_op[i]),
                                                     __builtin_bit_cast(v4h, ws_op[j]), zero, 0, 0, 0);
        const v16f p = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[i], bf, c, 0, 0, 0, 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
        return p;
    };

    // One group from LDS stage cb, tiles in the order (0,0) (1,0) (0,1) (1,1),
    // the fp8 product issued one step ahead of the FMAs that use it (see the
    // template).  On entry af[] and sa_op[] hold this group's activation
    // operands, bf and sw_op[0] its column-0 weight operands, wraw its column-1
    // weight words (read a step ahead, so the LDS latency is hidden: each
    // read goes out one step before its decode).  Column 1 is decoded once
    // column 0's products are issued; the next group's operands (LDS stage
    // nb) are read after their last use here, unless this is a segment's
    // last group.
    // STATIC: the four fp8 products of a group accumulate in place; column
    // 1's operand is decoded while column 0's products run, the next group's
    // column 0 once the ring has advanced (issuing all four products back to
    // back, with both columns decoded a group ahead, was slower: the wave
    // then stalls on the busy matrix unit with its loads and decode behind
    // the products).
    auto compute_static = [&](int nb, auto last) {
        constexpr bool LAST = decltype(last)::value;
        auto mf = [&](int i, const v8i& b, v16f& c) {
            c = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af[i], b, c, 0, 0, 0, 0, 0, 0);
        };
        mf(0, bf, acc[0][0]);
        mf(1, bf, acc[1][0]);
        bf1 = decode_w(ring0.c1);
        mf(0, bf1, acc[0][1]);
        if (!LAST)
            load_af(0, nb);
        mf(1, bf1, acc[1][1]);
        if (!LAST)
            load_af(1, nb);
        ring0 = ring1;
        ring1 = ring2;
        bfetch(ring2);
        bf = decode_w(ring0.c0);
    };
    // Per-group order, tiles t = (0,0) (1,0) (0,1) (1,1): at step t the fp8
    // product of tile t+1 is issued first, then the 16 FMAs of tile t (whose
    // product and scale tile were issued one step earlier and are done), then
    // the scale tile of tile t+1, then the operand work (LDS reads, weight
    // decode).  No FMA waits on an MFMA issued just before it, and each MFMA
    // goes out once the matrix unit has drained the previous one (an MFMA
    // issued while the unit is busy stalls its wave, and with it the FMAs
    // behind it).  The scale tile needs one buffer: it is overwritten only
    // after its FMAs.  Step 3 issues the next group's tile-0 product and scale
    // tile (not for a segment's last group), so the pipeline runs across the
    // barrier.  On entry pc and sc hold (in flight) this group's tile-0
    // product and scale tile, af[], sa_op[] and sw_op[] this group's
    // operands, bf its column-0 weight operand and wraw its column-1 weight
    // words.  The next group's operands (LDS stage nb) are read after their
    // last use here: column-0 words and s_w at step 0, rows 0 at step 1, rows
    // 1 at step 2 (with the decode of the column-0 words), column-1 words and
    // s_w at step 3.
    auto compute = [&](int cb, int nb, auto last) {
        constexpr bool LAST = decltype(last)::value;
        if constexpr (STATIC) {
            (void)cb;
            compute_static(nb, last);
            return;
        }
        (void)cb;
        v16f pn;
        // step 0: tile (0,0)
        pn = mfma_p(1, 0);                    // tile (1,0): rows 1 x column 0
        __builtin_amdgcn_sched_barrier(0);
        fma_tile(0, 0, pc, sc);
        __builtin_amdgcn_sched_barrier(0);
        sc = scale_tile(1, 0);
        __builtin_amdgcn_sched_barrier(0);
        bf = decode_w(wraw);                  // column 1: column 0's products are issued
        if (!LAST) {
            wraw = raw_w(0, nb);
            load_sw(0, nb);
        }
        __builtin_amdgcn_sched_barrier(0);
        pc = pn;
        // step 1: tile (1,0)
        pn = mfma_p(0, 1);                    // tile (0,1)
        __builtin_amdgcn_sched_barrier(0);
        fma_tile(1, 0, pc, sc);
        __builtin_amdgcn_sched_barrier(0);
        sc = scale_tile(0, 1);
        __builtin_amdgcn_sched_barrier(0);
        if (!LAST)
            load_a(0, nb);
        __builtin_amdgcn_sched_barrier(0);
        pc = pn;
        // step 2: tile (0,1)
        pn = mfma_p(1, 1);                    // tile (1,1)
        __builtin_amdgcn_sched_barrier(0);
        fma_tile(0, 1, pc, sc);
        __builtin_amdgcn_sched_barrier(0);
        sc = scale_tile(1, 1);
        __builtin_amdgcn_sched_barrier(0);
        if (!LAST) {
            load_a(1, nb);
            bf = decode_w(wraw);              // the next group's column 0
        }
        __builtin_amdgcn_sched_barrier(0);
        pc = pn;
        // step 3: tile (1,1)
        if (!LAST)
            pn = mfma_p(0, 0);                // the next group's tile (0,0)
        __builtin_amdgcn_sched_barrier(0);
        fma_tile(1, 1, pc, sc);
        __builtin_amdgcn_sched_barrier(0);
        if (!LAST) {
            sc = scale_tile(0, 0);
            wraw = raw_w(1, nb);
            load_sw(1, nb);
            pc = pn;
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    auto math_barrier = [] { asm volatile("s_barrier" ::: "memory"); };
    using NotLast = std::integral_constant<bool, false>;
    auto run_groups = [&](int n) {
        int g = 0;
        for (; g + kLinStages <= n; g += kLinStages) {
#pragma unroll
            for (int u = 0; u < kLinStages; ++u) {
                compute(u, (u + 1) % kLinStages, NotLast());
                math_barrier();
            }
        }
#pragma unroll
        for (int u = 0; u < kLinStages - 1; ++u) {
            if (g + u < n) {
                compute(u, (u + 1) % kLinStages, NotLast());
                math_barrier();
            }
        }
    };

    GemmCursor cur;
    // this lane's bias values of the current tile (bf16 bits), loaded when the
    // segment starts so the output code does not wait for them; STATIC: also
    // the channel scales s_w[n] (fp16 bits, from the scale slot of group 0 of
    // the wave's panel, where the per-channel pack keeps them)
    uint16_t bias_bits[TN], cscale_bits[TN];
    auto load_bias = [&] {
        const Rsrc rb = make_rsrc(bias, bias ? (uint32_t)(N * 2) : 0u);
#pragma unroll
        for (int j = 0; j < TN; ++j)
            bias_bits[j] = __builtin_amdgcn_raw_buffer_load_b16(
                rb, (int)(((int64_t)cur.tn * LBN + wn * WN + j * 32 + l32) * 2), 0, 0);
        if constexpr (STATIC) {
            const int64_t panel = (int64_t)cur.tn * kLinPanels + wn;
            const Rsrc rs = make_rsrc(w_packed + panel * G * kChunkBytes + kChunkCodeBytes,
                                      panel < panels ? (uint32_t)(kPanel * 2) : 0u);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                cscale_bits[j] = __builtin_amdgcn_raw_buffer_load_b16(rs, (j * 32 + l32) * 2, 0, 0);
        }
    };

    // ---- output: acc is in units of the weight operands (2^-9), so the
    // value before the activation is fmaf(acc, 2^9, bias), rounded once like
    // the unscaled sum.  Lane l holds column l % 32 of each 32 x 32 tile, rows
    // 8 (r/4) + 4 khalf + r%4 of register r; one lane-half swap pairs the two
    // column tiles so every bf16 store covers a full 128-byte row segment
    // (the template's output code, for this tile shape: one buffer range per
    // wave, the whole offset in the lane operand, rows past M outside the
    // range, columns past N at offset 2^31).
    auto store_tile = [&] {
        const int64_t row_base = (int64_t)cur.tm * LBM + wm * WM;
        const int64_t col_base = (int64_t)cur.tn * LBN + wn * WN;
        float b[TN], cs[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            b[j] = __uint_as_float((uint32_t)bias_bits[j] << 16);
            // STATIC: act_scale * s_w[n] times the 2^9 of the weight unit
            cs[j] = STATIC ? act_scale * (float)__builtin_bit_cast(_Float16, cscale_bits[j]) *
                                 kWeightUnitInv
                           : kWeightUnitInv;
        }
        lds_u8* const tw = (lds_u8*)(Ts + (uwave & (kLinMathWaves - 1)) * kTransposeBytes);
        if constexpr (QOUT) {
            quantize_tile_out<GELU>(acc, cs, b, tw, lane, row_base, col_base, M, N, qout);
            return;
        }
        const int64_t rows_in = max((int64_t)0, min(M - row_base, (int64_t)WM));
        const uint32_t row_bytes = (uint32_t)ldy * 2u;
        const Rsrc out_r = make_rsrc(y + row_base * ldy + col_base, (uint32_t)rows_in * row_bytes);
        // The tile through LDS, 16 bytes per lane and store: 8 stores of 8
        // rows each (a short store per element and row costs the vector
        // memory path as much as a full one).  Needs the wave's 64 columns
        // inside N and 16-byte aligned rows (wave-uniform); otherwise the
        // element stores below.
        if (col_base + WN <= N && ((reinterpret_cast<uintptr_t>(y) | (uint64_t)row_bytes) & 15u) == 0) {
            stage_tile_bf16<GELU>(acc, cs, b, tw, lane);
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const uint32_t row = (uint32_t)(8 * q) + ((uint32_t)lane >> 3), c = (uint32_t)lane & 7u;
                const v4u v = *(lds_v4u*)(tw + tile_chunk_offset(row, c));
                __builtin_amdgcn_raw_buffer_store_b128(v, out_r, (int)(row * row_bytes + c * 16u), 0, 0);
            }
            return;
        }
        const uint32_t voff = col_base + lane < N ? (uint32_t)lane * 2u : 0x80000000u;
        typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
        typedef float f2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float v0 = fmaf(acc[i][0][r], cs[0], b[0]);
                float v1 = fmaf(acc[i][1][r], cs[1], b[1]);
                if constexpr (GELU) {
                    v0 = gelu_tanh(v0);
                    v1 = gelu_tanh(v1);
                }
                const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v0),
                                                                 __float_as_uint(v1), false, false);
                const f2 pair = {__uint_as_float(sw[0]), __uint_as_float(sw[1])};
                const uint32_t pk = __builtin_bit_cast(uint32_t, __builtin_convertvector(pair, bf2));
                const uint32_t row0 = (uint32_t)(i * 32 + 8 * (r >> 2) + (r & 3));
                __builtin_amdgcn_raw_buffer_store_b16((uint16_t)pk, out_r,
                                                      (int)(voff + row0 * row_bytes), 0, 0);
                __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(pk >> 16), out_r,
                                                      (int)(voff + (row0 + 4) * row_bytes), 0, 0);
            }
        }
    };

    // Partial sums of a shared tile: the template's finisher (each math wave
    // its own 64 x 64 region, slot stores and loads with the sc1 policy, a
    // device-scope counter, contributors added in workgroup order; nobody
    // waits for another wave).
    constexpr int kRegionFloats = WM * WN;
    constexpr int kCoherent = 16;
    auto slot_rsrc = [&](int slot) {
        return make_rsrc(slots + ((int64_t)slot * kLinMathWaves + uwave) * kRegionFloats,
                         kRegionFloats * (uint32_t)sizeof(float));
    };
    typedef float v4f __attribute__((ext_vector_type(4)));
    auto finish_partial = [&]() -> bool {
        if constexpr (SPLIT) {
            const uint32_t lane_off = (uint32_t)lane * 16u;
            const Rsrc mine = slot_rsrc(cur.sg.slot);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const v4f v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                       acc[i][j][4 * q + 3]};
                        __builtin_amdgcn_raw_buffer_store_b128(
                            v, mine, (int)(lane_off + ((i * TN + j) * 4 + q) * 1024), 0, kCoherent);
                    }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            uint32_t* ctr = counters + (int64_t)cur.sg.sk_tile * kLinMathWaves + uwave;
            uint32_t arrived = 0;
            if (lane == 0)
                arrived = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            arrived = __builtin_amdgcn_readfirstlane(arrived);
            const GemmSchedule sch_ = fresh_schedule();
            int32_t b_first, b_last;
            sk_contributors(sch_, cur.sg.sk_tile, b_first, b_last);
            if (arrived != (uint32_t)(b_last - b_first))
                return false;
            asm volatile("" ::: "memory");
            // contributors in workgroup order (with two, this one's own share
            // stays in acc; with more, every share is read back from its
            // slot), a 32 x 32 tile (four 16-byte loads per lane) per
            // contributor in flight, so the finisher needs few registers
            const int32_t other = b_first == blk ? b_last : b_first;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int toff = (int)(lane_off + (i * TN + j) * 4 * 1024);
                    auto load_tile = [&](int32_t bb, v4f (&v)[4]) {
                        const Rsrc part = slot_rsrc(sk_slot(sch_, bb, cur.sg.sk_tile));
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            v[q] = __builtin_amdgcn_raw_buffer_load_b128(part, toff + q * 1024, 0, kCoherent);
                    };
                    if (b_last - b_first == 1) {
                        v4f v[4];
                        load_tile(other, v);
#pragma unroll
                        for (int q = 0; q < 4; ++q)
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                acc[i][j][4 * q + e] += v[q][e];
                    } else {
                        for (int32_t bb = b_first; bb <= b_last; ++bb) {
                            v4f v[4];
                            load_tile(bb, v);
#pragma unroll
                            for (int q = 0; q < 4; ++q)
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    acc[i][j][4 * q + e] =
                                        bb == b_first ? v[q][e] : acc[i][j][4 * q + e] + v[q][e];
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            if (lane == 0)
                __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return true;
        }
        return false;
    };

    auto reset_tile = [&] {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc[i][j][r] = 0.0f;
    };

    if (!cursor_begin(fresh_schedule(), blk, cur))
        return;
#pragma unroll
    for (int i = 0; i < TM; ++i)
        sa_op[i] = v2i{0, 0};
#pragma unroll
    for (int j = 0; j < TN; ++j)
        sw_op[j] = v2i{0, 0};
#pragma unroll
    for (int i = 0; i < TM; ++i)
        za_op[i] = v2i{0, 0};
#pragma unroll
    for (int j = 0; j < TN; ++j)
        ws_op[j] = v2i{0, 0};
    if constexpr (STATIC) {
        // the weight fetch cursor starts on the same segment; the ring then
        // runs continuously, three groups ahead of the multiplication
        set_fragment_indices();
        bcur = cur;
        bg = cur.sg.g0;
        bpanel = (int64_t)cur.tn * kLinPanels + wn;
        bfetch(ring0);
        bfetch(ring1);
        bfetch(ring2);
        bf = decode_w(ring0.c0);
    }
    lds_sync();
    for (;;) {
        const int L = cur.sg.g1 - cur.sg.g0;
        set_fragment_indices();
        load_bias();
        reset_tile();
        if constexpr (STATIC) {
            load_af(0, 0);
            load_af(1, 0);
        } else {
            load_a(0, 0);
            load_a(1, 0);
            bf = decode_w(raw_w(0, 0));
            wraw = raw_w(1, 0);
            load_sw(0, 0);
            load_sw(1, 0);
            pc = mfma_p(0, 0);
            sc = scale_tile(0, 0);
        }
        run_groups(L - 1);
        compute((L - 1) % kLinStages, 0, std::integral_constant<bool, true>());
        math_barrier();
        for (int p = L; p < padded_steps(L); ++p)
            math_barrier();
        set_fragment_indices();
        if (!SPLIT || cur.sg.sk_tile < 0 || finish_partial())
            store_tile();
        if (!cursor_next(fresh_schedule(), blk, cur))
            break;
    }
}

template <bool STATIC, bool QOUT, bool ASYM = false>
hipError_t launch_linear_mode(const GemmLaunch& a, hipStream_t stream)
{
    const dim3 grid((unsigned)a.sch.blocks), block(kLinThreads);
    auto go = [&](auto gs, auto gelu, auto split) {
        w4a4_linear_kernel<decltype(gs)::value, decltype(gelu)::value, decltype(split)::value, STATIC,
                           QOUT, ASYM><<<grid, block, 0, stream>>>(
            a.codes, a.flags, a.scales, a.w_packed, a.bias, a.y, a.M, a.N, a.K, a.ldy, a.sch,
            a.counters, a.slots, a.act_scale, a.qout, a.zeros, a.wsums);
    };
    auto with_split = [&](auto gs, auto gelu) {
        if (a.sch.sk_tiles > 0)
            go(gs, gelu, bool_c<true>());
        else
            go(gs, gelu, bool_c<false>());
    };
    auto with_gelu = [&](auto gs) {
        if (a.epilogue == 1)
            with_split(gs, bool_c<true>());
        else
            with_split(gs, bool_c<false>());
    };
    switch (a.lzs_group) {
    case 8:
        with_gelu(std::integral_constant<int, 8>());
        break;
    case 16:
        with_gelu(std::integral_constant<int, 16>());
        break;
    case 32:
        with_gelu(std::integral_constant<int, 32>());
        break;
    default:
        with_gelu(std::integral_constant<int, 64>());
        break;
    }
    return hipGetLastError();
}

}  // namespace
}  // namespace quartz
