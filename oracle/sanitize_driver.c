/*
 * Drives every entry point of the oracle (quartz_oracle.c) on small, ragged
 * shapes with exactly sized heap buffers, for a build with AddressSanitizer
 * and UndefinedBehaviorSanitizer: an index past any input or output, or
 * undefined arithmetic, in any of them ends the run with a report.
 * TEST INFRASTRUCTURE ONLY (built and run by the CPU test suite).
 *
 * Exit status 0 when every call returned its expected status.
 */
#include "quartz_oracle.c"

#include <stdio.h>

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;

static uint32_t next_u32(void)
{
    /* xorshift64*: a small deterministic generator for the inputs */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (uint32_t)((rng_state * 2685821657736338717ull) >> 32);
}

/* a finite bf16 pattern: random sign and mantissa, exponent in a band around 1 */
static uint16_t random_bf16(void)
{
    const uint32_t r = next_u32();
    const uint32_t e = 120u + (r >> 8) % 12u;
    return (uint16_t)(((r & 1u) << 15) | (e << 7) | ((r >> 1) & 0x7Fu));
}

static void* xmalloc(size_t n)
{
    void* p = malloc(n ? n : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

static int failures = 0;

static void expect(int got, int want, const char* what, int64_t M, int64_t N, int64_t K, int gs)
{
    if (got != want) {
        fprintf(stderr, "%s: status %d, want %d (M=%lld N=%lld K=%lld gs=%d)\n", what, got, want,
                (long long)M, (long long)N, (long long)K, gs);
        ++failures;
    }
}

static void run_case(int64_t M, int64_t N, int64_t K, int64_t pad, int gs)
{
    const int64_t ldx = K + pad, G = K / 64, S = K / gs;
    uint16_t* x = xmalloc((size_t)(M * ldx) * 2);
    uint16_t* w = xmalloc((size_t)(N * K) * 2);
    uint16_t* bias = xmalloc((size_t)N * 2);
    for (int64_t i = 0; i < M * ldx; ++i)
        x[i] = random_bf16();
    for (int64_t i = 0; i < N * K; ++i)
        w[i] = random_bf16();
    for (int64_t i = 0; i < N; ++i)
        bias[i] = random_bf16();
    int8_t* q8 = xmalloc((size_t)(M * K));
    int8_t* c = xmalloc((size_t)(M * K));
    uint8_t* flags = xmalloc((size_t)(M * S));
    uint16_t* scales = xmalloc((size_t)(M * G) * 2);
    int8_t* zeros = xmalloc((size_t)(M * G));
    uint8_t* codes = xmalloc((size_t)(G * M * 32));
    int8_t* c2 = xmalloc((size_t)(M * K));
    int8_t* wq = xmalloc((size_t)(N * K));
    uint16_t* sw = xmalloc((size_t)(N * G) * 2);
    uint16_t* swc = xmalloc((size_t)N * 2);
    int16_t* sums = xmalloc((size_t)(G * N) * 2);
    int32_t* acc = xmalloc((size_t)(M * N) * 4);
    double* y = xmalloc((size_t)(M * N) * 8);
    double* absum = xmalloc((size_t)(M * N) * 8);
    uint16_t* yb = xmalloc((size_t)(M * N) * 2);
    const int64_t count = M < N ? M : N;
    int64_t* rows = xmalloc((size_t)count * 8);
    int64_t* cols = xmalloc((size_t)count * 8);
    double* ys = xmalloc((size_t)count * 8);
    double* as = xmalloc((size_t)count * 8);
    for (int64_t i = 0; i < count; ++i) {
        rows[i] = M - 1 - i;
        cols[i] = i;
    }

    expect(qo_quantize_act(x, M, K, ldx, 64, gs, q8, c, flags, scales, zeros), QO_OK,
           "quantize_act", M, N, K, gs);
    expect(qo_quantize_act(x, M, K, ldx, 64, gs, NULL, c, flags, scales, NULL), QO_OK,
           "quantize_act (no q8, no zeros)", M, N, K, gs);
    qo_pack_codes(c, M, K, codes);
    qo_unpack_codes(codes, M, K, c2);
    if (memcmp(c, c2, (size_t)(M * K)) != 0) {
        fprintf(stderr, "pack/unpack round trip differs (M=%lld K=%lld)\n", (long long)M,
                (long long)K);
        ++failures;
    }
    expect(qo_quantize_weight(w, N, K, 64, wq, sw), QO_OK, "quantize_weight", M, N, K, gs);
    expect(qo_gemm_i32(c, flags, wq, M, N, K, gs, acc), QO_OK, "gemm_i32", M, N, K, gs);
    for (int epi = 0; epi < 2; ++epi) {
        expect(qo_linear_f64(c, flags, scales, wq, sw, bias, M, N, K, 64, gs, epi, y, absum), QO_OK,
               "linear_f64", M, N, K, gs);
        expect(qo_linear_f64(c, flags, scales, wq, sw, NULL, M, N, K, 64, gs, epi, y, NULL), QO_OK,
               "linear_f64 (no bias)", M, N, K, gs);
        expect(qo_linear_f64_sampled(c, flags, scales, wq, sw, bias, K, 64, gs, epi, rows, cols,
                                     count, ys, as),
               QO_OK, "linear_f64_sampled", M, N, K, gs);
    }
    qo_round_bf16(y, M * N, yb);

    expect(qo_quantize_act_asym(x, M, K, ldx, gs, q8, c, flags, scales, zeros), QO_OK,
           "quantize_act_asym", M, N, K, gs);
    expect(qo_weight_group_sums(wq, N, K, sums), QO_OK, "weight_group_sums", M, N, K, gs);
    expect(qo_linear_asym_f64(c, flags, scales, zeros, wq, sw, bias, M, N, K, gs, 1, y, absum),
           QO_OK, "linear_asym_f64", M, N, K, gs);

    expect(qo_quantize_act_static(x, M, K, ldx, 0.01f, gs, q8, c, flags), QO_OK,
           "quantize_act_static", M, N, K, gs);
    expect(qo_quantize_act_static(x, M, K, ldx, 0.01f, gs, NULL, c, flags), QO_OK,
           "quantize_act_static (no q8)", M, N, K, gs);
    expect(qo_quantize_weight_per_channel(w, N, K, wq, swc), QO_OK, "quantize_weight_per_channel",
           M, N, K, gs);
    expect(qo_linear_static_f64(c, flags, 0.01f, wq, swc, bias, M, N, K, gs, 1, y, absum), QO_OK,
           "linear_static_f64", M, N, K, gs);

    /* invalid arguments are rejected before any access */
    expect(qo_quantize_act(x, M, K + 1, ldx + 1, 64, gs, q8, c, flags, scales, zeros), QO_EINVAL,
           "quantize_act K % 64", M, N, K, gs);
    expect(qo_quantize_act(x, M, K, K - 1, 64, gs, q8, c, flags, scales, zeros), QO_EINVAL,
           "quantize_act ldx < K", M, N, K, gs);
    expect(qo_quantize_act_static(x, M, K, ldx, 0.0f, gs, q8, c, flags), QO_EINVAL,
           "quantize_act_static s = 0", M, N, K, gs);

    free(x); free(w); free(bias); free(q8); free(c); free(flags); free(scales); free(zeros);
    free(codes); free(c2); free(wq); free(sw); free(swc); free(sums); free(acc); free(y);
    free(absum); free(yb); free(rows); free(cols); free(ys); free(as);
}

int main(void)
{
    /* scalar helpers over their whole domains */
    for (uint32_t h = 0; h < 65536u; ++h) {
        volatile float f = qo_f16_to_f32((uint16_t)h);
        if (isfinite(f))
            (void)qo_f32_to_f16_rne_sat(f);
        (void)qo_bf16_to_f32((uint16_t)h);
    }
    for (uint32_t m = 0; m < 256u; ++m) {
        (void)qo_clz32(m);
        (void)qo_lzs_flag(m & 127u);
    }
    for (int v = -127; v <= 127; ++v) {
        int8_t q = (int8_t)v, c;
        (void)qo_lzs_subgroup(&q, 1, &c);
    }
    (void)qo_f64_to_bf16_rne(1e300);
    (void)qo_f64_to_bf16_rne(-3.0e-41);
    (void)qo_gelu_tanh(-30.0);
    (void)qo_rne(-2.5);
    (void)qo_num_threads();

    static const int64_t Ms[] = {1, 5, 13};
    static const int64_t Ns[] = {1, 7, 70};
    static const int64_t Ks[] = {64, 192};
    static const int gss[] = {1, 8, 16, 32, 64};
    for (size_t a = 0; a < sizeof(Ms) / sizeof(Ms[0]); ++a)
        for (size_t b = 0; b < sizeof(Ns) / sizeof(Ns[0]); ++b)
            for (size_t k = 0; k < sizeof(Ks) / sizeof(Ks[0]); ++k)
                for (size_t g = 0; g < sizeof(gss) / sizeof(gss[0]); ++g)
                    run_case(Ms[a], Ns[b], Ks[k], (int64_t)((a + g) % 2) * 8, gss[g]);
    if (failures) {
        fprintf(stderr, "%d failed calls\n", failures);
        return 1;
    }
    printf("oracle sanitizer driver: all calls clean\n");
    return 0;
}
