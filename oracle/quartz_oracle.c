/*
 * QuaRTZ CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct C reference of the W4A4 linear hot path of
 * "Post-Training Quantization via Residual Truncation and Zero Suppression for
 * Diffusion Models" (QuaRTZ, arXiv 2509.26436).  Only tests, the smoke check
 * and the CPU-baseline leg of the benchmark may call it; the product library
 * never links, loads or calls anything here, and nothing here is shared with
 * the HIP path (no common headers, tables or helpers).
 *
 * Every floating-point step is written out from its definition:
 *   - bf16 -> fp32 is a 16-bit left shift of the bit pattern (exact);
 *   - fp32 -> fp16 is IEEE-754 round-to-nearest-even, computed from the value
 *     in double precision, with overflow saturating to +-65504;
 *   - rounding to an integer is round-half-to-even, written out with floor();
 *   - clz is a bit-by-bit count.
 * Build: gcc -O2 -ffp-contract=off (no fast-math), so float arithmetic is
 * IEEE binary32 with round-to-nearest-even.
 *
 * Readings of the paper that the oracle adopts (each is listed with its reason
 * in the design notes of the repository):
 *   R1  Stage 1 (Eq. 1) is taken as the symmetric midtread quantizer that the
 *       error analysis of Appendix A assumes: s = max|x| / 127 over the
 *       64-element group, zero point z = 0, codes clamped to [-127, 127].
 *   R2  The 16-bit scale of Appendix C is IEEE fp16 (RNE, saturating); the
 *       codes are computed with the stored scale: r = 1/s (fp32, IEEE),
 *       q = clamp(rne(fp32(x * r)), -127, 127).
 *   R3  The Eq. 2 flag is max(29 - clz32(OR of magnitudes), 0) over a
 *       subgroup of G_s consecutive elements along K; subgroups nest inside
 *       the 64-element groups.
 *   R4  Residual truncation (Section 3, Appendix A) right-shifts the 7-bit
 *       magnitude by FLAG (truncation toward zero) and keeps the sign:
 *       c = sgn(q) * (|q| >> FLAG), c in [-7, 7].  The decoded integer is
 *       d = c * 2^FLAG.
 *   R5  Weights (Appendix C): symmetric RTN int4 per 64-group along K,
 *       sw = fp16(max|w| / 7), wq = clamp(rne(fp32(w * (1/sw))), -7, 7).
 *       No LZS on weights; GPTQ is not part of the hot path.
 *   R6  The integer MMA with a per-subgroup power-of-two (Section 4.4) equals
 *       sum_k d[m,k] * wq[n,k] over each 64-group (distributivity); the
 *       per-group float dequantization multiplies by s_a[m,g] * s_w[n,g].
 *   R8  The LDM setting (the experimental-details appendix): static
 *       per-tensor activation quantization takes one fp32 scale s fixed
 *       ahead of time (calibration is outside the hot path), r = fp32(1/s),
 *       q = clamp(rne(fp32(x * r)), -127, 127), then Stage 2 as in R3/R4;
 *       per-channel weight quantization takes s_w[n] = fp16(max over all of
 *       K of |w[n,k]| / 7) and wq = clamp(rne(fp32(w * (1/s_w[n]))), -7, 7).
 *       The layer output is y = s * s_w[n] * I[m,n] + bias with I the exact
 *       integer sum over all of K of d * wq.
 *   R9  Asymmetric mode (Eq. 1's zero point, repaired so that 255 signed
 *       levels cover the group's range including 0): lo = min(x_min, 0),
 *       hi = max(x_max, 0), s = fp16(fp32(hi - lo) / 254) (RNE, saturating),
 *       r = 1/s (fp32), z = -127 - rne(fp32(lo * r)) in [-127, 127],
 *       q = clamp(rne(fp32(x * r)) + z, -127, 127); Stage 2 on q as in R3/R4;
 *       the dequantized value is s * (d - z).  The layer output is
 *       y = sum_g s_a s_w (P_g - z[m,g] * W_g[n]) + bias, with
 *       W_g[n] = sum over the group of wq[n,k] (the weight group sums).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define QO_OK 0
#define QO_EINVAL 1

/* ---------------------------------------------------------------- scalars */

/* bf16 bit pattern -> float: the bf16 bits are the top half of the binary32. */
float qo_bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Round half to even, written out.  Exact for |v| < 2^52. */
double qo_rne(double v)
{
    double f = floor(v);
    double d = v - f;            /* exact: f and v share the binade or f = 0 */
    if (d > 0.5)
        return f + 1.0;
    if (d < 0.5)
        return f;
    /* tie: pick the even neighbour */
    return (fmod(f, 2.0) == 0.0) ? f : f + 1.0;
}

/* IEEE binary16 value of a bit pattern. */
float qo_f16_to_f32(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int m = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24);                  /* subnormal: m * 2^-24 */
    else if (e == 31)
        v = (m == 0) ? INFINITY : NAN;
    else
        v = ldexp(1024.0 + (double)m, e - 25);      /* (1 + m/1024) * 2^(e-15) */
    return (float)(sign ? -v : v);
}

/*
 * float -> IEEE binary16, round to nearest even; a result that would round to
 * infinity saturates to the largest finite value 65504 (sign kept).  NaN maps
 * to the canonical quiet NaN 0x7e00.
 */
uint16_t qo_f32_to_f16_rne_sat(float f)
{
    double a = fabs((double)f);
    uint16_t sign = signbit(f) ? 0x8000 : 0;
    if (isnan(f))
        return 0x7e00;
    if (a == 0.0)
        return sign;
    /* exponent of the leading bit: a = fr * 2^ex, fr in [0.5, 1) */
    int ex;
    frexp(a, &ex);
    int e = ex - 1;                       /* a in [2^e, 2^(e+1)) */
    if (e < -14)
        e = -14;                          /* subnormal range: quantum 2^-24 */
    double quantum = ldexp(1.0, e - 10);  /* 10 fraction bits */
    double n = qo_rne(a / quantum);       /* a / quantum is exact (power of 2) */
    double v = n * quantum;
    if (v > 65504.0)                      /* rounds to >= 65536: overflow */
        v = 65504.0;
    /* encode v exactly */
    if (v < ldexp(1.0, -14))
        return (uint16_t)(sign | (uint16_t)(v / ldexp(1.0, -24)));
    frexp(v, &ex);
    e = ex - 1;
    uint16_t mant = (uint16_t)(v / ldexp(1.0, e - 10) - 1024.0);
    return (uint16_t)(sign | (uint16_t)((e + 15) << 10) | mant);
}

/* Round a double to bf16 (RNE) and return the bit pattern; used to state the
 * expected bf16 output of the linear layer.  Overflow goes to infinity. */
uint16_t qo_f64_to_bf16_rne(double x)
{
    double a = fabs(x);
    uint16_t sign = signbit(x) ? 0x8000 : 0;
    if (isnan(x))
        return 0x7fc0;
    if (a == 0.0)
        return sign;
    int ex;
    frexp(a, &ex);
    int e = ex - 1;
    if (e < -126)
        e = -126;                         /* subnormal quantum 2^-133 */
    double quantum = ldexp(1.0, e - 7);   /* 7 fraction bits */
    double n = qo_rne(a / quantum);
    double v = n * quantum;
    if (v >= ldexp(1.0, 128))
        return (uint16_t)(sign | 0x7f80);
    if (v < ldexp(1.0, -126))
        return (uint16_t)(sign | (uint16_t)(v / ldexp(1.0, -133)));
    frexp(v, &ex);
    e = ex - 1;
    uint16_t mant = (uint16_t)(v / ldexp(1.0, e - 7) - 128.0);
    return (uint16_t)(sign | (uint16_t)((e + 127) << 7) | mant);
}

/* Count leading zeros of a 32-bit word, bit by bit; clz(0) = 32. */
int qo_clz32(uint32_t v)
{
    int n = 0;
    for (int bit = 31; bit >= 0; --bit) {
        if (v & (1u << bit))
            break;
        ++n;
    }
    return n;
}

/* Eq. 2: FLAG = max(29 - clz(m), 0) for the OR-aggregated magnitude m. */
int qo_lzs_flag(uint32_t m_or)
{
    int f = 29 - qo_clz32(m_or);
    return f > 0 ? f : 0;
}

/* GELU with the tanh approximation, in double. */
double qo_gelu_tanh(double x)
{
    const double k = sqrt(2.0 / M_PI);
    return 0.5 * x * (1.0 + tanh(k * (x + 0.044715 * x * x * x)));
}

/* ---------------------------------------------------- activation quantizer */

/*
 * Stage 1 of one 64-element group (Eq. 1 under reading R1/R2): returns the
 * fp16 scale bits and writes the int8 codes q[0..group-1].
 */
static uint16_t stage1_group(const uint16_t* x, int group, int8_t* q)
{
    float alpha = 0.0f;
    for (int k = 0; k < group; ++k) {
        float a = fabsf(qo_bf16_to_f32(x[k]));
        if (a > alpha)
            alpha = a;
    }
    float s_f = alpha / 127.0f;                  /* IEEE binary32 division */
    uint16_t s16 = qo_f32_to_f16_rne_sat(s_f);
    float s = qo_f16_to_f32(s16);
    float r = (s == 0.0f) ? 0.0f : 1.0f / s;     /* IEEE binary32 division */
    for (int k = 0; k < group; ++k) {
        float p = qo_bf16_to_f32(x[k]) * r;      /* binary32 product */
        double v = qo_rne((double)p);
        if (v > 127.0)
            v = 127.0;
        if (v < -127.0)
            v = -127.0;
        q[k] = (int8_t)v;
    }
    return s16;
}

/*
 * Stage 2 (Eq. 2 and the right shift that follows it) of one subgroup of n
 * int8 codes: returns FLAG, writes c = sgn(q) * (|q| >> FLAG).
 * The sign-magnitude split of Section 3: sgn = (q < 0), mag = |q| (7 bits;
 * -128 never comes out of Stage 1 and is saturated to magnitude 127 here so
 * that FLAG stays within {0..4}).
 */
int qo_lzs_subgroup(const int8_t* q, int n, int8_t* c)
{
    uint32_t m_or = 0;
    for (int i = 0; i < n; ++i) {
        int mag = q[i] < 0 ? -(int)q[i] : (int)q[i];
        if (mag > 127)
            mag = 127;
        m_or |= (uint32_t)mag;
    }
    int flag = qo_lzs_flag(m_or);
    for (int i = 0; i < n; ++i) {
        int neg = q[i] < 0;
        int mag = neg ? -(int)q[i] : (int)q[i];
        if (mag > 127)
            mag = 127;
        int t = mag >> flag;
        c[i] = (int8_t)(neg ? -t : t);
    }
    return flag;
}

/*
 * Full activation quantizer over x [M][ldx] (bf16 bits).  Outputs, all
 * row-major and caller-allocated:
 *   q8     int8 [M][K]            Stage-1 codes (may be NULL)
 *   c      int8 [M][K]            signed 4-bit values in [-7, 7]
 *   flags  u8   [M][K/lzs_group]  FLAG in 0..4
 *   scales u16  [M][K/group]      fp16 bits
 *   zeros  i8   [M][K/group]      zero points (always 0, reading R1; may be NULL)
 * group must be 64; lzs_group must divide it (1..64).
 */
int qo_quantize_act(const uint16_t* x, int64_t M, int64_t K, int64_t ldx,
                    int group, int lzs_group, int8_t* q8, int8_t* c,
                    uint8_t* flags, uint16_t* scales, int8_t* zeros)
{
    if (group != 64 || lzs_group < 1 || group % lzs_group != 0 || K % group != 0 || ldx < K)
        return QO_EINVAL;
    const int64_t G = K / group, S = K / lzs_group;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        int8_t q[64];
        for (int64_t g = 0; g < G; ++g) {
            const uint16_t* xg = x + m * ldx + g * group;
            scales[m * G + g] = stage1_group(xg, group, q);
            if (zeros)
                zeros[m * G + g] = 0;
            if (q8)
                memcpy(q8 + m * K + g * group, q, (size_t)group);
            for (int j = 0; j < group / lzs_group; ++j) {
                int64_t sub = g * (group / lzs_group) + j;
                flags[m * S + sub] = (uint8_t)qo_lzs_subgroup(
                    q + j * lzs_group, lzs_group, c + m * K + g * group + j * lzs_group);
            }
        }
    }
    return QO_OK;
}

/*
 * Storage layout of the 4-bit codes (the library's documented format):
 * each code is a sign-magnitude nibble, bit 3 = sign, bits 0..2 = |c|, and
 * c = 0 is always stored as 0.  The 32 bytes of (64-group g, row m) sit at
 * byte (g * M + m) * 32 (K-group-major).  Within them, elements 8j..8j+7 of
 * the group form the little-endian 32-bit word j; element 8j+i sits in nibble
 * (i/2) + 4*(i%2), i.e. even elements fill the low half-word and odd elements
 * the high one.
 */
void qo_pack_codes(const int8_t* c, int64_t M, int64_t K, uint8_t* codes)
{
    const int64_t G = K / 64;
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t g = 0; g < G; ++g) {
            uint8_t* out = codes + (g * M + m) * 32;
            for (int j = 0; j < 8; ++j) {
                uint32_t word = 0;
                for (int i = 0; i < 8; ++i) {
                    int v = c[m * K + g * 64 + 8 * j + i];
                    uint32_t nib = (uint32_t)(v < 0 ? 8 + (-v) : v);
                    int pos = (i / 2) + 4 * (i % 2);
                    word |= nib << (4 * pos);
                }
                out[4 * j + 0] = (uint8_t)(word & 0xff);
                out[4 * j + 1] = (uint8_t)((word >> 8) & 0xff);
                out[4 * j + 2] = (uint8_t)((word >> 16) & 0xff);
                out[4 * j + 3] = (uint8_t)((word >> 24) & 0xff);
            }
        }
    }
}

/* Inverse of qo_pack_codes (nibble 8 = "-0" decodes to 0). */
void qo_unpack_codes(const uint8_t* codes, int64_t M, int64_t K, int8_t* c)
{
    const int64_t G = K / 64;
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t g = 0; g < G; ++g) {
            const uint8_t* in = codes + (g * M + m) * 32;
            for (int j = 0; j < 8; ++j) {
                uint32_t word = (uint32_t)in[4 * j] | ((uint32_t)in[4 * j + 1] << 8) |
                                ((uint32_t)in[4 * j + 2] << 16) | ((uint32_t)in[4 * j + 3] << 24);
                for (int i = 0; i < 8; ++i) {
                    int pos = (i / 2) + 4 * (i % 2);
                    uint32_t nib = (word >> (4 * pos)) & 0xf;
                    int mag = (int)(nib & 7);
                    c[m * K + g * 64 + 8 * j + i] = (int8_t)((nib & 8) ? -mag : mag);
                }
            }
        }
    }
}

/* -------------------------------------------------------- weight quantizer */

/* Reading R5: symmetric round-to-nearest int4 in [-7, 7], fp16 group scales. */
int qo_quantize_weight(const uint16_t* w, int64_t N, int64_t K, int group,
                       int8_t* wq, uint16_t* sw)
{
    if (group != 64 || K % group != 0)
        return QO_EINVAL;
    const int64_t G = K / group;
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t g = 0; g < G; ++g) {
            const uint16_t* wg = w + n * K + g * group;
            float beta = 0.0f;
            for (int k = 0; k < group; ++k) {
                float a = fabsf(qo_bf16_to_f32(wg[k]));
                if (a > beta)
                    beta = a;
            }
            uint16_t s16 = qo_f32_to_f16_rne_sat(beta / 7.0f);
            float s = qo_f16_to_f32(s16);
            float r = (s == 0.0f) ? 0.0f : 1.0f / s;
            sw[n * G + g] = s16;
            for (int k = 0; k < group; ++k) {
                float p = qo_bf16_to_f32(wg[k]) * r;
                double v = qo_rne((double)p);
                if (v > 7.0)
                    v = 7.0;
                if (v < -7.0)
                    v = -7.0;
                wq[n * K + g * group + k] = (int8_t)v;
            }
        }
    }
    return QO_OK;
}

/* ------------------------------------------------------------------- GEMM */

/* Decoded activation integer d = c * 2^FLAG (reading R4). */
static int decoded(const int8_t* c, const uint8_t* flags, int64_t K, int lzs_group,
                   int64_t m, int64_t k)
{
    int f = flags[m * (K / lzs_group) + k / lzs_group];
    return c[m * K + k] * (1 << f);
}

/*
 * Exact integer accumulator I[m][n] = sum_k d[m,k] * wq[n,k] over all of K
 * (sum of the per-group integer MMA results of Section 4.4).
 */
int qo_gemm_i32(const int8_t* c, const uint8_t* flags, const int8_t* wq,
                int64_t M, int64_t N, int64_t K, int lzs_group, int32_t* out)
{
    if (lzs_group < 1 || K % lzs_group != 0)
        return QO_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t n = 0; n < N; ++n) {
            int64_t acc = 0;
            for (int64_t k = 0; k < K; ++k)
                acc += (int64_t)decoded(c, flags, K, lzs_group, m, k) * wq[n * K + k];
            out[m * N + n] = (int32_t)acc;
        }
    }
    return QO_OK;
}

/*
 * One output of the dequantized linear layer, in double:
 *   y = sum_g s_a[m,g] * s_w[n,g] * P_g[m,n] + bias[n]   (then GELU-tanh)
 * with P_g the exact integer sum over group g.  *absum receives
 * S = sum_g |s_a s_w P_g| + |bias| (the scale of the accumulation).
 */
static double linear_one(const int8_t* c, const uint8_t* flags, const uint16_t* scales,
                         const int8_t* wq, const uint16_t* sw, const uint16_t* bias,
                         int64_t K, int group, int lzs_group, int epilogue,
                         int64_t m, int64_t n, double* absum)
{
    const int64_t G = K / group;
    double y = 0.0, s = 0.0;
    for (int64_t g = 0; g < G; ++g) {
        int64_t p = 0;
        for (int64_t k = g * group; k < (g + 1) * group; ++k)
            p += (int64_t)decoded(c, flags, K, lzs_group, m, k) * wq[n * K + k];
        double t = (double)qo_f16_to_f32(scales[m * G + g]) *
                   (double)qo_f16_to_f32(sw[n * G + g]) * (double)p;
        y += t;
        s += fabs(t);
    }
    if (bias) {
        double b = (double)qo_bf16_to_f32(bias[n]);
        y += b;
        s += fabs(b);
    }
    if (epilogue == 1)
        y = qo_gelu_tanh(y);
    if (absum)
        *absum = s;
    return y;
}

int qo_linear_f64(const int8_t* c, const uint8_t* flags, const uint16_t* scales,
                  const int8_t* wq, const uint16_t* sw, const uint16_t* bias,
                  int64_t M, int64_t N, int64_t K, int group, int lzs_group,
                  int epilogue, double* y, double* absum)
{
    if (group != 64 || K % group != 0 || lzs_group < 1 || group % lzs_group != 0)
        return QO_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n)
            y[m * N + n] = linear_one(c, flags, scales, wq, sw, bias, K, group, lzs_group,
                                      epilogue, m, n, absum ? &absum[m * N + n] : NULL);
    return QO_OK;
}

/* Same, only for the listed (rows[i], cols[i]) outputs. */
int qo_linear_f64_sampled(const int8_t* c, const uint8_t* flags, const uint16_t* scales,
                          const int8_t* wq, const uint16_t* sw, const uint16_t* bias,
                          int64_t K, int group, int lzs_group, int epilogue,
                          const int64_t* rows, const int64_t* cols, int64_t count,
                          double* y, double* absum)
{
    if (group != 64 || K % group != 0 || lzs_group < 1 || group % lzs_group != 0)
        return QO_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        y[i] = linear_one(c, flags, scales, wq, sw, bias, K, group, lzs_group, epilogue,
                          rows[i], cols[i], absum ? &absum[i] : NULL);
    return QO_OK;
}

/* ------------------------------------------ asymmetric mode (reading R9) */

static void stage1_group_asym(const uint16_t* x, int group, int8_t* q, uint16_t* s16_out,
                              int8_t* z_out)
{
    float xmin = 0.0f, xmax = 0.0f;              /* the range always includes 0 */
    for (int k = 0; k < group; ++k) {
        float v = qo_bf16_to_f32(x[k]);
        if (v < xmin)
            xmin = v;
        if (v > xmax)
            xmax = v;
    }
    float span = xmax - xmin;                    /* binary32 subtraction */
    uint16_t s16 = qo_f32_to_f16_rne_sat(span / 254.0f);
    float s = qo_f16_to_f32(s16);
    float r = (s == 0.0f) ? 0.0f : 1.0f / s;
    double zl = qo_rne((double)(xmin * r));      /* in [-254, 0] */
    int z = -127 - (int)zl;
    if (z > 127)
        z = 127;
    if (z < -127)
        z = -127;
    for (int k = 0; k < group; ++k) {
        float p = qo_bf16_to_f32(x[k]) * r;
        double v = qo_rne((double)p) + (double)z;
        if (v > 127.0)
            v = 127.0;
        if (v < -127.0)
            v = -127.0;
        q[k] = (int8_t)v;
    }
    *s16_out = s16;
    *z_out = (int8_t)z;
}

/* Asymmetric activation quantizer: outputs as qo_quantize_act, zeros = z. */
int qo_quantize_act_asym(const uint16_t* x, int64_t M, int64_t K, int64_t ldx, int lzs_group,
                         int8_t* q8, int8_t* c, uint8_t* flags, uint16_t* scales, int8_t* zeros)
{
    if (lzs_group < 1 || 64 % lzs_group != 0 || K % 64 != 0 || ldx < K)
        return QO_EINVAL;
    const int64_t G = K / 64, S = K / lzs_group;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        int8_t q[64];
        for (int64_t g = 0; g < G; ++g) {
            stage1_group_asym(x + m * ldx + g * 64, 64, q, &scales[m * G + g], &zeros[m * G + g]);
            if (q8)
                memcpy(q8 + m * K + g * 64, q, 64);
            for (int j = 0; j < 64 / lzs_group; ++j) {
                int64_t sub = g * (64 / lzs_group) + j;
                flags[m * S + sub] = (uint8_t)qo_lzs_subgroup(
                    q + j * lzs_group, lzs_group, c + m * K + g * 64 + j * lzs_group);
            }
        }
    }
    return QO_OK;
}

/* Weight group sums W_g[n] = sum over group g of wq[n,k], int16 [N][K/64]. */
int qo_weight_group_sums(const int8_t* wq, int64_t N, int64_t K, int16_t* sums)
{
    if (K % 64 != 0)
        return QO_EINVAL;
    const int64_t G = K / 64;
    for (int64_t n = 0; n < N; ++n)
        for (int64_t g = 0; g < G; ++g) {
            int t = 0;
            for (int k = 0; k < 64; ++k)
                t += wq[n * K + g * 64 + k];
            sums[n * G + g] = (int16_t)t;
        }
    return QO_OK;
}

/*
 * One output of the asymmetric-mode layer, in double:
 *   y = sum_g s_a[m,g] s_w[n,g] (P_g[m,n] - z[m,g] W_g[n]) + bias[n]   (then GELU)
 * *absum receives S = sum_g |s_a s_w (P_g - z W_g)| + |bias|.
 */
static double linear_asym_one(const int8_t* c, const uint8_t* flags, const uint16_t* scales,
                              const int8_t* zeros, const int8_t* wq, const uint16_t* sw,
                              const uint16_t* bias, int64_t K, int lzs_group, int epilogue,
                              int64_t m, int64_t n, double* absum)
{
    const int64_t G = K / 64;
    double y = 0.0, a = 0.0;
    for (int64_t g = 0; g < G; ++g) {
        int64_t p = 0, wsum = 0;
        for (int64_t k = g * 64; k < (g + 1) * 64; ++k) {
            p += (int64_t)decoded(c, flags, K, lzs_group, m, k) * wq[n * K + k];
            wsum += wq[n * K + k];
        }
        int64_t pz = p - (int64_t)zeros[m * G + g] * wsum;
        double t = (double)qo_f16_to_f32(scales[m * G + g]) * (double)qo_f16_to_f32(sw[n * G + g]) *
                   (double)pz;
        y += t;
        a += fabs(t);
    }
    if (bias) {
        double b = (double)qo_bf16_to_f32(bias[n]);
        y += b;
        a += fabs(b);
    }
    if (epilogue == 1)
        y = qo_gelu_tanh(y);
    if (absum)
        *absum = a;
    return y;
}

int qo_linear_asym_f64(const int8_t* c, const uint8_t* flags, const uint16_t* scales,
                       const int8_t* zeros, const int8_t* wq, const uint16_t* sw,
                       const uint16_t* bias, int64_t M, int64_t N, int64_t K, int lzs_group,
                       int epilogue, double* y, double* absum)
{
    if (K % 64 != 0 || lzs_group < 1 || 64 % lzs_group != 0)
        return QO_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n)
            y[m * N + n] = linear_asym_one(c, flags, scales, zeros, wq, sw, bias, K, lzs_group,
                                           epilogue, m, n, absum ? &absum[m * N + n] : NULL);
    return QO_OK;
}

/* ------------------------------------------- LDM setting (reading R8) */

/*
 * Static per-tensor activation quantizer: Stage 1 with the given scale s
 * (fp32, s > 0), then Stage 2 per subgroup of lzs_group elements.  Outputs
 * as qo_quantize_act (q8 may be NULL); there are no per-group scales.
 */
int qo_quantize_act_static(const uint16_t* x, int64_t M, int64_t K, int64_t ldx, float s,
                           int lzs_group, int8_t* q8, int8_t* c, uint8_t* flags)
{
    if (!(s > 0.0f) || lzs_group < 1 || 64 % lzs_group != 0 || K % 64 != 0 || ldx < K)
        return QO_EINVAL;
    const float r = 1.0f / s;                    /* IEEE binary32 division */
    const int64_t S = K / lzs_group;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t j = 0; j < S; ++j) {
            int8_t q[64];
            for (int i = 0; i < lzs_group; ++i) {
                float p = qo_bf16_to_f32(x[m * ldx + j * lzs_group + i]) * r;
                double v = qo_rne((double)p);
                if (v > 127.0)
                    v = 127.0;
                if (v < -127.0)
                    v = -127.0;
                q[i] = (int8_t)v;
                if (q8)
                    q8[m * K + j * lzs_group + i] = q[i];
            }
            flags[m * S + j] = (uint8_t)qo_lzs_subgroup(q, lzs_group, c + m * K + j * lzs_group);
        }
    }
    return QO_OK;
}

/* Per-channel weight quantizer: one fp16 scale per output channel n. */
int qo_quantize_weight_per_channel(const uint16_t* w, int64_t N, int64_t K, int8_t* wq,
                                   uint16_t* sw)
{
    if (K % 64 != 0)
        return QO_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        float beta = 0.0f;
        for (int64_t k = 0; k < K; ++k) {
            float a = fabsf(qo_bf16_to_f32(w[n * K + k]));
            if (a > beta)
                beta = a;
        }
        uint16_t s16 = qo_f32_to_f16_rne_sat(beta / 7.0f);
        float sc = qo_f16_to_f32(s16);
        float r = (sc == 0.0f) ? 0.0f : 1.0f / sc;
        sw[n] = s16;
        for (int64_t k = 0; k < K; ++k) {
            float p = qo_bf16_to_f32(w[n * K + k]) * r;
            double v = qo_rne((double)p);
            if (v > 7.0)
                v = 7.0;
            if (v < -7.0)
                v = -7.0;
            wq[n * K + k] = (int8_t)v;
        }
    }
    return QO_OK;
}

/*
 * One output of the LDM-setting layer, in double:
 *   y = s * s_w[n] * I[m,n] + bias[n]   (then GELU-tanh),
 * I = sum over all k of d[m,k] * wq[n,k] (exact).  *absum receives
 * S = |s * s_w[n] * I| + |bias|.
 */
static double linear_static_one(const int8_t* c, const uint8_t* flags, float s, const int8_t* wq,
                                const uint16_t* sw, const uint16_t* bias, int64_t K,
                                int lzs_group, int epilogue, int64_t m, int64_t n, double* absum)
{
    int64_t I = 0;
    for (int64_t k = 0; k < K; ++k)
        I += (int64_t)decoded(c, flags, K, lzs_group, m, k) * wq[n * K + k];
    double t = (double)s * (double)qo_f16_to_f32(sw[n]) * (double)I;
    double y = t, a = fabs(t);
    if (bias) {
        double b = (double)qo_bf16_to_f32(bias[n]);
        y += b;
        a += fabs(b);
    }
    if (epilogue == 1)
        y = qo_gelu_tanh(y);
    if (absum)
        *absum = a;
    return y;
}

int qo_linear_static_f64(const int8_t* c, const uint8_t* flags, float s, const int8_t* wq,
                         const uint16_t* sw, const uint16_t* bias, int64_t M, int64_t N, int64_t K,
                         int lzs_group, int epilogue, double* y, double* absum)
{
    if (K % 64 != 0 || lzs_group < 1 || 64 % lzs_group != 0)
        return QO_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n)
            y[m * N + n] = linear_static_one(c, flags, s, wq, sw, bias, K, lzs_group, epilogue, m,
                                             n, absum ? &absum[m * N + n] : NULL);
    return QO_OK;
}

/* -------------------------------------------- LZS attention (reading R11) */

/*
 * The activation quantizer (Eq. 1 under R1/R2, then Eq. 2 and the right
 * shift per subgroup) applied to binary32 inputs instead of bf16 ones: the
 * form it takes on the softmax output, which is computed in binary32.  Per
 * 64-group: alpha = max |x|, s16 = fp16(alpha / 127), r = 1/s,
 * q = clamp(rne(fp32(x r)), -127, 127).  Outputs as qo_quantize_act
 * (row-major c [M][K], flags [M][K/lzs_group], scales [M][K/64]).
 */
int qo_quantize_f32(const float* x, int64_t M, int64_t K, int64_t ldx, int lzs_group, int8_t* c,
                    uint8_t* flags, uint16_t* scales)
{
    if (lzs_group < 1 || 64 % lzs_group != 0 || K % 64 != 0 || ldx < K)
        return QO_EINVAL;
    const int64_t G = K / 64, S = K / lzs_group;
#pragma omp parallel for schedule(static)
    for (int64_t m = 0; m < M; ++m) {
        for (int64_t g = 0; g < G; ++g) {
            const float* xg = x + m * ldx + g * 64;
            float alpha = 0.0f;
            for (int k = 0; k < 64; ++k) {
                float a = fabsf(xg[k]);
                if (a > alpha)
                    alpha = a;
            }
            uint16_t s16 = qo_f32_to_f16_rne_sat(alpha / 127.0f);
            float sv = qo_f16_to_f32(s16);
            float r = (sv == 0.0f) ? 0.0f : 1.0f / sv;
            int8_t q[64];
            for (int k = 0; k < 64; ++k) {
                double v = qo_rne((double)(xg[k] * r));
                if (v > 127.0)
                    v = 127.0;
                if (v < -127.0)
                    v = -127.0;
                q[k] = (int8_t)v;
            }
            scales[m * G + g] = s16;
            for (int j = 0; j < 64 / lzs_group; ++j) {
                int64_t sub = g * (64 / lzs_group) + j;
                flags[m * S + sub] = (uint8_t)qo_lzs_subgroup(q + j * lzs_group, lzs_group,
                                                               c + m * K + g * 64 + j * lzs_group);
            }
        }
    }
    return QO_OK;
}

/*
 * Row softmax of scores S [M][lds] (N columns) in double:
 *   P[i][j] = exp(S[i][j] - max_j S[i][j]) / sum_j exp(S[i][j] - max_j S[i][j]),
 * stored as binary32 (round to nearest) in P [M][N].
 */
int qo_softmax_rows(const double* S, int64_t M, int64_t N, int64_t lds, float* P)
{
    if (N <= 0 || lds < N)
        return QO_EINVAL;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < M; ++i) {
        const double* row = S + i * lds;
        double mx = row[0];
        for (int64_t j = 1; j < N; ++j)
            if (row[j] > mx)
                mx = row[j];
        double sum = 0.0;
        for (int64_t j = 0; j < N; ++j)
            sum += exp(row[j] - mx);
        for (int64_t j = 0; j < N; ++j)
            P[i * N + j] = (float)(exp(row[j] - mx) / sum);
    }
    return QO_OK;
}

/*
 * bf16 bit patterns (round to nearest even) of n float64 values: the bf16
 * output a layer stores for its float64 results, elementwise.
 */
void qo_round_bf16(const double* v, int64_t n, uint16_t* out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = qo_f64_to_bf16_rne(v[i]);
}

/* Number of threads the OpenMP loops above use. */
#ifdef _OPENMP
#include <omp.h>
#endif
int qo_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
