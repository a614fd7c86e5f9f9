/*
 * quartz.h -- C ABI of libquartz.so, the MI355X (gfx950) W4A4 linear-layer hot
 * path of QuaRTZ ("Post-Training Quantization via Residual Truncation and Zero
 * Suppression for Diffusion Models", arXiv 2509.26436).
 *
 * The activation side follows the paper's two stages: an 8-bit min-max
 * quantization per 64-element group (Eq. 1, symmetric reading: s = max|x|/127,
 * zero point 0) and leading-zero suppression of each subgroup of G_s codes to
 * 4 bits plus a shift FLAG = max(29 - clz(OR of magnitudes), 0) (Eq. 2), with
 * the magnitudes right-shifted by FLAG, truncating toward zero (Section 3 and
 * Appendix A).  Weights are symmetric round-to-nearest int4 per 64-element
 * group with 16-bit scales (Appendix C; GPTQ is an offline step outside this
 * library).  The GEMM multiplies the decoded integers d = c * 2^FLAG with the
 * 4-bit weights exactly per 64-group, which equals the paper's integer MMA
 * with a per-subgroup power-of-two shift (Section 4.4), then applies the two
 * fp16 group scales, the bias and an optional GELU.
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE pointers unless stated otherwise; the caller
 *     allocates and owns every buffer.  The library allocates nothing and
 *     keeps no state between calls.
 *   - Work is enqueued asynchronously on `stream` (0 = the null stream);
 *     outputs are valid once the stream reaches that point.
 *   - Arguments are validated on the host before anything is launched; on an
 *     error nothing is launched and no output is written.  A launch failure
 *     returns QUARTZ_ERR_HIP.  Nothing aborts, throws or prints.
 *   - Inputs must not alias outputs.  All base pointers must be 16-byte
 *     aligned (QUARTZ_ERR_ALIGN otherwise).
 *   - bf16 and fp16 values are passed as their 16-bit IEEE-style patterns.
 *   - Only group_size = 64 (Appendix C) is supported; lzs_group (the LZS
 *     subgroup size G_s of Section 3) must be 8, 16, 32 or 64.
 *   - Input precondition: finite activations and weights; NaN / Inf give
 *     unspecified codes.
 */
#ifndef QUARTZ_H
#define QUARTZ_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum quartz_status {
    QUARTZ_OK = 0,
    QUARTZ_ERR_NULL = 1,        /* a required pointer is NULL */
    QUARTZ_ERR_SHAPE = 2,       /* negative size, K % 64 != 0, ld too small, too large */
    QUARTZ_ERR_UNSUPPORTED = 3, /* group_size, lzs_group, mode or epilogue not supported */
    QUARTZ_ERR_ALIGN = 4,       /* a pointer is not 16-byte aligned */
    QUARTZ_ERR_HIP = 5,         /* the kernel launch failed */
    QUARTZ_ERR_WORKSPACE = 6    /* workspace smaller than the size query asks for */
} quartz_status;

enum { QUARTZ_MODE_SYMMETRIC = 0, QUARTZ_MODE_ASYMMETRIC = 1 };
enum { QUARTZ_EPI_NONE = 0, QUARTZ_EPI_GELU_TANH = 1 };

/*
 * Activation quantizer: Stage 1 (Eq. 1) and Stage 2 (Eq. 2 + right shift) in
 * one pass over x.
 *
 *   x_bf16  bf16 [M][ldx], row-major, K <= ldx <= 2^24, ldx % 8 == 0.
 *   M, K    rows (tokens) and reduction size; K % 64 == 0.
 *   mode    QUARTZ_MODE_SYMMETRIC (s = max|x| / 127 per 64-group, zero point 0), or
 *           QUARTZ_MODE_ASYMMETRIC: Eq. 1's zero point, with the range repaired
 *           so that the 255 signed levels cover it: lo = min(x_min, 0),
 *           hi = max(x_max, 0), s = fp16(fp32(hi - lo) / 254) (RNE,
 *           saturating), r = fp32(1/s), z = clamp(-127 - rne(fp32(lo r)),
 *           -127, 127), q = clamp(rne(fp32(x r)) + z, -127, 127); Stage 2 then
 *           acts on q; the decoded value is s * (c * 2^FLAG - z).  zeros is
 *           required (QUARTZ_ERR_NULL otherwise).
 * Outputs, K-group-major (all rows of 64-group 0, then all rows of group 1, ...),
 * so that one group of a tile of rows is one contiguous run for the GEMM:
 *   codes   u8  [K/64][M][32]   4-bit codes c in [-7, 7] of the 64 elements of
 *                         (group, row), sign-magnitude nibbles (bit 3 = sign,
 *                         bits 0..2 = |c|; c = 0 is stored as 0).  Elements
 *                         8j..8j+7 of the group form the little-endian 32-bit
 *                         word j of its 32 bytes; element 8j+i is nibble
 *                         (i/2) + 4*(i%2) of that word (even elements in the
 *                         low half-word).
 *   flags   u8  [K/64][M][64/lzs_group]  FLAG in 0..4 of each subgroup.
 *   scales  u16 [K/64][M]   fp16 scale s of each (group, row): fp16(max|x| / 127),
 *                         round-to-nearest-even, saturating at 65504.
 *   zeros   i8  [K/64][M] zero point z of each (group, row); may be NULL in
 *           the symmetric mode, which writes 0.
 * The decoded activation is x~ = s * (c * 2^FLAG - z).
 * M = 0 returns QUARTZ_OK without launching.
 */
quartz_status quartz_quantize_act(const void* x_bf16, int64_t M, int64_t K, int64_t ldx,
                                  int32_t group_size, int32_t lzs_group, int32_t mode,
                                  uint8_t* codes, uint8_t* flags, uint16_t* scales,
                                  int8_t* zeros, hipStream_t stream);

/* Size in bytes of the packed weight buffer for an N x K weight. */
size_t quartz_packed_weight_bytes(int64_t N, int64_t K, int32_t group_size);

/*
 * Weight pre-pack (once per layer): symmetric round-to-nearest int4 per
 * 64-group along K (Appendix C), s_w = fp16(max|w| / 7) (RNE, saturating),
 * wq = clamp(rne(w * (1/s_w)), -7, 7).
 *
 *   w_bf16    bf16 [N][K], row-major (the nn.Linear weight layout).
 *   w_packed  quartz_packed_weight_bytes(N, K, 64) bytes, opaque to callers:
 *             panels of 64 output columns; per (panel, group) 64 x 32 bytes of
 *             codes, eight sign-magnitude codes per 32-bit word (the
 *             activation-code nibble order with each sign bit moved next to
 *             a magnitude so that a mask, or a 4-bit rotation and the mask,
 *             yields the fp8 operands directly), followed by the 64 fp16
 *             scales; columns past N are zero.
 *   w_scales  u16 [N][K/64] plain copy of the fp16 scales, or NULL.
 * N = 0 returns QUARTZ_OK without launching.
 */
quartz_status quartz_pack_weight(const void* w_bf16, int64_t N, int64_t K, int32_t group_size,
                                 void* w_packed, uint16_t* w_scales, hipStream_t stream);

/*
 * W4A4 linear layer: for every output (m, n)
 *   y[m][n] = bf16( act( sum_g s_a[m,g] * s_w[n,g] * P_g[m,n] + bias[n] ) )
 * with P_g = sum over the 64 k of group g of (c[m,k] * 2^FLAG) * wq[n,k],
 * computed exactly (|P_g| <= 112 * 7 * 64 < 2^24); the scales and the sum
 * over groups are applied in fp32, act is the identity or GELU (tanh form).
 *
 *   codes, flags, scales, zeros   outputs of quartz_quantize_act in
 *                                 QUARTZ_MODE_SYMMETRIC for the same M, K,
 *                                 lzs_group (zeros is not read and may be
 *                                 NULL).  Codes of QUARTZ_MODE_ASYMMETRIC
 *                                 need quartz_w4a4_linear_asym: their zero
 *                                 points are not applied here.
 *   w_packed    output of quartz_pack_weight for N, K.
 *   bias_bf16   bf16 [N] or NULL.
 *   y_bf16      bf16 [M][ldy], N <= ldy <= 2^24.
 *   epilogue    QUARTZ_EPI_NONE or QUARTZ_EPI_GELU_TANH.
 * M = 0 or N = 0 returns QUARTZ_OK without launching.  The output has at most
 * 2^31 - 1 tiles of 256 x 128 (QUARTZ_ERR_SHAPE otherwise).
 * The kernel is persistent: one workgroup per compute unit walks its share of
 * the output tiles as one continuous pipeline (Section 4.4 fixes no order).
 */
quartz_status quartz_w4a4_linear(const uint8_t* codes, const uint8_t* flags,
                                 const uint16_t* scales, const int8_t* zeros,
                                 const void* w_packed, const void* bias_bf16, void* y_bf16,
                                 int64_t M, int64_t N, int64_t K, int64_t ldy,
                                 int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                 hipStream_t stream);

/*
 * The same W4A4 linear layer with a caller-provided workspace, which lets the
 * GEMM balance its work over the whole device: when the output tiles do not
 * fill a whole number of rounds of one workgroup per compute unit, the grid
 * becomes persistent and the tiles of the last rounds are cut along K
 * (stream-K); a tile shared by several workgroups gets their fp32 partial
 * sums added in a fixed order by the last one to finish, so results are
 * deterministic.  The values are those of quartz_w4a4_linear up to the fp32
 * summation order over groups (Section 4.4 fixes no order).
 *
 *   workspace        device memory, 16-byte aligned, at least
 *                    quartz_w4a4_linear_workspace_bytes(M, N, K, 64) bytes,
 *                    or NULL (then this is exactly quartz_w4a4_linear).
 *                    Its first use must find it zero-filled; every call leaves
 *                    it ready for the next one.  Calls that use one workspace
 *                    must not overlap in time (one stream, or synchronized).
 *   workspace_bytes  its size; a smaller size than the query gives returns
 *                    QUARTZ_ERR_WORKSPACE and launches nothing.
 * The other arguments are those of quartz_w4a4_linear.  The library does not
 * keep the workspace between calls; the caller owns it.
 *
 * quartz_w4a4_linear_workspace_bytes: the size for this M, N, K on the
 * current device (it depends on its number of compute units); 0 when the
 * tiles fill whole rounds (then NULL may be passed) or the sizes are invalid.
 */
size_t quartz_w4a4_linear_workspace_bytes(int64_t M, int64_t N, int64_t K, int32_t group_size);

quartz_status quartz_w4a4_linear_ws(const uint8_t* codes, const uint8_t* flags,
                                    const uint16_t* scales, const int8_t* zeros,
                                    const void* w_packed, const void* bias_bf16, void* y_bf16,
                                    int64_t M, int64_t N, int64_t K, int64_t ldy,
                                    int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * quartz_w4a4_linear_noalloc: quartz_w4a4_linear_ws for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments as quartz_w4a4_linear,
 * same results as quartz_w4a4_linear_ws with a workspace (the same schedule
 * and split, hence bit-identical outputs), but the stream-K partial sums and
 * counters live in a scratch array the library holds in device memory on
 * every GPU it runs on, until the process ends:
 *   - its size is quartz_w4a4_linear_noalloc_max_bytes() (64 MiB + 64 KiB,
 *     the workspace of a persistent grid of up to 256 workgroups); a shape
 *     whose workspace (quartz_w4a4_linear_workspace_bytes) is larger returns
 *     QUARTZ_ERR_WORKSPACE and launches nothing;
 *   - nothing is allocated: no hipMalloc, hipFree or allocating library call;
 *   - each call first clears the counters with a small kernel on `stream`
 *     (no memset node, so the call may be captured into a graph);
 *   - every call on one GPU shares that GPU's array: calls that overlap in
 *     time on one GPU (two streams, two threads) race and give wrong results.
 * Errors as for quartz_w4a4_linear_ws.
 */
quartz_status quartz_w4a4_linear_noalloc(const uint8_t* codes, const uint8_t* flags,
                                         const uint16_t* scales, const int8_t* zeros,
                                         const void* w_packed, const void* bias_bf16, void* y_bf16,
                                         int64_t M, int64_t N, int64_t K, int64_t ldy,
                                         int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                         hipStream_t stream);

size_t quartz_w4a4_linear_noalloc_max_bytes(void);

/*
 * W4A4 linear layer whose output is quantized on the fly for the next layer
 * (Appendix C applies the 4-bit compression on the fly; Eq. 1 and Eq. 2 as
 * for quartz_quantize_act): the bf16 values quartz_w4a4_linear_ws would
 * store, y[m][n] = bf16(act(sum_g s_a s_w P_g + bias[n])), are not written;
 * instead the epilogue quantizes each row's 64-column groups of y exactly as
 * quartz_quantize_act does with K = N (same codes, flags and scales,
 * bit for bit, as quantizing the stored bf16 output), and writes them in
 * quartz_quantize_act's layout.  This removes the bf16 round trip through
 * memory between two layers (the producer's store and the quantizer's load).
 *
 *   codes ... epilogue   as for quartz_w4a4_linear (K % 64 == 0).
 *   N             the next layer's K: N % 64 == 0 (QUARTZ_ERR_SHAPE otherwise).
 *   out_lzs_group the next layer's G_s: 8, 16, 32 or 64.
 *   out_mode      QUARTZ_MODE_SYMMETRIC.
 *   out_codes     u8  [N/64][M][32]
 *   out_flags     u8  [N/64][M][64/out_lzs_group]
 *   out_scales    u16 [N/64][M]
 *   out_zeros     i8  [N/64][M] or NULL (written as 0).
 *   workspace, workspace_bytes   as for quartz_w4a4_linear_ws (NULL, 0: no
 *                 split tiles); the values do not depend on it beyond the
 *                 fp32 summation order of quartz_w4a4_linear_ws.
 * M = 0 or N = 0 returns QUARTZ_OK without launching.
 */
quartz_status quartz_w4a4_linear_quantize(const uint8_t* codes, const uint8_t* flags,
                                          const uint16_t* scales, const int8_t* zeros,
                                          const void* w_packed, const void* bias_bf16, int64_t M,
                                          int64_t N, int64_t K, int32_t group_size,
                                          int32_t lzs_group, int32_t epilogue,
                                          int32_t out_lzs_group, int32_t out_mode,
                                          uint8_t* out_codes, uint8_t* out_flags,
                                          uint16_t* out_scales, int8_t* out_zeros, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream);

/*
 * The asymmetric mode (Eq. 1's zero point; the activation side is
 * QUARTZ_MODE_ASYMMETRIC of quartz_quantize_act).  With x~ = s_a (d - z),
 * d = c * 2^FLAG, the group product of the layer is
 *   sum over the group of (d - z) wq = P_g - z[m,g] * W_g[n],
 *   W_g[n] = sum over the 64 k of group g of wq[n,k]  (the weight group sums),
 * so that for every output (m, n)
 *   y[m][n] = bf16( act( sum_g s_a[m,g] s_w[n,g] (P_g - z[m,g] W_g[n]) + bias[n] ) ).
 * P_g - z W_g is exact (|.| < 2^17) before the fp32 scaling.
 *
 * quartz_weight_group_sums: W_g[n] from a packed weight (once per layer).
 *   w_packed   output of quartz_pack_weight for N, K.
 *   w_sums     i16 [K/64][N] (group-major), caller-allocated.
 *
 * quartz_w4a4_linear_asym: the layer above.
 *   codes, flags, scales, zeros   outputs of quartz_quantize_act in
 *                                 QUARTZ_MODE_ASYMMETRIC (zeros required).
 *   w_packed, w_sums              quartz_pack_weight and quartz_weight_group_sums.
 *   The other arguments are those of quartz_w4a4_linear_ws (the same
 *   workspace size query applies; NULL, 0: no split tiles).
 */
quartz_status quartz_weight_group_sums(const void* w_packed, int64_t N, int64_t K,
                                      int32_t group_size, int16_t* w_sums, hipStream_t stream);

quartz_status quartz_w4a4_linear_asym(const uint8_t* codes, const uint8_t* flags,
                                      const uint16_t* scales, const int8_t* zeros,
                                      const void* w_packed, const int16_t* w_sums,
                                      const void* bias_bf16, void* y_bf16, int64_t M, int64_t N,
                                      int64_t K, int64_t ldy, int32_t group_size,
                                      int32_t lzs_group, int32_t epilogue, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream);

/*
 * The LDM setting (the paper's experimental-details appendix): static
 * per-tensor activation quantization and per-channel weight quantization,
 * with the 4-bit LZS compression of Section 3 applied on the fly.
 *
 * quartz_quantize_act_static: Stage 1 with one scale s for the whole tensor,
 * fixed ahead of time (calibration is not part of this library):
 *   q = clamp(rne(fp32(x * r)), -127, 127),  r = fp32(1 / s)  (values beyond
 *   127 s clip), then Stage 2 exactly as quartz_quantize_act.
 *   scale      fp32 s, positive, normal and finite (QUARTZ_ERR_UNSUPPORTED
 *              otherwise).
 *   codes, flags   as for quartz_quantize_act; no scales or zero points.
 *   Other arguments and errors as for quartz_quantize_act.
 *
 * quartz_pack_weight_per_channel: one fp16 scale per output channel,
 *   s_w[n] = fp16(max over all of K of |w[n,k]| / 7) (RNE, saturating),
 *   wq = clamp(rne(w * (1/s_w[n])), -7, 7); the same packed layout and size
 *   as quartz_pack_weight (quartz_packed_weight_bytes), with s_w[n] in every
 *   group's scale slot, so quartz_unpack_weight reads it back alike.
 *   w_scales   u16 [N] copy of the channel scales, or NULL.
 *
 * quartz_w4a4_linear_static: for every output (m, n)
 *   y[m][n] = bf16( act( act_scale * s_w[n] * I[m,n] + bias[n] ) ),
 *   I[m,n] = sum over all k of (c[m,k] * 2^FLAG) * wq[n,k],
 * accumulated by the matrix cores in fp32: exact while every partial sum
 * stays below 2^24 in magnitude, which |I| <= 784 K guarantees for K <=
 * 21376 (beyond that, within fp32 rounding of the sum).
 *   codes, flags   output of quartz_quantize_act_static for M, K, lzs_group.
 *   act_scale      the s given to quartz_quantize_act_static (any finite fp32).
 *   w_packed       output of quartz_pack_weight_per_channel for N, K.
 *   bias_bf16, y_bf16, ldy, epilogue, workspace, workspace_bytes
 *                  as for quartz_w4a4_linear_ws (the same workspace size
 *                  query applies; NULL, 0: no split tiles).
 */
quartz_status quartz_quantize_act_static(const void* x_bf16, int64_t M, int64_t K, int64_t ldx,
                                         float scale, int32_t lzs_group, uint8_t* codes,
                                         uint8_t* flags, hipStream_t stream);

quartz_status quartz_pack_weight_per_channel(const void* w_bf16, int64_t N, int64_t K,
                                             void* w_packed, uint16_t* w_scales,
                                             hipStream_t stream);

quartz_status quartz_w4a4_linear_static(const uint8_t* codes, const uint8_t* flags,
                                        float act_scale, const void* w_packed,
                                        const void* bias_bf16, void* y_bf16, int64_t M, int64_t N,
                                        int64_t K, int64_t ldy, int32_t lzs_group,
                                        int32_t epilogue, void* workspace, size_t workspace_bytes,
                                        hipStream_t stream);

/*
 * Test / inspection helpers.
 *
 * quartz_unpack_weight: int8 [N][K] weight codes wq recovered from w_packed.
 * quartz_w4a4_gemm_i32: the exact integer accumulator
 *   acc[m][n] = sum_k (c[m,k] * 2^FLAG) * wq[n,k]   (int32 [M][N], row-major),
 * i.e. the sum of the per-group integer MMA results before any scaling
 * (Section 4.4's s32 accumulation): each group product is exact and the
 * groups are added in int32, so acc is exact for every K accepted
 * (|acc| <= 784 K <= 784 * 2^20 < 2^31).
 */
quartz_status quartz_unpack_weight(const void* w_packed, int64_t N, int64_t K,
                                   int32_t group_size, int8_t* wq_out, hipStream_t stream);

quartz_status quartz_w4a4_gemm_i32(const uint8_t* codes, const uint8_t* flags,
                                   const void* w_packed, int32_t* acc_out, int64_t M, int64_t N,
                                   int64_t K, int32_t group_size, int32_t lzs_group,
                                   hipStream_t stream);

/*
 * 3 x 3 convolution (stride 1, padding 1) of the UNet backbones evaluated in
 * Section 5 (LDM, SD v1.4, SDXL-Turbo), as the W4A4 layer on its im2col
 * matrix: row m = (image * H + h) * W + w is output pixel (h, w) of an image,
 * and K = 9 C runs over the taps (kh, kw) and the C input channels, c
 * fastest, with zero padding outside the image.  The im2col matrix is never
 * formed: with C % 64 == 0 every 64-group of an im2col row is the 64
 * channels of one input pixel (or zero padding), and a group's scale, FLAGs
 * and codes depend on its 64 values only, so quantizing the feature map
 * once gives the codes of every im2col row; the GEMM reads them at the
 * pixel each tap points to.  The result equals quartz_w4a4_linear_ws (or
 * quartz_w4a4_linear_static) on the quantized im2col matrix, bit for bit.
 *
 * quartz_w4a4_conv3x3: the per-group setting.
 *   codes, flags, scales  outputs of quartz_quantize_act for the feature map
 *                         x [images * H * W][C] (NHWC, K = C), symmetric mode.
 *   w_packed   quartz_pack_weight of the weight [N][9 C], K ordered
 *              (kh, kw, c) with c fastest.
 *   bias_bf16, y_bf16 [images * H * W][ldy], epilogue, workspace,
 *   workspace_bytes   as for quartz_w4a4_linear_ws, with M = images * H * W
 *              and K = 9 C (the same workspace size query applies).
 *   images >= 0, H, W >= 1, C > 0 with C % 64 == 0, images * H * W < 2^26,
 *   9 C <= 2^20: QUARTZ_ERR_SHAPE otherwise; other errors as for
 *   quartz_w4a4_linear_ws.
 *
 * quartz_w4a4_conv3x3_static: the LDM setting: codes and flags of
 *   quartz_quantize_act_static for the feature map with act_scale, w_packed
 *   of quartz_pack_weight_per_channel for the weight [N][9 C]; otherwise as
 *   quartz_w4a4_conv3x3 (equal to quartz_w4a4_linear_static on the im2col
 *   matrix).
 */
quartz_status quartz_w4a4_conv3x3(const uint8_t* codes, const uint8_t* flags,
                                  const uint16_t* scales, const void* w_packed,
                                  const void* bias_bf16, void* y_bf16, int64_t images, int64_t H,
                                  int64_t W, int64_t C, int64_t N, int64_t ldy,
                                  int32_t group_size, int32_t lzs_group, int32_t epilogue,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream);

quartz_status quartz_w4a4_conv3x3_static(const uint8_t* codes, const uint8_t* flags,
                                         float act_scale, const void* w_packed,
                                         const void* bias_bf16, void* y_bf16, int64_t images,
                                         int64_t H, int64_t W, int64_t C, int64_t N, int64_t ldy,
                                         int32_t lzs_group, int32_t epilogue, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream);

/*
 * LZS attention: the attention setting of the paper's hardware appendix
 * (Table 8: heads x 128, G_s 8 / 16 / 32), read as follows (the paper leaves
 * the operation open): per head, O = softmax(Q K^T / sqrt(d)) V, non-causal,
 * where Q, K, V and the softmax output are all activations and so each goes
 * through the activation quantizer (Eq. 1, Eq. 2) -- Q and K per token along
 * d, V^T per channel along the keys, the softmax output P (computed in fp32)
 * per query row in 64-key groups -- and both products are exact per-group
 * integer products with the two fp16 group scales applied in fp32, as in the
 * linear layer (Section 4.4).  S is kept in fp32 between the products.
 *
 * quartz_quantize_vt: V^T quantized along the keys.
 *   v_bf16   bf16 [heads * L][ldv]: row h * L + j is key j of head h, d channels.
 *   codes    u8  [L/64][heads * d][32]   (row h * d + c: channel c of head h)
 *   flags    u8  [L/64][heads * d][64/lzs_group],  scales u16 [L/64][heads * d]
 *   L % 64 == 0, d % 64 == 0, d <= ldv, ldv % 8 == 0.
 *
 * quartz_attn_scores: one head's scores, s[i][j] = scale * sum over the
 * 64-groups of d of s_q s_k P_g (fp32), i < Lq, j < Lk, row stride lds >= Lk.
 *   q_*   quartz_quantize_act outputs for queries with K = d; the head's rows
 *         are rows q_row0 .. q_row0 + Lq - 1 of planes of q_plane rows (the M
 *         of that call); k_* likewise for the keys.
 *
 * quartz_softmax_quantize: s fp32 [M][lds] (N columns, N % 64 == 0) ->
 *   P = exp(s - rowmax) / rowsum in fp32, then quartz_quantize_act's Stage 1
 *   and Stage 2 on the fp32 values of P with K = N: codes [N/64][M][32],
 *   flags [N/64][M][64/lzs_group], scales [N/64][M].
 *
 * quartz_attn_pv: one head's output o[i][c] = bf16(sum over 64-key groups of
 *   s_p s_v P_g) for i < Lq, c < d (row stride ldo >= d), from the quantized
 *   softmax output (quartz_softmax_quantize with M = Lq, N = Lk) and V^T
 *   (quartz_quantize_vt; the head's channels are rows vt_row0 .. + d - 1 of
 *   planes of vt_plane rows).  workspace / workspace_bytes as for
 *   quartz_w4a4_linear_ws (size: quartz_attn_pv_workspace_bytes; NULL, 0: no
 *   split tiles).
 *
 * quartz_lzs_attention: all heads end to end.
 *   q_bf16, k_bf16, v_bf16   bf16 [heads][L][d], contiguous.
 *   o_bf16   bf16 [L][ldo], ldo >= heads * d, ldo % 4 == 0: head h in
 *            columns h d .. h d + d - 1; nothing else of o is written.
 *   workspace  quartz_lzs_attention_workspace_bytes(heads, L, d, lzs_group)
 *              bytes.  It holds the quantized Q, K, V^T of all heads and:
 *              for d = 64 and 128, the same expanded to fp8 e4m3 for the fused
 *              kernel (two sweeps over the keys per query row, the first for
 *              the row's max and sum, the second for P, its quantization and
 *              the PV product; S never leaves registers); for other d, one
 *              head's fp32 scores and quantized softmax output of the stage
 *              pipeline above, run head by head, and the PV split workspace,
 *              which must be zero-filled before its first use (every call
 *              leaves it zero again).
 *   L % 64 == 0 (L <= 2^16), d % 64 == 0.  Both paths compute the quantities
 *   defined above; they differ only in fp32 rounding (the fused kernel's
 *   exponentials are base-2 hardware exponentials of x log2(e) / sqrt(d)).
 *   Calls that share a workspace must not overlap.
 * Errors as for the other entry points; lzs_group must be 8, 16, 32 or 64.
 */
quartz_status quartz_quantize_vt(const void* v_bf16, int64_t heads, int64_t L, int64_t d,
                                 int64_t ldv, int32_t lzs_group, uint8_t* codes, uint8_t* flags,
                                 uint16_t* scales, hipStream_t stream);

quartz_status quartz_attn_scores(const uint8_t* q_codes, const uint8_t* q_flags,
                                 const uint16_t* q_scales, int64_t q_plane, int64_t q_row0,
                                 const uint8_t* k_codes, const uint8_t* k_flags,
                                 const uint16_t* k_scales, int64_t k_plane, int64_t k_row0,
                                 int64_t Lq, int64_t Lk, int64_t d, int32_t lzs_group, float scale,
                                 float* s, int64_t lds, hipStream_t stream);

quartz_status quartz_softmax_quantize(const float* s, int64_t M, int64_t N, int64_t lds,
                                      int32_t lzs_group, uint8_t* codes, uint8_t* flags,
                                      uint16_t* scales, hipStream_t stream);

size_t quartz_attn_pv_workspace_bytes(int64_t Lq, int64_t Lk, int64_t d);

quartz_status quartz_attn_pv(const uint8_t* p_codes, const uint8_t* p_flags,
                             const uint16_t* p_scales, const uint8_t* vt_codes,
                             const uint8_t* vt_flags, const uint16_t* vt_scales, int64_t vt_plane,
                             int64_t vt_row0, int64_t Lq, int64_t Lk, int64_t d,
                             int32_t lzs_group, void* o_bf16, int64_t ldo, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

size_t quartz_lzs_attention_workspace_bytes(int64_t heads, int64_t L, int64_t d,
                                            int32_t lzs_group);

quartz_status quartz_lzs_attention(const void* q_bf16, const void* k_bf16, const void* v_bf16,
                                   int64_t heads, int64_t L, int64_t d, int32_t lzs_group,
                                   void* o_bf16, int64_t ldo, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/*
 * quartz_w4a4_linear_schedule (host only, needs no GPU): the GEMM work
 * schedule for a persistent grid of at most `blocks` workgroups (the entry
 * points use the device's compute-unit count), with (split = 1, as
 * quartz_w4a4_linear_ws) or without (split = 0, as quartz_w4a4_linear) tiles
 * cut along K, for tiles of 128 x 256 (tiles = 0: quartz_w4a4_linear and its
 * variants, quartz_w4a4_linear_quantize, quartz_w4a4_linear_static and
 * quartz_w4a4_linear_asym) or of 256 x 128 (tiles = 1: the convolutions, the
 * exact integer accumulator and the attention products).
 *   schedule  host int32[10]: tiles_n, groups, split, blocks, whole tiles of
 *             workgroup 0, sk_first, sk_tiles, sk_blocks, sk_q, sk_r.
 *   segments  host int32[capacity][10], one row per (workgroup, segment):
 *             workgroup, segment index, tile, g0, g1 (groups [g0, g1)),
 *             split-tile index or -1, slot or -1, first and last workgroup
 *             sharing the tile (or -1), and the slot the finishing workgroup
 *             reads for this workgroup's share (or -1).
 * Returns the number of segments (rows past `capacity` are not written), -1
 * for invalid arguments (tiles not 0 or 1 included), -2 if the schedule is
 * inconsistent (a library bug).
 */
int64_t quartz_w4a4_linear_schedule(int64_t M, int64_t N, int64_t K, int32_t blocks,
                                    int32_t split, int32_t tiles, int32_t* schedule,
                                    int32_t* segments, int64_t capacity);

/* Static, NUL-terminated description of a status code (host memory). */
const char* quartz_status_string(quartz_status s);

#ifdef __cplusplus
}
#endif

#endif /* QUARTZ_H */
