/*
 * rfq.h -- C ABI of librfq: Residual Fallback Quantization (RFQ) with MXFP4
 * and HiF4 codes on AMD Instinct MI355X (gfx950).
 *
 * The library computes the data-parallel forward path of RFQ (Sec. 4.3 of the
 * paper): an MX activation quantizer that emits a primary MXFP4 code and an
 * MXFP4 code of the residual the primary code lost (Eq. 8-10), and a
 * block-scaled FP4 product that contracts both codes against MXFP4 weights
 * (Eq. 11, Algorithm 1).  The rfq_hif4_* calls at the end do the same with
 * the HiF4 format of Sec. 3.3 (64-element blocks); the number format below
 * is MXFP4's, HiF4's is described with those calls.
 *
 * Number format (Sec. 3.2, Eq. 3-4, element format of Sec. 3.2.2):
 *   - a block is 32 consecutive elements of one row along K (the reduction
 *     dimension); K must be a multiple of 32;
 *   - one E8M0 scale byte per block, value 2^(byte - 127); the block exponent
 *     is floor(log2 amax) - 2 clamped to [-127, 127], an all-zero block gets
 *     byte 0x00;
 *   - one 4-bit E2M1 code per element, sign<<3 | magnitude index, magnitudes
 *     {0, 0.5, 1, 1.5, 2, 3, 4, 6}; round to nearest, ties to even,
 *     saturating at +-6; the sign of an element that rounds to zero is kept;
 *   - codes are packed two per byte, element 2j in the low nibble of byte j;
 *   - layouts: codes[rows][K/2] bytes and scales[rows][K/32] bytes, both
 *     row-major and dense.
 *
 * Conventions shared by every call:
 *   - Ownership: the caller allocates and owns every buffer.  All data
 *     pointers are device pointers (HIP device memory of the current device).
 *     The library never allocates, frees or retains a pointer after return.
 *   - Asynchrony: every compute call is enqueued on hip_stream (a hipStream_t
 *     passed as void*; NULL selects the null stream) and returns before the
 *     work completes.  The caller synchronizes.
 *   - Errors: every call returns an rfq_status.  Arguments are validated on
 *     the host before any HIP call is made, so argument errors are reported
 *     without touching the device.  RFQ_ERR_DEVICE means the current device
 *     is not a gfx950 GPU; RFQ_ERR_LAUNCH means a HIP launch failed.  Faults
 *     inside kernels surface at the caller's next synchronization, as in HIP.
 *   - Empty work: rows == 0 (or N == 0 for the product) is a valid no-op;
 *     the pointers of such a call are not read and may be NULL.
 *   - Size limits (RFQ_ERR_SHAPE beyond them; one launch covers at most
 *     2^32 - 1 work items): K <= 2^31 in every call; quantizers at most
 *     2^32 - 64 MX blocks (rows * K / 32); products M, N < 2^31 and
 *     ceil(M/128) * ceil(N/128) * 256 < 2^32 (about M * N < 2^38, far beyond
 *     what fits in memory); dequantization and the phi map rows * K <= 2^56.
 *     Calls with further limits state them.
 *   - Thread safety: calls may be issued from several host threads; calls on
 *     one stream execute in issue order.
 */
#ifndef RFQ_H
#define RFQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes and dtype codes are 32-bit integers with named values (not
 * enum types), so that every value a caller passes or receives is defined
 * behaviour in C and in C++; unknown values are rejected or named as such. */
typedef int32_t rfq_status;
enum {
    RFQ_OK = 0,
    RFQ_ERR_NULL = 1,    /* a required pointer is NULL, or an optional pair is half given */
    RFQ_ERR_SHAPE = 2,   /* negative size, K < 32 or not a multiple of 32, or a size limit */
    RFQ_ERR_DTYPE = 3,   /* unknown rfq_dtype value */
    RFQ_ERR_ALIGN = 4,   /* a pointer violates the alignment stated for it */
    RFQ_ERR_DEVICE = 5,  /* no current HIP device, or it is not gfx950 */
    RFQ_ERR_LAUNCH = 6   /* a kernel launch failed */
};

typedef int32_t rfq_dtype;
enum {
    RFQ_F32 = 0,   /* IEEE binary32 */
    RFQ_BF16 = 1   /* bfloat16 (upper half of a binary32) */
};

/* Rules that build a fallback-indicator map (the paper defines phi(p, r) as
 * an input of Algorithm 1 but gives no rule; these two are this library's). */
enum {
    RFQ_PHI_RESIDUAL_NONZERO = 0,   /* phi = 1 where a residual code of the tile is nonzero */
    RFQ_PHI_SCALE_AT_LEAST = 1      /* phi = 1 where a primary scale byte of the tile >= threshold */
};

/*
 * RFQ activation quantizer: primary code Q(X) (Eq. 8) and, when r_codes and
 * r_scales are given, the residual DeltaX = X - deq(Q(X)) (Eq. 9) quantized
 * with its own block scales (Eq. 10).  The residual is formed in registers
 * and never written to memory.
 *   x        [M][K] row-major, element type x_dtype; 16-byte aligned.
 *   q_codes  [M][K/2] bytes, 16-byte aligned.    q_scales [M][K/32] bytes.
 *   r_codes  [M][K/2] bytes, 16-byte aligned, or NULL.
 *   r_scales [M][K/32] bytes, or NULL.  Both residual pointers are NULL
 *            (plain MXFP4) or both non-NULL.
 * Non-finite inputs are outside the contract (results unspecified).
 */
rfq_status rfq_quantize_act(const void *x, rfq_dtype x_dtype, int64_t M, int64_t K,
                            uint8_t *q_codes, uint8_t *q_scales,
                            uint8_t *r_codes, uint8_t *r_scales,
                            void *hip_stream);

/*
 * Weight quantizer Q(Y) (Eq. 8), primary code only.  The weight is given as
 * W[N][K] (the transpose of the paper's Y, K contiguous), blocks along K.
 *   w        [N][K] row-major, element type w_dtype; 16-byte aligned.
 *   w_codes  [N][K/2] bytes, 16-byte aligned.    w_scales [N][K/32] bytes.
 */
rfq_status rfq_quantize_weight(const void *w, rfq_dtype w_dtype, int64_t N, int64_t K,
                               uint8_t *w_codes, uint8_t *w_scales,
                               void *hip_stream);

/*
 * RFQ product, Eq. (11) / Algorithm 1:
 *   Z[m][n] = sum_k deq(q)[m][k] * deq(w)[n][k]  +  sum_k deq(r)[m][k] * deq(w)[n][k]
 * with every block of the residual taken (fallback indicator phi = 1), or
 * without the second sum (phi = 0, plain MXFP4) when r_codes and r_scales are
 * both NULL.  Products of codes are exact; accumulation is in fp32 in an
 * unspecified order.  The output is fp32, or bf16 rounded to nearest even.
 *   q_codes, r_codes, w_codes: 16-byte aligned, layouts as above.
 *   z        [M][N] row-major, z_dtype; 16-byte aligned.
 */
rfq_status rfq_gemm(const uint8_t *q_codes, const uint8_t *q_scales,
                    const uint8_t *r_codes, const uint8_t *r_scales,
                    const uint8_t *w_codes, const uint8_t *w_scales,
                    int64_t M, int64_t N, int64_t K,
                    void *z, rfq_dtype z_dtype, void *hip_stream);

/*
 * The RFQ product of rfq_gemm with the reduction over K split across
 * several workgroups per output tile where that is faster: products with few
 * output tiles (at most 128 tiles of 128 x 128, or at most 192 with
 * K >= 8192) and at least 33 activation rows (24 with K >= 12288, 17 with
 * K >= 8192 where the few-row product's grid holds between one and two
 * workgroups per CU, e.g. N = 5120), e.g. an MLP down projection for a few
 * dozen to a few hundred tokens; not for 33-64 rows with 11264 <= N < 16384,
 * where rfq_gemm's few-row product is faster.  Where the few-row grid's last
 * round of workgroups is at most a quarter full (e.g. N = 5120) with up to
 * 16 rows and K >= 12288, the few-row product itself splits K in three
 * parts.
 * Each part of K writes its fp32 partial sums to the workspace; one pass then
 * adds the parts in a fixed order and rounds to z_dtype, so the result is
 * deterministic but its fp32 summation order differs from rfq_gemm's (both
 * agree within the product's rounding).  Where the shape does not split, or
 * workspace_bytes is below rfq_gemm_workspace_bytes(M, N, K), it is rfq_gemm.
 *   workspace: device memory owned by the caller, 16-byte aligned, not read
 *            before it is written; NULL only with workspace_bytes == 0.
 *   workspace_bytes: its size, >= 0.
 * Other arguments and errors as rfq_gemm.  Calls that share a workspace must
 * be ordered (one stream, or events).  Asynchronous on hip_stream.
 */
rfq_status rfq_gemm_split(const uint8_t *q_codes, const uint8_t *q_scales,
                          const uint8_t *r_codes, const uint8_t *r_scales,
                          const uint8_t *w_codes, const uint8_t *w_scales,
                          int64_t M, int64_t N, int64_t K,
                          void *z, rfq_dtype z_dtype, void *workspace,
                          int64_t workspace_bytes, void *hip_stream);

/*
 * rfq_gemm_split without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The split product's partials go to a
 * static device array of 32 MiB held by every GPU the library runs on until
 * the process ends; no call allocates, frees or calls an allocating routine.
 * Results are those of rfq_gemm_split with a large enough workspace.  Calls
 * that overlap on one GPU (other streams or host threads) share the array
 * and race; order them (one stream, or events).
 * Arguments as rfq_gemm.  Errors as rfq_gemm, plus RFQ_ERR_SHAPE where the
 * split would need more than the 32 MiB (rfq_gemm_workspace_bytes above
 * 33554432; the library's split plan stays within it) and RFQ_ERR_DEVICE if
 * the array's device address cannot be obtained.  Asynchronous on hip_stream.
 */
rfq_status rfq_gemm_split_noalloc(const uint8_t *q_codes, const uint8_t *q_scales,
                                  const uint8_t *r_codes, const uint8_t *r_scales,
                                  const uint8_t *w_codes, const uint8_t *w_scales,
                                  int64_t M, int64_t N, int64_t K,
                                  void *z, rfq_dtype z_dtype, void *hip_stream);

/*
 * Workspace rfq_gemm_split uses for this shape: parts * M * N * 4 bytes for
 * the fp32 partials (at most 32 MiB), or 0 where it does not split (up to
 * 32 rows, 23 with K >= 12288, except the uneven few-row grids above;
 * 33-64 rows with 11264 <= N < 16384, K not a multiple of 512,
 * more than 128 tiles of 128 x 128 with K < 8192 or more than 192, or sizes
 * that rfq_gemm rejects).  Assumes 16-byte aligned scale tensors (with others the
 * product runs unsplit).  Host-only; no device call.
 */
int64_t rfq_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * Dequantization, one term of Eq. (12): out[r][k] = value(code) * 2^(scale-127),
 * exact in fp32 (scale byte 0xFF gives NaN).
 *   codes [rows][K/2] 16-byte aligned; scales [rows][K/32]; out [rows][K]
 *   fp32, 16-byte aligned.
 */
rfq_status rfq_dequant(const uint8_t *codes, const uint8_t *scales, int64_t rows,
                       int64_t K, float *out, void *hip_stream);

/*
 * SwiGLU intermediate of a gated MLP followed by the RFQ quantizer: h =
 * bf16(silu(g) * u) with silu(g) = g / (1 + exp(-g)) in fp32 arithmetic,
 * then Q(h) and Q(h - deq Q(h)) exactly as rfq_quantize_act on bf16 input.
 * This chains two RFQ products (gate/up, then down) without a bf16 round trip
 * of h through memory.
 *   g, u     [M][Nh] row-major, element type dt; 16-byte aligned.  Nh is
 *            the K of the following product (multiple of 32).
 *   q_codes, q_scales, r_codes, r_scales: as rfq_quantize_act with K = Nh (residual pair optional).
 *   h_out    [M][Nh] bf16, 16-byte aligned, or NULL; when given, h is also
 *            written (for inspection).
 */
rfq_status rfq_swiglu_quantize_act(const void *g, const void *u, rfq_dtype dt,
                                   int64_t M, int64_t Nh,
                                   uint8_t *q_codes, uint8_t *q_scales,
                                   uint8_t *r_codes, uint8_t *r_scales,
                                   void *h_out, void *hip_stream);

/*
 * RFQ product with the fallback indicator of Algorithm 1 / Eq. (11) given as
 * a map: Z = sum_r Xq Yq + sum_r phi(p, r) Xr Yq, where phi(p, r) is one byte
 * per activation tile of 64 rows (p = m / 64) by 256 reduction columns
 * (r = k / 256); a nonzero byte includes the tile's residual term.  Tiles
 * with phi = 0 skip the residual matrix-core work.
 *   phi      [ceil(M/64)][ceil(K/256)] bytes, device memory, any alignment.
 *            NULL means phi = 1 everywhere (then, and when r_codes is NULL,
 *            the call is exactly rfq_gemm).
 *   Other arguments, layouts and errors as rfq_gemm; with a map, K must not
 *   exceed 2^20 (RFQ_ERR_SHAPE).
 */
rfq_status rfq_gemm_phi(const uint8_t *q_codes, const uint8_t *q_scales,
                        const uint8_t *r_codes, const uint8_t *r_scales,
                        const uint8_t *w_codes, const uint8_t *w_scales, const uint8_t *phi,
                        int64_t M, int64_t N, int64_t K, void *z, rfq_dtype z_dtype,
                        void *hip_stream);

/*
 * Builds a fallback-indicator map for rfq_gemm_phi over the same tiles
 * (64 rows by 256 reduction columns; ragged edge tiles cover what exists).
 *   rule RFQ_PHI_RESIDUAL_NONZERO: phi = 1 where some residual code of the
 *        tile has a nonzero magnitude; the other tiles' residual terms are
 *        exactly zero, so the product equals phi = 1 (up to the sign of a zero
 *        output).  Reads r_codes [M][K/2] (16-byte aligned); q_scales unused.
 *   rule RFQ_PHI_SCALE_AT_LEAST: phi = 1 where some primary scale byte of the
 *        tile is >= threshold (a large block maximum marks an outlier);
 *        reads q_scales [M][K/32]; r_codes unused.
 *   phi  [ceil(M/64)][ceil(K/256)] bytes (0 or 1), written.
 * Errors: RFQ_ERR_SHAPE for an unknown rule or the K conditions of
 * rfq_quantize_act; RFQ_ERR_NULL for a missing input the rule reads or phi.
 */
rfq_status rfq_fallback_map(const uint8_t *r_codes, const uint8_t *q_scales, int64_t M,
                            int64_t K, int rule, int threshold, uint8_t *phi,
                            void *hip_stream);

/*
 * Gate/up product of a gated MLP with the SwiGLU intermediate and its RFQ
 * quantization fused into the product's epilogue: Z = RFQ product (Eq. 11)
 * of the activation codes with interleaved gate/up weights, then, per row and
 * per 32 hidden units, g and u are the bf16 roundings of Z's gate and up
 * columns, h = bf16(silu(g) * u) as in rfq_swiglu_quantize_act, and Q(h),
 * Q(h - deq Q(h)) (Eq. 8-10) are written.  Neither Z nor g and u reach
 * memory.  For M > 128 the codes are bit-identical to rfq_gemm with bf16 Z
 * (gate and up columns) followed by rfq_swiglu_quantize_act, which then runs
 * the same product kernel (with 256- or 128-wide tiles, which accumulate
 * each output in the same order); with up to 128 rows rfq_gemm runs its few-row
 * kernel, whose fp32 summation order differs, so g or u, and through them h
 * and its codes, can differ where a bf16 rounding boundary lies between the
 * two sums (both stay within the product's tolerance).
 *   q_codes, q_scales, r_codes, r_scales: activation codes as for rfq_gemm
 *            ([M][K/2], [M][K/32]; residual pair optional, NULL gives phi = 0).
 *   wgu_codes [2 Nh][K/2], wgu_scales [2 Nh][K/32]: quantized weights whose
 *            rows are gate and up rows interleaved in groups of 32: rows
 *            64 j .. 64 j + 31 are gate rows 32 j .., rows 64 j + 32 ..
 *            64 j + 63 are up rows 32 j .. (weights are quantized row by row,
 *            so interleaving the fp32 weights or their codes is the same).
 *   M, Nh, K: Nh a multiple of 32 (it is the K of the down product); K a
 *            multiple of 512; every code tensor below 4 GiB.
 *   hq_codes [M][Nh/2], hq_scales [M][Nh/32], hr_codes, hr_scales: codes of
 *            h as rfq_quantize_act with K = Nh (residual pair optional).
 *   h_out    [M][Nh] bf16, or NULL; when given, h is also written.
 * Alignment: all code tensors, the activation and weight scale tensors and
 * h_out 16-byte aligned.  Errors: RFQ_ERR_SHAPE for the shape conditions
 * above, otherwise as rfq_gemm.  Asynchronous on hip_stream.
 */
rfq_status rfq_gemm_swiglu_quantize(const uint8_t *q_codes, const uint8_t *q_scales,
                                    const uint8_t *r_codes, const uint8_t *r_scales,
                                    const uint8_t *wgu_codes, const uint8_t *wgu_scales,
                                    int64_t M, int64_t Nh, int64_t K,
                                    uint8_t *hq_codes, uint8_t *hq_scales,
                                    uint8_t *hr_codes, uint8_t *hr_scales,
                                    void *h_out, void *hip_stream);

/*
 * Streaming form of the RFQ product (Algorithm 1 with the quantization of the
 * activation tile inside the product loop; Eq. 8-11): Z = (deq q + deq r)
 * deq(w)^T where q, r are the primary and residual MXFP4 codes of X exactly
 * as rfq_quantize_act would write them, but formed block by block in
 * registers right before the products that use them - neither the residual
 * nor any activation code is written to memory.  Meant for few activation
 * rows (decode): each 16-row slice of W re-quantizes the activations it
 * multiplies, so the quantization is repeated N/16 times.
 *   x        [M][K] row-major, x_dtype (bf16 or fp32); 16-byte aligned.
 *   residual nonzero: primary and residual terms (phi = 1); zero: primary
 *            only (plain MXFP4, phi = 0).
 *   w_codes  [N][K/2], w_scales [N][K/32]: rfq_quantize_weight output;
 *            both 16-byte aligned.
 *   M, N, K: K a multiple of 512; M at most 1048560; N at most 268435440
 *            (2^24 - 1 column slices of 16); X and the weight codes below
 *            2 GiB each.
 *   z        [M][N] row-major, z_dtype; 16-byte aligned.
 * For M <= 64, and for M <= 128 with N <= 12160, the result is
 * bit-identical to rfq_quantize_act followed by rfq_gemm (which multiplies
 * such few rows with its few-row kernel, in the same accumulation order);
 * otherwise it agrees within the product's rounding (fp32 accumulation in an
 * unspecified order).  Errors: RFQ_ERR_SHAPE for the shape conditions above,
 * otherwise as rfq_gemm.  Asynchronous on hip_stream.
 */
rfq_status rfq_gemm_stream(const void *x, rfq_dtype x_dtype, int residual,
                           const uint8_t *w_codes, const uint8_t *w_scales,
                           int64_t M, int64_t N, int64_t K,
                           void *z, rfq_dtype z_dtype, void *hip_stream);

/*
 * HiF4 form of the path (Sec. 3.3, Eq. 5-6).  A block is 64 consecutive
 * elements of a row along K (K a positive multiple of 64, else
 * RFQ_ERR_SHAPE).  Per block one uint32 metadata word:
 *   bits 0-7   E6M2 macro scale byte E << 2 | M: S = 2^(E-48) (1 + M/4) (Eq. 5);
 *   bits 8-15  E1_8: bit g is the micro-exponent of elements 8g .. 8g+7;
 *   bits 16-31 E1_16: bit j is the micro-exponent of elements 4j .. 4j+3.
 * Per element a 4-bit S1P2 code sign << 3 | k (magnitude k/4, k = 0..7),
 * two per byte, element 2j in the low nibble of byte j.  Element i of a
 * block is V_i = S 2^(E1_8[i/8] + E1_16[i/4]) (-1)^sign k/4 (Eq. 6).
 * Layouts: codes [rows][K/2] bytes, meta [rows][K/64] uint32, row-major.
 *
 * The paper defines the decode, not the encoder.  This library encodes a
 * block as follows: S is the smallest E6M2 value with 7 S >= the block's
 * largest magnitude (byte 255 beyond 7 times the largest value, where
 * elements saturate); a 4-element group needs the smallest e in {0, 1, 2}
 * with 1.75 2^e S >= its largest magnitude; E1_8 of an 8-element group is 1
 * when one of its two 4-element groups needs 2, and E1_16 = max(e - E1_8, 0);
 * k = |x| / (S 2^(E1_8 + E1_16) / 4) rounded to nearest, ties to even, at most
 * 7; the sign is kept, also for a zero.
 */

/*
 * HiF4 RFQ quantizer: primary HiF4 code of x and, when r_codes and r_meta are
 * given, the HiF4 code of the residual x - deq(primary) (Eq. 8-10 with HiF4
 * codes); the residual is exact in fp32 and never written to memory.
 * Without the residual pair this is the weight quantizer.
 *   x        [rows][K] row-major, x_dtype; 16-byte aligned.
 *   q_codes  [rows][K/2], q_meta [rows][K/64]; 4-byte aligned.
 *   r_codes, r_meta: the same shapes, or both NULL.
 * Non-finite inputs are outside the contract.  At most about 2^31 blocks
 * (rows * K / 64) per call.
 */
rfq_status rfq_hif4_quantize(const void *x, rfq_dtype x_dtype, int64_t rows, int64_t K,
                             uint8_t *q_codes, uint32_t *q_meta,
                             uint8_t *r_codes, uint32_t *r_meta, void *hip_stream);

/*
 * HiF4 dequantization (Eq. 6): out[r][k] = V of the code, exact in fp32 and
 * in bf16 (every HiF4 value has at most 6 significant bits and an exponent
 * in [-52, 19]).  The bf16 form is the weight operand of rfq_hif4_gemm_wbf16.
 *   codes [rows][K/2], meta [rows][K/64] (4-byte aligned); out [rows][K] of
 *   out_dtype (RFQ_F32 or RFQ_BF16), 16-byte aligned.
 */
rfq_status rfq_hif4_dequant(const uint8_t *codes, const uint32_t *meta, int64_t rows, int64_t K,
                            void *out, rfq_dtype out_dtype, void *hip_stream);

/*
 * HiF4 RFQ product (Eq. 11 with HiF4 codes, phi = 1; phi = 0 when r_codes and
 * r_meta are both NULL):
 *   Z[m][n] = sum_k V_q[m][k] V_w[n][k] + sum_k V_r[m][k] V_w[n][k].
 * Every product of two HiF4 values is exact; accumulation is fp32 in an
 * unspecified order.  The output is fp32, or bf16 rounded to nearest even.
 *   q_codes, r_codes, w_codes: [M][K/2], [M][K/2], [N][K/2], 16-byte aligned.
 *   q_meta, r_meta, w_meta: [M][K/64], [M][K/64], [N][K/64], 4-byte aligned.
 *   z        [M][N] row-major, z_dtype; 16-byte aligned.
 *   M, N below 2^31 and ceil(M/128) ceil(N/256) < 2^23.
 */
rfq_status rfq_hif4_gemm(const uint8_t *q_codes, const uint32_t *q_meta,
                         const uint8_t *r_codes, const uint32_t *r_meta,
                         const uint8_t *w_codes, const uint32_t *w_meta,
                         int64_t M, int64_t N, int64_t K,
                         void *z, rfq_dtype z_dtype, void *hip_stream);

/*
 * HiF4 RFQ product with the weights given as bf16 values: Z = sum_k V_q w +
 * sum_k V_r w (phi = 0 without the residual pair).  Meant for weights that are
 * decoded once (rfq_hif4_dequant with bf16 output): constant weights at
 * inference, or weights re-quantized once per training step.  The product then
 * decodes only the activation codes.  Any bf16 w is accepted; every product
 * of a HiF4 value and a bf16 value is exact in fp32.  With w the bf16 decode
 * of HiF4 weight codes the result is bit-identical to rfq_hif4_gemm on those
 * codes.
 *   q_codes, q_meta, r_codes, r_meta: as rfq_hif4_gemm.
 *   w_bf16   [N][K] bf16, 16-byte aligned.
 *   z        [M][N] row-major, z_dtype; 16-byte aligned.
 * Shape limits and errors as rfq_hif4_gemm.
 */
rfq_status rfq_hif4_gemm_wbf16(const uint8_t *q_codes, const uint32_t *q_meta,
                               const uint8_t *r_codes, const uint32_t *r_meta,
                               const void *w_bf16, int64_t M, int64_t N, int64_t K,
                               void *z, rfq_dtype z_dtype, void *hip_stream);

/*
 * rfq_hif4_gemm with the reduction over K split across several workgroups per
 * output tile where that is faster: products whose 128 x 256 tiles number
 * fewer than 256 and whose 128 x 128 tiles number at most 128 (up to a few
 * hundred activation rows against a narrow weight, e.g. an MLP down
 * projection), with K at least 512, from 49 activation rows (where
 * N <= 4096 from 24 with K >= 12288, from 40 below); with fewer rows, where
 * the few-row product's grid leaves its last round of workgroups partly
 * empty (e.g. N = 5120), that product split over K in 2 to 4 parts.  From
 * 1024 rows, where K is not split, the workspace instead receives the
 * weights decoded to bf16 (N * K * 2 bytes, at most 1 GiB) and the product
 * of rfq_hif4_gemm_wbf16 runs on them: the bits of rfq_hif4_gemm, without
 * decoding W again for every 128 rows.
 * Each part of K writes its fp32 partial
 * sums to the workspace; one pass then adds the parts in a fixed order and
 * rounds to z_dtype, so the result is deterministic but its fp32 summation
 * order differs from rfq_hif4_gemm's (both agree within the product's
 * rounding).  Where the shape does not split, or workspace_bytes is below
 * rfq_hif4_gemm_workspace_bytes(M, N, K), it is rfq_hif4_gemm.
 *   workspace: device memory owned by the caller, 16-byte aligned, not read
 *            before it is written; NULL only with workspace_bytes == 0.
 *   workspace_bytes: its size, >= 0.
 * Other arguments, shape limits and errors as rfq_hif4_gemm.  Calls that
 * share a workspace must be ordered (one stream, or events).  Asynchronous
 * on hip_stream.
 */
rfq_status rfq_hif4_gemm_split(const uint8_t *q_codes, const uint32_t *q_meta,
                               const uint8_t *r_codes, const uint32_t *r_meta,
                               const uint8_t *w_codes, const uint32_t *w_meta,
                               int64_t M, int64_t N, int64_t K,
                               void *z, rfq_dtype z_dtype, void *workspace,
                               int64_t workspace_bytes, void *hip_stream);

/*
 * Workspace rfq_hif4_gemm_split uses for this shape: parts * M * N * 4 bytes
 * for the fp32 partials (at most 16 MiB), N * K * 2 bytes where it decodes
 * the weights into it (at most 1 GiB), or 0 where it does neither.
 * Host-only; no device call.
 */
int64_t rfq_hif4_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * Measurement support, not a step of the method: the sustained rate of the
 * FP4 matrix cores that the product (Eq. 11) runs on, without memory
 * traffic.  256 workgroups of 8 waves (one per CU of the MI355X, two waves
 * per SIMD); each wave holds two activation and four weight fragments of
 * E2M1 codes in registers and issues 8 * iters MFMAs
 * (v_mfma_scale_f32_32x32x64_f8f6f4, 2 * 32 * 32 * 64 flops each, scale 1.0)
 * into eight 32 x 32 fp32 accumulators.  The operand bits are random
 * (random_operands nonzero; fixed per work item) or the constant code 0x2
 * (1.0), since the clock the chip holds depends on them.  One launch is
 * 256 * 8 * 8 * iters * 131072 flops.
 *   iters    1 .. 2^24.
 *   sink     [256 * 512] fp32, 16-byte aligned, device memory owned by the
 *            caller: work item t writes the sum of its accumulator elements
 *            to sink[t] (with constant operands 8192 * iters, exact up to
 *            iters = 2048).
 * Errors: RFQ_ERR_SHAPE for iters out of range, RFQ_ERR_NULL, RFQ_ERR_ALIGN,
 * RFQ_ERR_DEVICE, RFQ_ERR_LAUNCH.  Asynchronous on hip_stream.
 */
rfq_status rfq_mfma_fp4_loop(int64_t iters, int random_operands, float *sink, void *hip_stream);

/*
 * Measurement support, not a step of the method: rfq_mfma_fp4_loop on the
 * bf16 matrix cores that the HiF4 product (Sec. 3.3) runs on.  Same grid,
 * wave layout, accumulator pattern, arguments, sink and errors; each wave
 * issues 8 * iters v_mfma_f32_32x32x16_bf16 (2 * 32 * 32 * 16 flops each),
 * so one launch is 256 * 8 * 8 * iters * 32768 flops.  Random operands are
 * finite bf16 values in [0.5, 2) of either sign (random sign and mantissa,
 * fixed per work item); constant operands are 1.0, which gives
 * sink[t] = 2048 * iters (exact up to iters = 8192).
 */
rfq_status rfq_mfma_bf16_loop(int64_t iters, int random_operands, float *sink, void *hip_stream);

/* Static, never-NULL description of a status code. */
const char *rfq_status_str(rfq_status s);

/* Version of this interface; changes whenever a signature or layout changes. */
int rfq_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RFQ_H */
