/*
 * focus.h -- C ABI of the FOCUS scale-learning hot path for MI355X (gfx950).
 *
 * FOCUS (arXiv 2608.01847) learns FP4 block scales by gradient descent. For every linear layer of
 * a block being calibrated, one step of the method
 *   1. fake-quantises the weights with the learned scales (Sec. 3.2 Eq. 4, Sec. 3.3 Eq. 6-7,
 *      Sec. 3.4 Eq. 8):  S_dq = Q_fmt(S_fp),  S_q = S_dq * c,  W_hat = Q_E2M1(W / S_q) * S_dq
 *   2. fake-quantises the activations with dynamic absmax scales (Sec. 3.2, Sec. 4.1)
 *   3. runs the reconstruction GEMM Y_hat = X_hat W_hat^T against the full-precision output Y_ref
 *      with the loss L = sum((Y_hat - Y_ref)^2) / (M N)
 *   4. back-propagates with the straight-through estimator (Sec. 3.2) to the scales S_fp and the
 *      Coupled-Relaxation / Dual-Granularity coefficients c (Eq. 6-8).
 * Only the FP4 codes and the dequantisation scales are exported (Fig. 3(d)).
 *
 * Conventions for every call:
 *   - All tensor pointers are DEVICE pointers owned by the caller, row-major and contiguous. The
 *     library allocates nothing; scratch memory comes from the caller's workspace `ws`.
 *   - Blocks and sub-blocks run along K, the contiguous (input-feature / reduction) dimension.
 *     MXFP4: block B = 32, one E8M0 scale byte per block. NVFP4: block B = 16, one E4M3 byte per
 *     block plus one fp32 tensor scale alpha.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL is the null stream). Argument
 *     checks happen on the host before anything is launched; a failed check returns an error and
 *     launches nothing. No call synchronises except focus_check_flags.
 *   - A workspace must be at least focus_workspace_size() bytes, 256-byte aligned, and zero-filled
 *     once before its first use (its first 256 bytes hold the sticky domain-error flag that
 *     focus_check_flags reads and clears). Calls that overlap on one workspace race.
 *   - Sizes of 0 are valid no-ops. Each dimension must be below 2^31 and rows*K below 2^46.
 *   - Tensor pointers must be 16-byte aligned (they are read and written with vector accesses);
 *     a misaligned pointer is rejected with FOCUS_ERR_SHAPE.
 *   - Results are deterministic: every floating-point reduction has a fixed order and no kernel of
 *     the scale-learning step uses atomics. The only atomics in the library are integer additions
 *     to focus_kl_top's radix-select histogram in LDS, whose counts do not depend on their order.
 */
#ifndef FOCUS_H
#define FOCUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FOCUS_OK = 0,
    FOCUS_ERR_NULL = 1,      /* a required pointer is NULL */
    FOCUS_ERR_SHAPE = 2,     /* bad sizes (negative, too large, K not a multiple of the block size)
                                or a tensor pointer that is not 16-byte aligned */
    FOCUS_ERR_DTYPE = 3,     /* unknown dtype or unsupported dtype combination */
    FOCUS_ERR_CONFIG = 4,    /* bad focus_qconfig (format, sub_block, ste_clip, scale_layout, e8m0_rounding) */
    FOCUS_ERR_WORKSPACE = 5, /* workspace NULL, misaligned or smaller than focus_workspace_size() */
    FOCUS_ERR_DOMAIN = 6,    /* focus_check_flags: a kernel met a NaN scale or a c <= 0 / non-finite */
    FOCUS_ERR_HIP = 7,       /* the HIP runtime reported an error */
    FOCUS_ERR_SCRATCH = 8    /* focus_recon_gemm_fwd_mxfp4_noalloc: the sizes need more than its fixed scratch */
} focus_status;

typedef enum { FOCUS_MXFP4 = 0, FOCUS_NVFP4 = 1 } focus_format;
typedef enum { FOCUS_F32 = 0, FOCUS_BF16 = 1 } focus_dtype;

/* Quantisation configuration.
 *   format    : focus_format.
 *   sub_block : elements per coefficient c (Sec. 3.4 Eq. 8); one of 2, 4, 8, 16, 32 and a divisor
 *               of the block size. sub_block == block size is Coupled-Relaxation Scaling with one
 *               coefficient per block (Sec. 3.3 Eq. 6-7); the paper's default is 8.
 *   ste_clip  : 1 -> the straight-through derivative of Q_E2M1 is the clamp's, m = [|u| <= 6];
 *               0 -> m = 1 everywhere.
 *   scale_layout : layout of the scale bytes that focus_fakequant_fwd and focus_export_packed write:
 *               FOCUS_SCALES_ROW_MAJOR (0) [rows][K/B], the deployable layout; FOCUS_SCALES_BLOCK_MAJOR
 *               (1) [K/B][rows], the layout focus_recon_gemm_fwd_mxfp4 reads. Other calls ignore it.
 *   e8m0_rounding : MXFP4 only (NVFP4 requires 0). FOCUS_E8M0_CEIL (0): Q_E8M0 rounds up, 2^e the
 *               smallest power of two >= s (Sec. 3.1 Eq. 3, "ceiling in practice"); activation blocks use
 *               s = fl32(amax / 6) and focus_scales_init sets S_fp = fl32(amax / 6).
 *               FOCUS_E8M0_FLOOR (1): the OCP MX rule, e = floor(log2 s) clamped to [-127, 127];
 *               activation blocks take e = floor(log2 amax) - 2 (2 = exponent of E2M1's largest
 *               value, elements above 6 S saturate) and focus_scales_init sets S_fp = fl32(amax / 4),
 *               whose floor exponent is that same OCP exponent. The straight-through derivative of
 *               Q_E8M0 is 1 in both modes.
 *   code_layout : layout of the packed codes that focus_fakequant_fwd, focus_export_packed and
 *               focus_fakequant_weights write: FOCUS_CODES_ROW_MAJOR (0) [rows][K/2], the deployable
 *               layout and that of the MXFP4 GEMMs' X operand; FOCUS_CODES_K_SLAB (1) [K/128][rows][64],
 *               slab s holding every row's 64 bytes of k = 128 s .. 128 s + 127 (a GEMM step's tile of
 *               the operand is then one contiguous run), the layout of focus_recon_gemm_fwd_mxfp4's W
 *               operand; it needs K % 128 == 0 wherever codes are written. Byte order within a row's
 *               64 bytes is the row-major one. Other calls ignore it.
 * A zero-initialised trailing field keeps the defaults (row-major codes). */
typedef enum { FOCUS_SCALES_ROW_MAJOR = 0, FOCUS_SCALES_BLOCK_MAJOR = 1 } focus_scale_layout;
typedef enum { FOCUS_E8M0_CEIL = 0, FOCUS_E8M0_FLOOR = 1 } focus_e8m0_rounding;
typedef enum { FOCUS_CODES_ROW_MAJOR = 0, FOCUS_CODES_K_SLAB = 1 } focus_code_layout;
typedef struct {
    int32_t format;
    int32_t sub_block;
    int32_t ste_clip;
    int32_t scale_layout;
    int32_t e8m0_rounding;
    int32_t code_layout;
} focus_qconfig;

typedef void *focus_stream; /* a hipStream_t */

/* Which call a workspace is sized for (first argument of focus_workspace_size). */
typedef enum {
    FOCUS_CALL_SCALES_INIT = 0,
    FOCUS_CALL_FAKEQUANT_FWD = 1,
    FOCUS_CALL_FAKEQUANT_BWD = 2,
    FOCUS_CALL_RECON_GEMM_FWD = 3,
    FOCUS_CALL_RECON_GEMM_BWD = 4,
    FOCUS_CALL_EXPORT_PACKED = 5,
    FOCUS_CALL_ADAMW = 6,
    FOCUS_CALL_RECON_GEMM_DX = 7,
    FOCUS_CALL_FAKEQUANT_ACT_BWD = 8,
    FOCUS_CALL_KL_TOP = 9,
    FOCUS_CALL_FAKEQUANT_WEIGHTS = 10
} focus_call;

/* Workspace bytes a call needs for the given sizes (M = tokens, N = rows / out features,
 * K = in features; unused sizes are ignored). Host-only; returns 0 for invalid arguments. */
size_t focus_workspace_size(int call, const focus_qconfig *q, int64_t M, int64_t N, int64_t K);

/* Absmax initialisation of the learnable scales (Sec. 3.2 "initialized via absmax", Eq. 2-3).
 *   W [N][K] (w_dtype) frozen weights.
 *   MXFP4: s_fp[n][i] = fl32(max_{block i}|w| / 6)              ([N][K/32] fp32)
 *   NVFP4: alpha = fl32(max|W| / 2688) (1 if W is all zero), written to *alpha_out (device fp32);
 *          s_fp[n][i] = Delta_fp = fl32(max_{block i}|w| / fl32(alpha * 6))   ([N][K/16] fp32)
 *   c [N][K/sub_block] fp32 is set to 1 (Sec. 3.3, Sec. 3.4). alpha_out may be NULL for MXFP4.
 *   With N == 0 or K == 0 nothing is launched and nothing is written (*alpha_out included). */
focus_status focus_scales_init(const focus_qconfig *q, const void *W, int w_dtype, int64_t N, int64_t K,
                               float *s_fp, float *c, float *alpha_out,
                               void *ws, size_t ws_bytes, focus_stream stream);

/* Fake quantisation forward of one tensor X [rows][K] (x_dtype) into X_hat [rows][K] (xhat_dtype).
 * Weight mode (s_fp != NULL; Eq. 4, 6-8, 1):
 *   S_dq = Q_fmt(s_fp) per block (MXFP4: 2^E8M0(s_fp), rounded up; NVFP4: fl32(alpha * Q_E4M3(s_fp))),
 *   S_q = fl32(S_dq * c) per sub-block (c == NULL means every c = 1), u = fl32(x / S_q),
 *   code = Q_E2M1(u) (nearest, ties to even, saturating at 6), x_hat = fl32(q * S_dq).
 *   NVFP4 needs `alpha` (device fp32 [1], the frozen tensor scale).
 * Activation mode (s_fp == NULL, c and alpha must be NULL): scales recomputed from X by absmax
 *   (Sec. 3.2 dynamic activation quantisation): MXFP4 S = 2^E8M0(fl32(amax/6)); NVFP4 alpha_x =
 *   fl32(max|X| / 2688) over the whole X (1 if X is all zero), S = fl32(alpha_x * Q_E4M3(fl32(amax /
 *   fl32(alpha_x * 6)))); alpha_x is written to *alpha_out_opt when it is non-NULL.
 * Optional outputs: codes_opt, packed FP4 codes (code = sign<<3 | magnitude index, the even-k code in
 *   the low nibble) in q->code_layout ([rows][K/2] or K-slabs [K/128][rows][64]; the slabs need
 *   K % 128 == 0, FOCUS_ERR_SHAPE otherwise); scale_bytes_opt in q->scale_layout (E8M0 byte e+127, or
 *   E4M3 byte).
 *   X_hat may be NULL when codes_opt is not (the packed form alone, e.g. for the MXFP4 GEMMs);
 *   X_hat and codes_opt both NULL is FOCUS_ERR_NULL. With rows == 0 nothing is read or written and
 *   X, X_hat and codes_opt may be NULL.
 * A zero dequantisation (or quantisation) scale quantises its block to signed zeros. */
focus_status focus_fakequant_fwd(const focus_qconfig *q, const void *X, int x_dtype, int64_t rows, int64_t K,
                                 const float *s_fp, const float *c, const float *alpha,
                                 void *X_hat, int xhat_dtype, uint8_t *codes_opt,
                                 uint8_t *scale_bytes_opt, float *alpha_out_opt,
                                 void *ws, size_t ws_bytes, focus_stream stream);

/* Straight-through backward of the weight fake quantisation (Sec. 3.2 STE through Eq. 6-8), given
 * G = dL/dW_hat [N][K] fp32. With u = w / S_q and m the clamp mask:
 *   grad_c[n][k]  = -(1/c^2) * sum_{j in sub-block k} G_j m_j w_j               ([N][K/sub_block])
 *   grad_s[n][i]  = f * sum_{j in block i} G_j (q_j - m_j u_j)                   ([N][K/B])
 * where f = 1 for MXFP4 (STE through Q_E8M0) and f = alpha for NVFP4 (Delta_fp, alpha frozen).
 * Outputs are fp32 and overwritten. Blocks with a zero scale get zero gradients. */
focus_status focus_fakequant_bwd(const focus_qconfig *q, const float *G, int64_t N, int64_t K,
                                 const void *W, int w_dtype, const float *s_fp, const float *c,
                                 const float *alpha, float *grad_s, float *grad_c,
                                 void *ws, size_t ws_bytes, focus_stream stream);

/* Reconstruction GEMM forward with the MSE epilogue: the forward of one scale-learning step
 * (Sec. 4.1: the fake-quantised layer is run on calibration tokens and compared with the
 * full-precision model). The loss here is the per-layer mean squared error to the full-precision
 * output Y_ref, a layer-local stand-in for the paper's end-to-end KL-Top objective (Sec. 4.1); dY is
 * the gradient the backward consumes, and focus_kl_top provides the end-to-end one.
 *   X_hat [M][K], W_hat [N][K] in op_dtype (FOCUS_BF16: bf16 MFMA with fp32 accumulation;
 *   FOCUS_F32: fp32), Y_hat = X_hat W_hat^T.
 *   Y_ref == NULL: plain GEMM, Y_hat is written to dY [M][N] (op_dtype).
 *   Y_ref != NULL ([M][N], op_dtype): D = Y_hat - Y_ref, dY = fl(2 D / (M N)) (op_dtype),
 *     *loss_out (device double) = sum(D^2) / (M N) and, if col_sq_opt != NULL, col_sq_opt[n]
 *     (device double [N]) = sum over tokens of D[t][n]^2.
 *   With M == 0 or N == 0 nothing is launched and nothing is written: dY, *loss_out and col_sq_opt
 *   keep their contents (a mean over no elements is undefined). */
focus_status focus_recon_gemm_fwd(const void *X_hat, const void *W_hat, int op_dtype,
                                  int64_t M, int64_t N, int64_t K, const void *Y_ref, void *dY,
                                  double *loss_out, double *col_sq_opt,
                                  void *ws, size_t ws_bytes, focus_stream stream);

/* Reconstruction GEMM forward from packed MXFP4 operands, with the same epilogue and outputs as
 * focus_recon_gemm_fwd (Y_ref and dY bf16; the same per-layer MSE stand-in for Sec. 4.1's KL-Top). Under MXFP4, X_hat and W_hat are exactly FP4 codes
 * times E8M0 block scales along K (Sec. 3.1, Eq. 1 and 3), so Y_hat = X_hat W_hat^T is computed from
 * that representation with the block-scaled FP4 MFMA: every product is exact and the sums are
 * accumulated in fp32, i.e. the same result as the bf16 path up to the accumulation order.
 *   X_codes [M][K/2] (FOCUS_CODES_ROW_MAJOR) and W_codes in K-slabs [K/128][N][64]
 *     (FOCUS_CODES_K_SLAB of focus_export_packed / focus_fakequant_weights / focus_fakequant_fwd):
 *     two E2M1 codes per byte, even k in the low nibble, 16-byte aligned. The weights, exported once
 *     per step, come in the layout that gives each GEMM step one contiguous run of W; the activation
 *     codes stay row-major, the layout the backward reads fastest (token-major tiles);
 *   X_scales [K/32][M], W_scales [K/32][N]: E8M0 bytes (e + 127) in the block-major layout
 *     (FOCUS_SCALES_BLOCK_MAJOR of focus_fakequant_fwd / focus_export_packed), 4-byte aligned.
 *   Requires K % 128 == 0, M % 4 == 0 and N % 8 == 0 (FOCUS_ERR_SHAPE otherwise). The workspace is
 *   that of FOCUS_CALL_RECON_GEMM_FWD. */
focus_status focus_recon_gemm_fwd_mxfp4(const uint8_t *X_codes, const uint8_t *X_scales, const uint8_t *W_codes,
                                        const uint8_t *W_scales, int64_t M, int64_t N, int64_t K,
                                        const void *Y_ref, void *dY, double *loss_out, double *col_sq_opt,
                                        void *ws, size_t ws_bytes, focus_stream stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): focus_recon_gemm_fwd_mxfp4 without a workspace argument. Same
 * arguments, checks, kernels and results (bit for bit); the scratch the forward needs lives in a
 * fixed 32 MiB device array of the library, one per GPU, held until the process ends. The call
 * allocates and frees nothing. Sizes are limited by that array:
 *   256 + 8 * (ceil(M / 256) * N + (col_sq_opt ? 0 : N))  <=  32 MiB
 * (every layer up to N = 16,320 at 65,536 tokens); larger sizes return FOCUS_ERR_SCRATCH and launch
 * nothing. The array keeps the last call's contents, none of which a call reads before writing it.
 * Calls that overlap on one GPU (on different streams, or from different threads) race on it; calls
 * on one stream are ordered. The first call on each GPU looks up that GPU's copy of the array. */
focus_status focus_recon_gemm_fwd_mxfp4_noalloc(const uint8_t *X_codes, const uint8_t *X_scales,
                                                const uint8_t *W_codes, const uint8_t *W_scales, int64_t M, int64_t N,
                                                int64_t K, const void *Y_ref, void *dY, double *loss_out,
                                                double *col_sq_opt, focus_stream stream);

/* Reconstruction GEMM backward with the fused straight-through epilogue: the gradient of the loss
 * with respect to the block scales and the coefficients, through the straight-through estimator on
 * every non-differentiable operation (Sec. 3.2) applied to W_hat = Q_E2M1(W / (S_dq c)) S_dq
 * (Eq. 6-7, and Eq. 8 per sub-block).
 *   G = dY^T X_hat ([N][K], the reduction runs over the M tokens, fp32 accumulation) is formed
 *   tile by tile and reduced at once into grad_s [N][K/B] and grad_c [N][K/sub_block] exactly as
 *   in focus_fakequant_bwd, from W [N][K] (w_dtype), s_fp, c (NULL = ones) and alpha (NVFP4).
 *   dY [M][N] and X_hat [M][K] are in op_dtype. If G_out_opt != NULL the fp32 G is also written.
 *   Long token ranges are split across workgroups; the per-split partial gradients are summed in a
 *   fixed order. With M == 0 the gradients are zero (an empty sum) and dY, X_hat may be NULL. */
focus_status focus_recon_gemm_bwd(const focus_qconfig *q, const void *dY, const void *X_hat, int op_dtype,
                                  int64_t M, int64_t N, int64_t K,
                                  const void *W, int w_dtype, const float *s_fp, const float *c,
                                  const float *alpha, float *grad_s, float *grad_c, float *G_out_opt,
                                  void *ws, size_t ws_bytes, focus_stream stream);

/* Reconstruction GEMM backward with the fused straight-through epilogue (Sec. 3.2 STE through
 * Eq. 6-8, as focus_recon_gemm_bwd), X_hat given as packed MXFP4 (MXFP4 only: FOCUS_ERR_CONFIG for
 * NVFP4). Under MXFP4, X_hat is exactly an E2M1 code times
 * its block's E8M0 power of two (Sec. 3.1, Eq. 1 and 3); the library rebuilds the bf16 operand from
 * that representation without loss, so grad_s and grad_c are those of focus_recon_gemm_bwd on the
 * bf16 X_hat up to the fp32 accumulation order.
 *   dY [M][N] bf16; X_codes [M][K/2] (two codes per byte, even k in the low nibble) and X_scales
 *   [K/32][M] (E8M0 bytes, block-major): the codes_opt / scale_bytes_opt outputs of
 *   focus_fakequant_fwd in activation mode with FOCUS_CODES_ROW_MAJOR and FOCUS_SCALES_BLOCK_MAJOR. W,
 *   s_fp, c, grad_s, grad_c as in focus_recon_gemm_bwd. Requires M % 4 == 0 and N % 8 == 0
 *   (FOCUS_ERR_SHAPE otherwise); dY,
 *   X_codes and W 16-byte aligned, X_scales 4-byte aligned. The workspace is that of
 *   FOCUS_CALL_RECON_GEMM_BWD. A scale byte 255 (NaN, never written by the library) makes its
 *   block's values NaN. With M == 0 the gradients are zero and dY, X_codes, X_scales may be NULL. */
focus_status focus_recon_gemm_bwd_mxfp4(const focus_qconfig *q, const void *dY, const uint8_t *X_codes,
                                        const uint8_t *X_scales, int64_t M, int64_t N, int64_t K,
                                        const void *W, int w_dtype, const float *s_fp, const float *c,
                                        float *grad_s, float *grad_c, void *ws, size_t ws_bytes,
                                        focus_stream stream);

/* Export of the deployable tensor (Fig. 3(d): only FP4 codes and dequantisation scales are kept;
 * the coefficients and S_q are discarded): packed codes and scale bytes as in focus_fakequant_fwd,
 * in q->code_layout and q->scale_layout (the deployable defaults: [N][K/2] and [N][K/B]). The NVFP4
 * tensor scale is the caller's frozen alpha. */
focus_status focus_export_packed(const focus_qconfig *q, const void *W, int w_dtype, int64_t N, int64_t K,
                                 const float *s_fp, const float *c, const float *alpha,
                                 uint8_t *packed, uint8_t *scale_bytes,
                                 void *ws, size_t ws_bytes, focus_stream stream);

/* One linear layer of focus_fakequant_weights: the tensors focus_fakequant_fwd takes in weight mode. */
typedef struct {
    const void *W;          /* [rows][K] frozen weights (the call's w_dtype) */
    int64_t rows, K;
    const float *s_fp;      /* [rows][K/B] learned scales */
    const float *c;         /* [rows][K/sub_block] coefficients, or NULL (every c = 1) */
    const float *alpha;     /* NVFP4: the frozen tensor scale (device fp32 [1]); not read for MXFP4 */
    void *W_hat;            /* [rows][K] fake-quantised weights (what_dtype), or NULL */
    uint8_t *codes;         /* packed codes in q->code_layout, or NULL */
    uint8_t *scale_bytes;   /* scale bytes in q->scale_layout, or NULL */
} focus_weight_layer;

#define FOCUS_MAX_WEIGHT_LAYERS 16

/* Weight fake quantisation (Sec. 3.2 Eq. 4, Sec. 3.3 Eq. 6-7, Sec. 3.4 Eq. 8) of up to
 * FOCUS_MAX_WEIGHT_LAYERS linear layers under one q, e.g. all the linears of the decoder block being
 * calibrated. Each layer's W_hat, codes and scale bytes are bit for bit those that focus_fakequant_fwd
 * in weight mode writes for it (with W_hat NULL: those of focus_export_packed, Fig. 3(d)), in
 * q->code_layout and q->scale_layout; bf16 weights go out in one launch for the whole group, so small
 * layers cost no launch and tail latency of their own (fp32 weights, or a group of more than 2^23
 * 64 x 256 tiles: one launch per layer, same results).
 *   layers: HOST array of n_layers entries, read during the call (the tensors stay device memory
 *     owned by the caller); every layer is checked as focus_fakequant_fwd checks a weight-mode call
 *     (W_hat and codes both NULL is FOCUS_ERR_NULL), and one failed check launches nothing.
 *   n_layers: 0 .. FOCUS_MAX_WEIGHT_LAYERS (0 is a no-op; more is FOCUS_ERR_SHAPE). Layers may
 *     differ in rows and K; a layer with rows == 0 is skipped.
 *   ws: focus_workspace_size(FOCUS_CALL_FAKEQUANT_WEIGHTS, q, 0, 0, 0) bytes (the domain flag, which a
 *     NaN scale or a bad coefficient of any layer raises). */
focus_status focus_fakequant_weights(const focus_qconfig *q, int w_dtype, int what_dtype,
                                     const focus_weight_layer *layers, int n_layers,
                                     void *ws, size_t ws_bytes, focus_stream stream);

/* Input gradient of a linear layer for end-to-end chaining (Sec. 3.2: the whole quantised model is
 * trained end to end, so the gradient reaching a layer's output flows on to its input):
 *   dX_hat [M][K] = dY [M][N] * W_hat [N][K]        (op_dtype operands, fp32 accumulation)
 * dY is the gradient of the layer output (e.g. from focus_kl_top or from the next layer), W_hat the
 * fake-quantised weight of the forward. The result is the gradient of the fake-quantised input;
 * focus_fakequant_act_bwd carries it through the activation quantisation. N % 16 == 0 (N == 0
 * writes zeros; dY and W_hat may then be NULL); all pointers 16-byte aligned; ws: focus_workspace_size(FOCUS_CALL_RECON_GEMM_DX, NULL, M, N, K)
 * bytes (it holds the transposed W_hat). bf16 runs on the MFMA path where the shapes allow it. */
focus_status focus_recon_gemm_dx(const void *dY, const void *W_hat, int op_dtype, int64_t M, int64_t N, int64_t K,
                                 void *dX_hat, void *ws, size_t ws_bytes, focus_stream stream);

/* Straight-through backward of the dynamic activation fake quantisation (Sec. 3.2: STE on every
 * non-differentiable operation): dX = m * dX_hat with m = [|x / S| <= 6] (q->ste_clip = 1; m = 1 when
 * 0), the block scale S recomputed from X exactly as focus_fakequant_fwd forms it (format and
 * E8M0 rounding from q); a block whose scale is zero passes no gradient. The absmax scales pass no
 * gradient (a masked element is written as +0). X [rows][K] (x_dtype), dX_hat and dX [rows][K]
 * (g_dtype; dX may alias dX_hat). Under the
 * default rounded-up E8M0 every MXFP4 mask is 1. ws: focus_workspace_size(
 * FOCUS_CALL_FAKEQUANT_ACT_BWD, q, 0, rows, K) bytes (NVFP4 recomputes the tensor scale). */
focus_status focus_fakequant_act_bwd(const focus_qconfig *q, const void *X, int x_dtype, int64_t rows, int64_t K,
                                     const void *dX_hat, int g_dtype, void *dX, void *ws, size_t ws_bytes,
                                     focus_stream stream);

/* KL-Top objective on logits (Sec. 4.1: the end-to-end training loss, k = 1000). For each of the T
 * token rows of the teacher logits Z_teacher [T][V] (the full-precision model) and the student
 * logits Z_student [T][V] (the quantised model), with I the indices of the teacher's k largest
 * logits (ties at the k-th value taken in increasing index order; every index when k >= V):
 *   p_t = softmax(Z_teacher[row, I]),  p_s = softmax(Z_student[row, I])
 *   loss = (1/T) sum_rows sum_{i in I} p_t[i] (log p_t[i] - log p_s[i])      -> *loss_out (device fp64)
 *   dZ_student[row, i] = (p_s[i] - p_t[i]) / T for i in I, 0 elsewhere       (dtype, written in full)
 * dtype FOCUS_BF16 or FOCUS_F32 for all three arrays (element-aligned). k >= 1 (else FOCUS_ERR_CONFIG);
 * T >= 1 and 1 <= V <= 2^31 (else FOCUS_ERR_SHAPE).
 * The logits must be finite: a NaN or infinity raises the domain flag (results unspecified). ws:
 * focus_workspace_size(FOCUS_CALL_KL_TOP, NULL, T, V, 0) bytes. Deterministic (fixed-order sums). */
focus_status focus_kl_top(const void *Z_student, const void *Z_teacher, int dtype, int64_t T, int64_t V, int32_t k,
                          void *dZ_student, double *loss_out, void *ws, size_t ws_bytes, focus_stream stream);

/* AdamW hyper-parameters (Sec. 4.1: AdamW with a constant learning rate; MXFP4 uses 2e-2 for the
 * block scales and 5e-2 for the coefficients c, NVFP4 5e-3 and 1e-3).
 *   lr           : learning rate, >= 0.
 *   beta1, beta2 : decay rates of the first and second moment, in [0, 1).
 *   eps          : added to the bias-corrected root of the second moment, > 0.
 *   weight_decay : decoupled weight decay, >= 0 (the parameter is scaled by 1 - lr * weight_decay
 *                  before the moment step).
 *   log2_domain  : 0 -> the step is taken on the parameter p itself; 1 -> on theta = log2(p), with
 *                  dL/dtheta = dL/dp * p * ln 2, the moments kept for theta and p written back as
 *                  2^theta (p must be positive and finite: the scales S_fp / Delta_fp). */
typedef struct {
    float lr;
    float beta1;
    float beta2;
    float eps;
    float weight_decay;
    int32_t log2_domain;
} focus_adamw_config;

/* One AdamW step on n fp32 parameters (Loshchilov & Hutter's AdamW with bias-corrected moments), in
 * place. With g the gradient (of theta in the log2 domain) and t >= 1 the 1-based step count:
 *   theta = theta - lr*weight_decay*theta;  m = beta1*m + (1-beta1)*g;  v = beta2*v + (1-beta2)*g^2
 *   theta = theta - (lr / (1-beta1^t)) * m / (sqrt(v) / sqrt(1-beta2^t) + eps)
 * (the bias corrections are formed in double on the host and rounded to fp32 once).
 *   param, exp_avg, exp_avg_sq [n] fp32 device, read and written; grad [n] fp32 device, read.
 *   The moments start at zero (caller-owned, e.g. the same shapes as S_fp and c). All four
 *   pointers 16-byte aligned; n <= 2^40.
 * Errors: FOCUS_ERR_CONFIG (bad hyper-parameters or t < 1), FOCUS_ERR_NULL, FOCUS_ERR_SHAPE, FOCUS_ERR_WORKSPACE
 * (ws needs focus_workspace_size(FOCUS_CALL_ADAMW, ...) bytes). In the log2 domain a parameter
 * that is not positive and finite is left unchanged and raises the domain flag. */
focus_status focus_adamw_step(const focus_adamw_config *cfg, int64_t t, int64_t n, float *param, const float *grad,
                              float *exp_avg, float *exp_avg_sq, void *ws, size_t ws_bytes, focus_stream stream);

/* Synchronises `stream`, reads and clears the workspace's sticky domain flag. Returns
 * FOCUS_ERR_DOMAIN if any call on this workspace met a NaN scale or a coefficient c that is
 * <= 0 or not finite, a log2-domain AdamW step met a parameter that is not positive and
 * finite, or focus_kl_top met a logit that is not finite, since the last check (outputs of such blocks are unspecified), FOCUS_OK
 * otherwise, FOCUS_ERR_HIP on a runtime error. */
focus_status focus_check_flags(void *ws, focus_stream stream);

/* Static description of a status code. */
const char *focus_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif /* FOCUS_H */
