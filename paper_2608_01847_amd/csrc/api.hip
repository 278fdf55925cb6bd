// extern "C" entry points of libfocus: host-side argument checks, workspace layout and dispatch.
// Every check runs before anything is launched; a failed check launches nothing.
#include "../../include/focus.h"
#include "focus_device.h"
#include "gemm_common.h"
#include "internal.h"

#include <cmath>
#include <initializer_list>
#include <mutex>

using namespace focus;

namespace {

constexpr int64_t kMaxDim = (int64_t(1) << 31) - 1;
constexpr int64_t kMaxElems = int64_t(1) << 46;

focus_status check_q(const focus_qconfig *q) {
    if (!q) return FOCUS_ERR_NULL;
    if (q->format != FOCUS_MXFP4 && q->format != FOCUS_NVFP4) return FOCUS_ERR_CONFIG;
    const int B = block_of(q->format), sb = q->sub_block;
    if (!(sb == 2 || sb == 4 || sb == 8 || sb == 16 || sb == 32) || B % sb != 0) return FOCUS_ERR_CONFIG;
    if (q->ste_clip != 0 && q->ste_clip != 1) return FOCUS_ERR_CONFIG;
    if (q->scale_layout != FOCUS_SCALES_ROW_MAJOR && q->scale_layout != FOCUS_SCALES_BLOCK_MAJOR) return FOCUS_ERR_CONFIG;
    if (q->e8m0_rounding != FOCUS_E8M0_CEIL && q->e8m0_rounding != FOCUS_E8M0_FLOOR) return FOCUS_ERR_CONFIG;
    if (q->e8m0_rounding == FOCUS_E8M0_FLOOR && q->format != FOCUS_MXFP4) return FOCUS_ERR_CONFIG;
    if (q->code_layout != FOCUS_CODES_ROW_MAJOR && q->code_layout != FOCUS_CODES_K_SLAB) return FOCUS_ERR_CONFIG;
    return FOCUS_OK;
}

int slab_of(const focus_qconfig *q) { return q->code_layout == FOCUS_CODES_K_SLAB ? 1 : 0; }

// codes in K-slabs of 128 elements need whole slabs
focus_status check_code_layout(const focus_qconfig *q, const void *codes, int64_t K) {
    return codes && slab_of(q) && K % 128 != 0 ? FOCUS_ERR_SHAPE : FOCUS_OK;
}

int floor_of(const focus_qconfig *q) { return q->e8m0_rounding == FOCUS_E8M0_FLOOR ? 1 : 0; }

bool dtype_ok(int d) { return d == FOCUS_F32 || d == FOCUS_BF16; }

focus_status check_rows_k(int64_t rows, int64_t K, int B) {
    if (rows < 0 || K < 0 || rows > kMaxDim || K > kMaxDim) return FOCUS_ERR_SHAPE;
    if (K % B != 0) return FOCUS_ERR_SHAPE;
    if (rows > 0 && K > 0 && rows > kMaxElems / K) return FOCUS_ERR_SHAPE;
    return FOCUS_OK;
}

focus_status check_ws(const void *ws, size_t bytes, size_t need) {
    if (!ws || (reinterpret_cast<uintptr_t>(ws) % 256) != 0 || bytes < need) return FOCUS_ERR_WORKSPACE;
    return FOCUS_OK;
}

// tensors are read and written with 16-byte vector accesses
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool all_aligned(std::initializer_list<const void *> ps) {
    for (const void *p : ps)
        if (p && !aligned16(p)) return false;
    return true;
}

uint32_t *flag_of(void *ws) { return reinterpret_cast<uint32_t *>(ws); }
float *partials_of(void *ws) { return reinterpret_cast<float *>(reinterpret_cast<char *>(ws) + kWsHeader); }

focus_status hip_status(hipError_t e) { return e == hipSuccess ? FOCUS_OK : FOCUS_ERR_HIP; }

size_t round256(size_t b) { return (b + 255) / 256 * 256; }

// dX_hat workspace: header, the transposed W_hat [K][N] (fp32 size, the larger), then the forward's own
size_t dx_ws(int64_t M, int64_t N, int64_t K) {
    return kWsHeader + round256((size_t)N * (size_t)K * sizeof(float)) +
           std::max(plan_fwd(kF32, M, K, N).ws_bytes, plan_fwd(kBF16, M, K, N).ws_bytes);
}

size_t fwd_ws(int64_t M, int64_t N, int64_t K) {
    return std::max(plan_fwd(kF32, M, N, K).ws_bytes, plan_fwd(kBF16, M, N, K).ws_bytes);
}

size_t bwd_ws(int fmt, int sb, int64_t M, int64_t N, int64_t K) {
    size_t m = 0;
    for (int dt : {kF32, kBF16})
        for (bool g : {false, true}) m = std::max(m, plan_bwd(dt, fmt, sb, M, N, K, g).ws_bytes);
    return m;
}

#define FOCUS_TRY(x)                  \
    do {                              \
        focus_status s_ = (x);        \
        if (s_ != FOCUS_OK) return s_; \
    } while (0)

// argument checks shared by the two entry points of the forward from packed MXFP4 operands
focus_status check_fwd_mx_args(const uint8_t *X_codes, const uint8_t *X_scales, const uint8_t *W_codes,
                               const uint8_t *W_scales, int64_t M, int64_t N, int64_t K, const void *Y_ref,
                               const void *dY, const double *loss_out) {
    if (!X_codes || !X_scales || !W_codes || !W_scales || !dY) return FOCUS_ERR_NULL;
    if (Y_ref && !loss_out) return FOCUS_ERR_NULL;
    if (M < 0 || N < 0 || K < 0 || M > kMaxDim || N > kMaxDim || K > kMaxDim) return FOCUS_ERR_SHAPE;
    if (K % 128 != 0 || N % 8 != 0 || M % 4 != 0) return FOCUS_ERR_SHAPE;
    if ((M > 0 && K > kMaxElems / M) || (N > 0 && K > kMaxElems / N) || (M > 0 && N > kMaxElems / M))
        return FOCUS_ERR_SHAPE;
    if (!all_aligned({X_codes, W_codes, Y_ref, dY})) return FOCUS_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(X_scales) | reinterpret_cast<uintptr_t>(W_scales)) & 3u) return FOCUS_ERR_SHAPE;
    return FOCUS_OK;
}

// ---- fixed device scratch of the allocation-free forward ---------------------------------------
// 32 MiB per GPU: the kWsHeader bytes the workspace layout skips, ceil(M / 256) x N partial sums of
// D^2 (fp64) and, when the caller passes no col_sq, N column sums. Every hidden-2560 layer at 65,536
// tokens fits (at most 20 MB).
constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;

size_t noalloc_fwd_scratch_bytes(int64_t M, int64_t N, bool have_col_sq) {
    const size_t mtiles = (size_t)((M + kMfmaTileM - 1) / kMfmaTileM);
    return kWsHeader + (mtiles * (size_t)N + (have_col_sq ? 0 : (size_t)N)) * sizeof(double);
}

}  // namespace

// One copy per GPU, held until the process ends, shared by every call on that GPU (calls that
// overlap on one GPU race). In host code this name stands for a host-side shadow, not a device
// address: only the address scratch_address() looks up may reach a kernel or a copy.
static __device__ __align__(256) double scratch[kNoAllocScratchBytes / sizeof(double)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices];

// Device address of `scratch` on the current device, looked up once per device with that device
// current (each GPU holds its own copy at its own address).
hipError_t scratch_address(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

size_t focus_workspace_size(int call, const focus_qconfig *q, int64_t M, int64_t N, int64_t K) {
    if (call == FOCUS_CALL_ADAMW) return kWsHeader;  // the domain flag only; q may be NULL
    if (call == FOCUS_CALL_RECON_GEMM_DX) {            // q may be NULL
        if (M < 0 || N < 0 || K < 0 || M > kMaxDim || N > kMaxDim || K > kMaxDim) return 0;
        return dx_ws(M, N, K);
    }
    if (call == FOCUS_CALL_KL_TOP) {  // M = tokens; q may be NULL
        if (M < 0 || M > kMaxDim) return 0;
        return kWsHeader + round256((size_t)M * sizeof(double)) + sizeof(double);
    }
    if (check_q(q) != FOCUS_OK) return 0;
    const int B = block_of(q->format);
    switch (call) {
        case FOCUS_CALL_SCALES_INIT:
        case FOCUS_CALL_FAKEQUANT_FWD:
        case FOCUS_CALL_FAKEQUANT_ACT_BWD:
            return kWsHeader + (kAbsmaxParts + 64) * sizeof(float);  // partial maxima + tensor scale slot
        case FOCUS_CALL_FAKEQUANT_BWD:
        case FOCUS_CALL_EXPORT_PACKED:
        case FOCUS_CALL_FAKEQUANT_WEIGHTS:
            return kWsHeader;
        case FOCUS_CALL_RECON_GEMM_FWD:
            if (M < 0 || N < 0 || K < 0 || M > kMaxDim || N > kMaxDim || K > kMaxDim) return 0;
            return fwd_ws(M, N, K);
        case FOCUS_CALL_RECON_GEMM_BWD:
            if (check_rows_k(N, K, B) != FOCUS_OK || M < 0 || M > kMaxDim) return 0;
            return bwd_ws(q->format, q->sub_block, M, N, K);
        default:
            return 0;
    }
}

focus_status focus_scales_init(const focus_qconfig *q, const void *W, int w_dtype, int64_t N, int64_t K,
                               float *s_fp, float *c, float *alpha_out, void *ws, size_t ws_bytes,
                               focus_stream stream) {
    FOCUS_TRY(check_q(q));
    if (!W || !s_fp || !c) return FOCUS_ERR_NULL;
    if (q->format == FOCUS_NVFP4 && !alpha_out) return FOCUS_ERR_NULL;
    if (!dtype_ok(w_dtype)) return FOCUS_ERR_DTYPE;
    FOCUS_TRY(check_rows_k(N, K, block_of(q->format)));
    if (!all_aligned({W})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, focus_workspace_size(FOCUS_CALL_SCALES_INIT, q, 0, N, K)));
    if (N == 0 || K == 0) return FOCUS_OK;
    return hip_status(launch_scales_init(q->format, w_dtype, W, N, K, s_fp, c, q->sub_block, floor_of(q), alpha_out,
                                         partials_of(ws), (hipStream_t)stream));
}

focus_status focus_fakequant_fwd(const focus_qconfig *q, const void *X, int x_dtype, int64_t rows, int64_t K,
                                 const float *s_fp, const float *c, const float *alpha, void *X_hat,
                                 int xhat_dtype, uint8_t *codes_opt, uint8_t *scale_bytes_opt,
                                 float *alpha_out_opt, void *ws, size_t ws_bytes, focus_stream stream) {
    FOCUS_TRY(check_q(q));
    // X_hat may be left out when codes are asked for; an empty tensor (rows == 0) may come as NULL
    if (rows != 0 && (!X || (!X_hat && !codes_opt))) return FOCUS_ERR_NULL;
    const bool weight_mode = s_fp != nullptr;
    if (weight_mode && q->format == FOCUS_NVFP4 && !alpha) return FOCUS_ERR_NULL;
    if (!weight_mode && (c || alpha)) return FOCUS_ERR_CONFIG;
    if (!dtype_ok(x_dtype) || !dtype_ok(xhat_dtype)) return FOCUS_ERR_DTYPE;
    FOCUS_TRY(check_rows_k(rows, K, block_of(q->format)));
    FOCUS_TRY(check_code_layout(q, codes_opt, K));
    if (!all_aligned({X, X_hat, codes_opt})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, focus_workspace_size(FOCUS_CALL_FAKEQUANT_FWD, q, 0, rows, K)));
    if (rows == 0 || K == 0) return FOCUS_OK;
    hipStream_t st = (hipStream_t)stream;
    if (weight_mode)
        return hip_status(launch_fq_weight(q->format, x_dtype, xhat_dtype, X, rows, K, s_fp, c, q->sub_block,
                                           alpha, floor_of(q), X_hat, codes_opt, scale_bytes_opt, q->scale_layout,
                                           slab_of(q), flag_of(ws), st));
    return hip_status(launch_fq_act(q->format, x_dtype, xhat_dtype, X, rows, K, X_hat, codes_opt,
                                    scale_bytes_opt, q->scale_layout, slab_of(q), floor_of(q), alpha_out_opt, partials_of(ws),
                                    flag_of(ws), st));
}

focus_status focus_fakequant_bwd(const focus_qconfig *q, const float *G, int64_t N, int64_t K, const void *W,
                                 int w_dtype, const float *s_fp, const float *c, const float *alpha,
                                 float *grad_s, float *grad_c, void *ws, size_t ws_bytes, focus_stream stream) {
    FOCUS_TRY(check_q(q));
    if (!G || !W || !s_fp || !grad_s || !grad_c) return FOCUS_ERR_NULL;
    if (q->format == FOCUS_NVFP4 && !alpha) return FOCUS_ERR_NULL;
    if (!dtype_ok(w_dtype)) return FOCUS_ERR_DTYPE;
    FOCUS_TRY(check_rows_k(N, K, block_of(q->format)));
    if (!all_aligned({G, W})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, focus_workspace_size(FOCUS_CALL_FAKEQUANT_BWD, q, 0, N, K)));
    if (N == 0 || K == 0) return FOCUS_OK;
    return hip_status(launch_fq_bwd(q->format, w_dtype, G, N, K, W, s_fp, c, q->sub_block, alpha, q->ste_clip,
                                    floor_of(q), grad_s, grad_c, flag_of(ws), (hipStream_t)stream));
}

focus_status focus_recon_gemm_fwd(const void *X_hat, const void *W_hat, int op_dtype, int64_t M, int64_t N,
                                  int64_t K, const void *Y_ref, void *dY, double *loss_out, double *col_sq_opt,
                                  void *ws, size_t ws_bytes, focus_stream stream) {
    if (!X_hat || !W_hat || !dY) return FOCUS_ERR_NULL;
    if (Y_ref && !loss_out) return FOCUS_ERR_NULL;
    if (!dtype_ok(op_dtype)) return FOCUS_ERR_DTYPE;
    if (M < 0 || N < 0 || K < 0 || M > kMaxDim || N > kMaxDim || K > kMaxDim) return FOCUS_ERR_SHAPE;
    if (K % 16 != 0) return FOCUS_ERR_SHAPE;
    if ((M > 0 && K > kMaxElems / M) || (N > 0 && K > kMaxElems / N) || (M > 0 && N > kMaxElems / M))
        return FOCUS_ERR_SHAPE;
    if (!all_aligned({X_hat, W_hat, Y_ref, dY})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, fwd_ws(M, N, K)));
    if (M == 0 || N == 0) return FOCUS_OK;
    const FwdPlan p = plan_fwd(op_dtype, M, N, K);
    return hip_status(launch_recon_fwd(p, op_dtype, X_hat, W_hat, M, N, K, Y_ref, dY, loss_out, col_sq_opt, ws,
                                       (hipStream_t)stream));
}

focus_status focus_recon_gemm_fwd_mxfp4(const uint8_t *X_codes, const uint8_t *X_scales, const uint8_t *W_codes,
                                        const uint8_t *W_scales, int64_t M, int64_t N, int64_t K,
                                        const void *Y_ref, void *dY, double *loss_out, double *col_sq_opt,
                                        void *ws, size_t ws_bytes, focus_stream stream) {
    FOCUS_TRY(check_fwd_mx_args(X_codes, X_scales, W_codes, W_scales, M, N, K, Y_ref, dY, loss_out));
    FOCUS_TRY(check_ws(ws, ws_bytes, fwd_ws(M, N, K)));
    if (M == 0 || N == 0) return FOCUS_OK;
    if (!mfma_fwd_mx_supported(M, N, K)) return FOCUS_ERR_SHAPE;
    return hip_status(launch_recon_fwd_mx(X_codes, X_scales, W_codes, W_scales, M, N, K, Y_ref, dY, loss_out,
                                          col_sq_opt, ws, (hipStream_t)stream));
}

focus_status focus_recon_gemm_fwd_mxfp4_noalloc(const uint8_t *X_codes, const uint8_t *X_scales,
                                                const uint8_t *W_codes, const uint8_t *W_scales, int64_t M, int64_t N,
                                                int64_t K, const void *Y_ref, void *dY, double *loss_out,
                                                double *col_sq_opt, focus_stream stream) {
    FOCUS_TRY(check_fwd_mx_args(X_codes, X_scales, W_codes, W_scales, M, N, K, Y_ref, dY, loss_out));
    if (noalloc_fwd_scratch_bytes(M, N, col_sq_opt != nullptr) > kNoAllocScratchBytes) return FOCUS_ERR_SCRATCH;
    if (M == 0 || N == 0) return FOCUS_OK;
    if (!mfma_fwd_mx_supported(M, N, K)) return FOCUS_ERR_SHAPE;
    void *ptr = nullptr;
    if (scratch_address(&ptr) != hipSuccess) return FOCUS_ERR_HIP;
    // the scratch takes the place of the workspace: its first kWsHeader bytes are left unused, then
    // the per-(m-tile, column) partial sums and, without col_sq_opt, the column sums; the kernels
    // write all of it before it is read, so nothing is cleared
    return hip_status(launch_recon_fwd_mx(X_codes, X_scales, W_codes, W_scales, M, N, K, Y_ref, dY, loss_out,
                                          col_sq_opt, ptr, (hipStream_t)stream));
}

focus_status focus_recon_gemm_bwd(const focus_qconfig *q, const void *dY, const void *X_hat, int op_dtype,
                                  int64_t M, int64_t N, int64_t K, const void *W, int w_dtype,
                                  const float *s_fp, const float *c, const float *alpha, float *grad_s,
                                  float *grad_c, float *G_out_opt, void *ws, size_t ws_bytes,
                                  focus_stream stream) {
    FOCUS_TRY(check_q(q));
    // with no tokens (M == 0) the token operands are never read and may be NULL; the gradients are zero
    if ((M != 0 && (!dY || !X_hat)) || !W || !s_fp || !grad_s || !grad_c) return FOCUS_ERR_NULL;
    if (q->format == FOCUS_NVFP4 && !alpha) return FOCUS_ERR_NULL;
    if (!dtype_ok(op_dtype) || !dtype_ok(w_dtype)) return FOCUS_ERR_DTYPE;
    FOCUS_TRY(check_rows_k(N, K, block_of(q->format)));
    if (M < 0 || M > kMaxDim || (M > 0 && K > kMaxElems / M) || (M > 0 && N > kMaxElems / M))
        return FOCUS_ERR_SHAPE;
    if (!all_aligned({dY, X_hat, W, G_out_opt})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, bwd_ws(q->format, q->sub_block, M, N, K)));
    if (N == 0 || K == 0) return FOCUS_OK;
    const BwdPlan p = plan_bwd(op_dtype, q->format, q->sub_block, M, N, K, G_out_opt != nullptr);
    return hip_status(launch_recon_bwd(p, op_dtype, q->format, q->sub_block, q->ste_clip, floor_of(q), dY, X_hat, M, N, K, W,
                                       w_dtype, s_fp, c, alpha, grad_s, grad_c, G_out_opt, ws, flag_of(ws),
                                       (hipStream_t)stream));
}

focus_status focus_recon_gemm_bwd_mxfp4(const focus_qconfig *q, const void *dY, const uint8_t *X_codes,
                                        const uint8_t *X_scales, int64_t M, int64_t N, int64_t K, const void *W,
                                        int w_dtype, const float *s_fp, const float *c, float *grad_s,
                                        float *grad_c, void *ws, size_t ws_bytes, focus_stream stream) {
    FOCUS_TRY(check_q(q));
    if (q->format != FOCUS_MXFP4) return FOCUS_ERR_CONFIG;
    // with no tokens (M == 0) the token operands are never read and may be NULL; the gradients are zero
    if ((M != 0 && (!dY || !X_codes || !X_scales)) || !W || !s_fp || !grad_s || !grad_c) return FOCUS_ERR_NULL;
    if (!dtype_ok(w_dtype)) return FOCUS_ERR_DTYPE;
    FOCUS_TRY(check_rows_k(N, K, 32));
    if (M < 0 || M > kMaxDim || (M > 0 && K > kMaxElems / M) || (M > 0 && N > kMaxElems / M))
        return FOCUS_ERR_SHAPE;
    if (M % 4 != 0 || N % 8 != 0) return FOCUS_ERR_SHAPE;
    if (!all_aligned({dY, X_codes, W})) return FOCUS_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(X_scales) & 3u) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, bwd_ws(q->format, q->sub_block, M, N, K)));
    if (N == 0 || K == 0) return FOCUS_OK;
    if (!mfma_bwd_mx_supported(M, N, K)) return FOCUS_ERR_SHAPE;
    const BwdPlan p = plan_bwd(FOCUS_BF16, q->format, q->sub_block, M, N, K, false);
    return hip_status(launch_recon_bwd_mx(p, q->sub_block, q->ste_clip, floor_of(q), dY, X_codes, X_scales, M, N, K,
                                          W, w_dtype, s_fp, c, grad_s, grad_c, ws, flag_of(ws), (hipStream_t)stream));
}

focus_status focus_export_packed(const focus_qconfig *q, const void *W, int w_dtype, int64_t N, int64_t K,
                                 const float *s_fp, const float *c, const float *alpha, uint8_t *packed,
                                 uint8_t *scale_bytes, void *ws, size_t ws_bytes, focus_stream stream) {
    FOCUS_TRY(check_q(q));
    if (!W || !s_fp || !packed || !scale_bytes) return FOCUS_ERR_NULL;
    if (q->format == FOCUS_NVFP4 && !alpha) return FOCUS_ERR_NULL;
    if (!dtype_ok(w_dtype)) return FOCUS_ERR_DTYPE;
    FOCUS_TRY(check_rows_k(N, K, block_of(q->format)));
    FOCUS_TRY(check_code_layout(q, packed, K));
    if (!all_aligned({W, packed})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, focus_workspace_size(FOCUS_CALL_EXPORT_PACKED, q, 0, N, K)));
    if (N == 0 || K == 0) return FOCUS_OK;
    return hip_status(launch_fq_weight(q->format, w_dtype, w_dtype, W, N, K, s_fp, c, q->sub_block, alpha,
                                       floor_of(q), nullptr, packed, scale_bytes, q->scale_layout, slab_of(q), flag_of(ws),
                                       (hipStream_t)stream));
}

focus_status focus_fakequant_weights(const focus_qconfig *q, int w_dtype, int what_dtype,
                                     const focus_weight_layer *layers, int n_layers, void *ws, size_t ws_bytes,
                                     focus_stream stream) {
    FOCUS_TRY(check_q(q));
    if (n_layers < 0 || n_layers > FOCUS_MAX_WEIGHT_LAYERS) return FOCUS_ERR_SHAPE;
    if (n_layers > 0 && !layers) return FOCUS_ERR_NULL;
    if (!dtype_ok(w_dtype) || !dtype_ok(what_dtype)) return FOCUS_ERR_DTYPE;
    WeightLayer L[FOCUS_MAX_WEIGHT_LAYERS];
    for (int i = 0; i < n_layers; i++) {
        const focus_weight_layer &l = layers[i];
        if (l.rows != 0 && (!l.W || !l.s_fp || (!l.W_hat && !l.codes))) return FOCUS_ERR_NULL;
        if (l.rows != 0 && q->format == FOCUS_NVFP4 && !l.alpha) return FOCUS_ERR_NULL;
        FOCUS_TRY(check_rows_k(l.rows, l.K, block_of(q->format)));
        FOCUS_TRY(check_code_layout(q, l.codes, l.K));
        if (!all_aligned({l.W, l.W_hat, l.codes})) return FOCUS_ERR_SHAPE;
        L[i] = WeightLayer{l.W, l.rows, l.K, l.s_fp, l.c, q->format == FOCUS_NVFP4 ? l.alpha : nullptr,
                           l.W_hat, l.codes, l.scale_bytes};
    }
    FOCUS_TRY(check_ws(ws, ws_bytes, focus_workspace_size(FOCUS_CALL_FAKEQUANT_WEIGHTS, q, 0, 0, 0)));
    if (n_layers == 0) return FOCUS_OK;
    return hip_status(launch_fq_weight_group(q->format, w_dtype, what_dtype, L, n_layers, q->sub_block, floor_of(q),
                                             q->scale_layout, slab_of(q), flag_of(ws), (hipStream_t)stream));
}

focus_status focus_recon_gemm_dx(const void *dY, const void *W_hat, int op_dtype, int64_t M, int64_t N, int64_t K,
                                 void *dX_hat, void *ws, size_t ws_bytes, focus_stream stream) {
    if (!dX_hat || (N > 0 && (!dY || !W_hat))) return FOCUS_ERR_NULL;  // empty operands may be NULL
    if (!dtype_ok(op_dtype)) return FOCUS_ERR_DTYPE;
    if (M < 0 || N < 0 || K < 0 || M > kMaxDim || N > kMaxDim || K > kMaxDim) return FOCUS_ERR_SHAPE;
    if (N % 16 != 0) return FOCUS_ERR_SHAPE;  // the contraction runs over N
    if ((M > 0 && K > kMaxElems / M) || (N > 0 && K > kMaxElems / N) || (M > 0 && N > kMaxElems / M))
        return FOCUS_ERR_SHAPE;
    if (!all_aligned({dY, W_hat, dX_hat})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, dx_ws(M, N, K)));
    if (M == 0 || K == 0) return FOCUS_OK;
    const hipStream_t st = (hipStream_t)stream;
    char *wt = static_cast<char *>(ws) + kWsHeader;
    char *ws_fwd = wt + round256((size_t)N * (size_t)K * sizeof(float));
    if (N == 0) {  // an empty sum: dX_hat = 0
        const size_t esz = op_dtype == FOCUS_BF16 ? 2 : 4;
        return hip_status(launch_zero_fill(dX_hat, (size_t)M * (size_t)K * esz, st));
    }
    hipError_t e = launch_transpose(op_dtype, W_hat, N, K, wt, st);
    if (e != hipSuccess) return hip_status(e);
    // dX_hat [M][K] = dY [M][N] (W_hat^T [K][N])^T: the forward GEMM's plain product with N as the
    // contraction
    const FwdPlan p = plan_fwd(op_dtype, M, K, N);
    return hip_status(launch_recon_fwd(p, op_dtype, dY, wt, M, K, N, nullptr, dX_hat, nullptr, nullptr, ws_fwd, st));
}

focus_status focus_fakequant_act_bwd(const focus_qconfig *q, const void *X, int x_dtype, int64_t rows, int64_t K,
                                     const void *dX_hat, int g_dtype, void *dX, void *ws, size_t ws_bytes,
                                     focus_stream stream) {
    FOCUS_TRY(check_q(q));
    if (!X || !dX_hat || !dX) return FOCUS_ERR_NULL;
    if (!dtype_ok(x_dtype) || !dtype_ok(g_dtype)) return FOCUS_ERR_DTYPE;
    FOCUS_TRY(check_rows_k(rows, K, block_of(q->format)));
    if (!all_aligned({X, dX_hat, dX})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, focus_workspace_size(FOCUS_CALL_FAKEQUANT_ACT_BWD, q, 0, rows, K)));
    if (rows == 0 || K == 0) return FOCUS_OK;
    return hip_status(launch_fq_act_bwd(q->format, x_dtype, g_dtype, X, rows, K, floor_of(q), q->ste_clip, dX_hat, dX,
                                        partials_of(ws), (hipStream_t)stream));
}

focus_status focus_kl_top(const void *Z_student, const void *Z_teacher, int dtype, int64_t T, int64_t V, int32_t k,
                          void *dZ_student, double *loss_out, void *ws, size_t ws_bytes, focus_stream stream) {
    if (!Z_student || !Z_teacher || !dZ_student || !loss_out) return FOCUS_ERR_NULL;
    if (!dtype_ok(dtype)) return FOCUS_ERR_DTYPE;
    if (k < 1) return FOCUS_ERR_CONFIG;
    if (T < 1 || V < 1 || T > kMaxDim || V > (int64_t(1) << 31) || V > kMaxElems / T) return FOCUS_ERR_SHAPE;
    const size_t esz = dtype == FOCUS_BF16 ? 2 : 4;
    if ((reinterpret_cast<uintptr_t>(Z_student) | reinterpret_cast<uintptr_t>(Z_teacher) |
         reinterpret_cast<uintptr_t>(dZ_student)) % esz)
        return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, focus_workspace_size(FOCUS_CALL_KL_TOP, nullptr, T, V, 0)));
    double *row_loss = reinterpret_cast<double *>(static_cast<char *>(ws) + kWsHeader);
    return hip_status(launch_kl_top(dtype, Z_student, Z_teacher, T, V, k, dZ_student, row_loss, loss_out, flag_of(ws),
                                    (hipStream_t)stream));
}

focus_status focus_adamw_step(const focus_adamw_config *cfg, int64_t t, int64_t n, float *param, const float *grad,
                              float *exp_avg, float *exp_avg_sq, void *ws, size_t ws_bytes, focus_stream stream) {
    if (!cfg) return FOCUS_ERR_NULL;
    const bool finite = std::isfinite(cfg->lr) && std::isfinite(cfg->eps) && std::isfinite(cfg->weight_decay);
    if (!finite || !(cfg->lr >= 0.f) || !(cfg->beta1 >= 0.f && cfg->beta1 < 1.f) ||
        !(cfg->beta2 >= 0.f && cfg->beta2 < 1.f) || !(cfg->eps > 0.f) || !(cfg->weight_decay >= 0.f) ||
        (cfg->log2_domain != 0 && cfg->log2_domain != 1) || t < 1)
        return FOCUS_ERR_CONFIG;
    if (n < 0 || n > (int64_t(1) << 40)) return FOCUS_ERR_SHAPE;  // keeps the grid below 2^31 workgroups
    if (!param || !grad || !exp_avg || !exp_avg_sq) return FOCUS_ERR_NULL;
    if (!all_aligned({param, grad, exp_avg, exp_avg_sq})) return FOCUS_ERR_SHAPE;
    FOCUS_TRY(check_ws(ws, ws_bytes, kWsHeader));
    if (n == 0) return FOCUS_OK;
    return hip_status(launch_adamw(cfg->lr, cfg->beta1, cfg->beta2, cfg->eps, cfg->weight_decay, cfg->log2_domain,
                                   t, n, param, grad, exp_avg, exp_avg_sq, flag_of(ws), (hipStream_t)stream));
}

focus_status focus_check_flags(void *ws, focus_stream stream) {
    if (!ws) return FOCUS_ERR_WORKSPACE;
    if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return FOCUS_ERR_HIP;
    uint32_t flag = 0;
    if (hipMemcpy(&flag, ws, sizeof(flag), hipMemcpyDeviceToHost) != hipSuccess) return FOCUS_ERR_HIP;
    if (flag) {
        const uint32_t zero = 0;
        if (hipMemcpy(ws, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess) return FOCUS_ERR_HIP;
        return FOCUS_ERR_DOMAIN;
    }
    return FOCUS_OK;
}

const char *focus_status_string(int status) {
    switch (status) {
        case FOCUS_OK: return "ok";
        case FOCUS_ERR_NULL: return "a required pointer is NULL";
        case FOCUS_ERR_SHAPE: return "invalid sizes (negative, too large, or K not a multiple of the block size)";
        case FOCUS_ERR_DTYPE: return "unknown or unsupported dtype";
        case FOCUS_ERR_CONFIG: return "invalid quantisation configuration or argument combination";
        case FOCUS_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
        case FOCUS_ERR_DOMAIN: return "a kernel met a NaN scale or a coefficient c <= 0 or not finite";
        case FOCUS_ERR_HIP: return "HIP runtime error";
        case FOCUS_ERR_SCRATCH: return "the sizes need more scratch than the allocation-free call's fixed 32 MiB";
        default: return "unknown status";
    }
}

}  // extern "C"
