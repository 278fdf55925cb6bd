// Launchers shared between the translation units of libfocus (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace focus {

constexpr int kStreamGridCap = 4096;  // workgroups of a grid-stride streaming kernel
constexpr int kAbsmaxParts = 1024;    // partial maxima of the tensor-absmax pass
constexpr size_t kWsHeader = 256;     // workspace bytes reserved for the domain flag

hipError_t launch_fq_weight(int fmt, int in_dt, int out_dt, const void *W, int64_t rows, int64_t K,
                            const float *s_fp, const float *c, int sb, const float *alpha, int e8m0_floor,
                            void *w_hat, uint8_t *codes, uint8_t *scale_bytes, int block_major, int code_slab,
                            uint32_t *flag, hipStream_t st);
// One layer of a grouped weight fake quantisation (the arguments of launch_fq_weight).
struct WeightLayer {
    const void *W;
    int64_t rows, K;
    const float *s_fp, *c, *alpha;
    void *w_hat;
    uint8_t *codes, *scale_bytes;
};
constexpr int kMaxWeightLayers = 16;
// All layers in one launch where their tiles fit one grid (bf16 weights), else one launch per layer;
// layer outputs are those of launch_fq_weight either way.
hipError_t launch_fq_weight_group(int fmt, int in_dt, int out_dt, const WeightLayer *layers, int n, int sb,
                                  int e8m0_floor, int block_major, int code_slab, uint32_t *flag, hipStream_t st);
hipError_t launch_fq_act(int fmt, int in_dt, int out_dt, const void *X, int64_t rows, int64_t K,
                         void *x_hat, uint8_t *codes, uint8_t *scale_bytes, int block_major, int code_slab, int e8m0_floor,
                         float *alpha_out, float *partial, uint32_t *flag, hipStream_t st);
hipError_t launch_scales_init(int fmt, int in_dt, const void *W, int64_t rows, int64_t K, float *s_fp,
                              float *c, int sb, int e8m0_floor, float *alpha_out, float *partial, hipStream_t st);
hipError_t launch_fq_bwd(int fmt, int w_dt, const float *G, int64_t rows, int64_t K, const void *W,
                         const float *s_fp, const float *c, int sb, const float *alpha, int ste_clip,
                         int e8m0_floor, float *grad_s, float *grad_c, uint32_t *flag, hipStream_t st);

// ---- reconstruction GEMMs ----------------------------------------------------------------------
// Geometry of a forward launch: output tiles of tm x tn; column partial sums [mtiles][N] (double).
struct FwdPlan {
    int path;       // 0 = VALU (fp32 / small), 1 = MFMA bf16
    int64_t mtiles;
    size_t ws_bytes;
};
// Geometry of a backward launch: G tiles of tn x tk, the token range split `splits` ways with
// `chunk` tokens per split; partial gradient sums [splits][N][K/B] and [splits][N][K/sb] (float).
struct BwdPlan {
    int path;
    int64_t splits;
    int64_t chunk;
    size_t ws_bytes;
};

FwdPlan plan_fwd(int op_dt, int64_t M, int64_t N, int64_t K);
BwdPlan plan_bwd(int op_dt, int fmt, int sb, int64_t M, int64_t N, int64_t K, bool want_G);

hipError_t launch_recon_fwd(const FwdPlan &p, int op_dt, const void *X, const void *W, int64_t M,
                            int64_t N, int64_t K, const void *Yref, void *dY, double *loss_out,
                            double *col_sq_opt, void *ws, hipStream_t st);
// column sums of D^2 from the per-m-tile partials, then the loss
hipError_t launch_fwd_finish(int64_t mtiles, int64_t M, int64_t N, const double *colpart, double *col_sq,
                             double *loss_out, hipStream_t st);
// the forward from packed MXFP4 operands (MFMA path only)
hipError_t launch_recon_fwd_mx(const void *Xc, const void *Xs, const void *Wc, const void *Ws, int64_t M, int64_t N,
                               int64_t K, const void *Yref, void *dY, double *loss_out, double *col_sq_opt, void *ws,
                               hipStream_t st);
hipError_t launch_recon_bwd(const BwdPlan &p, int op_dt, int fmt, int sb, int ste_clip, int e8m0_floor, const void *dY,
                            const void *X, int64_t M, int64_t N, int64_t K, const void *W, int w_dt,
                            const float *s_fp, const float *c, const float *alpha, float *grad_s,
                            float *grad_c, float *G_out, void *ws, uint32_t *flag, hipStream_t st);

// the backward from X_hat as packed MXFP4 (MFMA path only; the plan is that of the bf16 operands)
hipError_t launch_recon_bwd_mx(const BwdPlan &p, int sb, int ste_clip, int e8m0_floor, const void *dY, const void *Xc,
                               const void *Xs, int64_t M, int64_t N, int64_t K, const void *W, int w_dt,
                               const float *s_fp, const float *c, float *grad_s, float *grad_c, void *ws,
                               uint32_t *flag, hipStream_t st);

hipError_t launch_fq_act_bwd(int fmt, int in_dt, int g_dt, const void *X, int64_t rows, int64_t K, int e8m0_floor,
                             int ste_clip, const void *dX_hat, void *dX, float *partial, hipStream_t st);
hipError_t launch_zero_fill(void *p, size_t bytes, hipStream_t st);
hipError_t launch_transpose(int dt, const void *in, int64_t R, int64_t C, void *out, hipStream_t st);
hipError_t launch_kl_top(int dt, const void *Zs, const void *Zt, int64_t T, int64_t V, int k, void *dZs,
                         double *row_loss, double *loss, uint32_t *flag, hipStream_t st);

hipError_t launch_adamw(float lr, float beta1, float beta2, float eps, float weight_decay, int log2_domain,
                        int64_t t, int64_t n, float *param, const float *grad, float *exp_avg, float *exp_avg_sq,
                        uint32_t *flag, hipStream_t st);

}  // namespace focus
