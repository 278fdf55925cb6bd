// Pieces shared by the VALU and MFMA reconstruction GEMMs.
#pragma once

#include "focus_device.h"

namespace focus {

__device__ __forceinline__ float load1(const void *base, int dtype, int64_t i) {
    return dtype == kBF16 ? bf16_bits_to_f32(reinterpret_cast<const uint16_t *>(base)[i])
                          : reinterpret_cast<const float *>(base)[i];
}

__device__ __forceinline__ void store1(void *base, int dtype, int64_t i, float v) {
    if (dtype == kBF16) reinterpret_cast<uint16_t *>(base)[i] = (uint16_t)f32_to_bf16_bits(v);
    else reinterpret_cast<float *>(base)[i] = v;
}

// Straight-through terms of one weight element given g = dL/dW_hat (Sec. 3.2 STE through Eq. 6-8):
// W_hat = Q(w / (S_dq c)) S_dq with Q -> clamp, so dW_hat/dc = -m w / c^2 and
// dW_hat/dS_dq = q - m u. The caller sums tc over the sub-block (then scales by -1/c^2) and ts over
// the block.
__device__ __forceinline__ void ste_terms(float g, float w, float sdq, float cval, bool ste_clip,
                                          float &tc, float &ts) {
    Quantized z = quantize_element(w, sdq * cval, sdq, ste_clip);
    tc = z.m ? g * w : 0.0f;
    ts = g * (z.q - (z.m ? z.u : 0.0f));
}

// ---- MFMA path geometry (gemm_mfma.hip) -------------------------------------------------------
constexpr int kMfmaTileM = 256;       // forward output tile: tokens
constexpr int kMfmaTileN = 256;       // backward output tile: out features
constexpr int kMfmaTileK = 256;       // backward output tile: in features
constexpr int kMfmaTokenStep = 64;    // backward reduction step over tokens
constexpr int kMfmaConcurrentWgs = 256;  // one 128 KB-LDS workgroup per CU, 256 CUs

bool mfma_fwd_supported(int64_t M, int64_t N, int64_t K);
bool mfma_bwd_supported(int64_t M, int64_t N, int64_t K);
hipError_t launch_fwd_mfma(const void *X, const void *W, int64_t M, int64_t N, int64_t K, const void *Yref,
                           void *dY, float dscale, double *colpart, hipStream_t st);
// the same product from packed MXFP4 operands (X codes [M][K/2], W codes in K-slabs [K/128][N][64],
// block-major E8M0 bytes [K/32][rows]; K % 128 == 0)
bool mfma_fwd_mx_supported(int64_t M, int64_t N, int64_t K);
hipError_t launch_fwd_mfma_mx(const void *Xc, const void *Xs, const void *Wc, const void *Ws, int64_t M, int64_t N,
                              int64_t K, const void *Yref, void *dY, float dscale, double *colpart, hipStream_t st);
hipError_t launch_bwd_mfma(int fmt, int w_dt, const void *dY, const void *X, int64_t M, int64_t N, int64_t K,
                           int64_t chunk, int64_t splits, const void *W, const float *s_fp, const float *c,
                           int sb, const float *alpha, int ste_clip, int e8m0_floor, float *part_s,
                           float *part_c, uint32_t *flag, hipStream_t st);

// the backward from X_hat as packed MXFP4 (codes [M][K/2], E8M0 bytes block-major [K/32][M])
bool mfma_bwd_mx_supported(int64_t M, int64_t N, int64_t K);
hipError_t launch_bwd_mfma_mx(int w_dt, const void *dY, const void *Xc, const void *Xs, int64_t M, int64_t N,
                              int64_t K, int64_t chunk, int64_t splits, const void *W, const float *s_fp,
                              const float *c, int sb, int ste_clip, int e8m0_floor, float *part_s, float *part_c,
                              uint32_t *flag, hipStream_t st);

}  // namespace focus
