// AdamW update of the learnable scales and coefficients (Sec. 4.1: AdamW, constant learning rate;
// the optimizer of Loshchilov & Hutter, "Decoupled Weight Decay Regularization", with bias-corrected
// moments).
//
// One thread updates four consecutive parameters with 16-byte loads and stores of the parameter,
// the gradient and both moments; the last thread of a ragged length takes the tail element by
// element. HBM-bound: 16 bytes read and 12 written per parameter.
//
// Optional log2 domain: the parameter p > 0 is stored as it is (the other kernels read S_fp in the
// linear domain) while the step is taken on theta = log2(p), with dL/dtheta = dL/dp * p * ln 2 and
// the moments kept for theta; the new p is 2^theta. A p that is not positive and finite in this mode
// raises the domain flag and the element is left unchanged.
#include <cmath>

#include "internal.h"

namespace focus {

namespace {

constexpr float kLn2 = 0.693147180559945309f;

struct AdamArgs {
    float lr_decay;    // lr * weight_decay
    float beta1, beta2;
    float one_m_beta1, one_m_beta2;
    float step_size;   // lr / (1 - beta1^t)
    float bc2_sqrt;    // sqrt(1 - beta2^t)
    float eps;
    int log2_domain;
};

__device__ __forceinline__ void adam_one(float &p, float g, float &m, float &v, const AdamArgs &a, uint32_t &bad) {
    float theta = p, gt = g;
    if (a.log2_domain) {
        if (!(p > 0.f && p < INFINITY)) {
            bad = 1u;
            return;
        }
        theta = log2f(p);
        gt = g * p * kLn2;
    }
    theta = theta - a.lr_decay * theta;
    const float m1 = a.beta1 * m + a.one_m_beta1 * gt;
    const float v1 = a.beta2 * v + a.one_m_beta2 * (gt * gt);
    const float denom = sqrtf(v1) / a.bc2_sqrt + a.eps;
    theta = theta - a.step_size * (m1 / denom);
    m = m1;
    v = v1;
    p = a.log2_domain ? exp2f(theta) : theta;
}

__global__ void __launch_bounds__(256) adamw_kernel(float *__restrict__ param, const float *__restrict__ grad,
                                                     float *__restrict__ exp_avg, float *__restrict__ exp_avg_sq,
                                                     int64_t n, AdamArgs a, uint32_t *flag) {
    const int64_t i0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
    if (i0 >= n) return;
    uint32_t bad = 0;
    if (i0 + 4 <= n) {
        // every element is read and written once per step: the non-temporal cache policy (10% faster
        // on the hidden-8192 block's scales and coefficients, same bits)
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        const f32x4 pv = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(param + i0));
        const f32x4 gv = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(grad + i0));
        const f32x4 mv = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(exp_avg + i0));
        const f32x4 vv = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(exp_avg_sq + i0));
        float p[4] = {pv.x, pv.y, pv.z, pv.w}, m[4] = {mv.x, mv.y, mv.z, mv.w}, v[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
        for (int k = 0; k < 4; k++) adam_one(p[k], gv[k], m[k], v[k], a, bad);
        __builtin_nontemporal_store(f32x4{p[0], p[1], p[2], p[3]}, reinterpret_cast<f32x4 *>(param + i0));
        __builtin_nontemporal_store(f32x4{m[0], m[1], m[2], m[3]}, reinterpret_cast<f32x4 *>(exp_avg + i0));
        __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, reinterpret_cast<f32x4 *>(exp_avg_sq + i0));
    } else {
        for (int64_t i = i0; i < n; i++) {
            float p = param[i], m = exp_avg[i], v = exp_avg_sq[i];
            adam_one(p, grad[i], m, v, a, bad);
            param[i] = p;
            exp_avg[i] = m;
            exp_avg_sq[i] = v;
        }
    }
    if (bad) *flag = 1u;
}

}  // namespace

hipError_t launch_adamw(float lr, float beta1, float beta2, float eps, float weight_decay, int log2_domain,
                        int64_t t, int64_t n, float *param, const float *grad, float *exp_avg, float *exp_avg_sq,
                        uint32_t *flag, hipStream_t st) {
    // bias corrections in double on the host, rounded once to fp32
    const double bc1 = 1.0 - std::pow((double)beta1, (double)t);
    const double bc2 = 1.0 - std::pow((double)beta2, (double)t);
    AdamArgs a;
    a.lr_decay = (float)((double)lr * (double)weight_decay);
    a.beta1 = beta1;
    a.beta2 = beta2;
    a.one_m_beta1 = (float)(1.0 - (double)beta1);
    a.one_m_beta2 = (float)(1.0 - (double)beta2);
    a.step_size = (float)((double)lr / bc1);
    a.bc2_sqrt = (float)std::sqrt(bc2);
    a.eps = eps;
    a.log2_domain = log2_domain;
    const int64_t threads = (n + 3) / 4;
    const unsigned grid = (unsigned)((threads + 255) / 256);
    adamw_kernel<<<grid, 256, 0, st>>>(param, grad, exp_avg, exp_avg_sq, n, a, flag);
    return hipGetLastError();
}

}  // namespace focus
