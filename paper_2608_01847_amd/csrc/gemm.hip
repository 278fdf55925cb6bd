// Reconstruction GEMMs of the FOCUS step: planning, the LDS-tiled VALU kernels (fp32 operands,
// and any shape) with the fused MSE / straight-through epilogues, and the deterministic
// reductions that finish both. The bf16 MFMA kernels live in gemm_mfma.hip.
#include "focus_device.h"
#include "gemm_common.h"
#include "internal.h"

namespace focus {

// ------------------------------------------------------------------------------------------------
// VALU forward: 64 x 64 output tile, 256 threads, 4 x 4 outputs per thread, K steps of 16.
// Epilogue: D = Y_hat - Y_ref, dY = D * dscale, per-column sums of D^2 over the tile's rows (fp64),
// written as colpart[mtile][n]. Plain mode (Yref == nullptr) stores Y_hat.
template <int DT>
__global__ void __launch_bounds__(256)
fwd_valu_kernel(const void *__restrict__ X, const void *__restrict__ W, int64_t M, int64_t N, int64_t K,
                const void *__restrict__ Yref, void *__restrict__ dY, float dscale,
                double *__restrict__ colpart) {
    __shared__ float As[16][68];
    __shared__ float Bs[16][68];
    __shared__ double cs[16][64];
    const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
    const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
    float acc[4][4] = {};
    for (int64_t k0 = 0; k0 < K; k0 += 16) {
        for (int i = threadIdx.x; i < 64 * 16; i += 256) {
            const int r = i / 16, kk = i % 16;
            const int64_t gk = k0 + kk;
            const int64_t gm = m0 + r, gn = n0 + r;
            As[kk][r] = (gm < M && gk < K) ? load1(X, DT, gm * K + gk) : 0.0f;
            Bs[kk][r] = (gn < N && gk < K) ? load1(W, DT, gn * K + gk) : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; kk++) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                a[i] = As[kk][ty * 4 + i];
                b[i] = Bs[kk][tx * 4 + i];
            }
#pragma unroll
            for (int i = 0; i < 4; i++)
#pragma unroll
                for (int j = 0; j < 4; j++) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
    double colsum[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const int64_t m = m0 + ty * 4 + i;
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int64_t n = n0 + tx * 4 + j;
            if (m < M && n < N) {
                const int64_t o = m * N + n;
                if (Yref) {
                    const float d = acc[i][j] - load1(Yref, DT, o);
                    store1(dY, DT, o, d * dscale);
                    colsum[j] += (double)d * (double)d;
                } else {
                    store1(dY, DT, o, acc[i][j]);
                }
            }
        }
    }
    if (!Yref) return;
#pragma unroll
    for (int j = 0; j < 4; j++) cs[ty][tx * 4 + j] = colsum[j];
    __syncthreads();
    if (threadIdx.x < 64 && n0 + threadIdx.x < N) {
        double s = 0.0;
        for (int r = 0; r < 16; r++) s += cs[r][threadIdx.x];
        colpart[(int64_t)blockIdx.y * N + n0 + threadIdx.x] = s;
    }
}

// ------------------------------------------------------------------------------------------------
// VALU backward: G tile of 64 (n) x 64 (k) reduced over the tokens [z*chunk, min(M,(z+1)*chunk)),
// then the fused straight-through epilogue (sums per sub-block and per block, see ste_terms).
template <int DT, int FMT, int WDT>
__global__ void __launch_bounds__(256)
bwd_valu_kernel(const void *__restrict__ dY, const void *__restrict__ X, int64_t M, int64_t N, int64_t K,
                int64_t chunk, const void *__restrict__ W, const float *__restrict__ s_fp,
                const float *__restrict__ c, int sb, const float *__restrict__ alpha_ptr, int ste_clip, int e8m0_floor,
                float *__restrict__ part_s, float *__restrict__ part_c, float *__restrict__ G_out,
                uint32_t *flag) {
    constexpr int B = block_of(FMT);
    __shared__ float As[16][68];
    __shared__ float Bs[16][68];
    __shared__ float Tc[64][65];
    __shared__ float Ts[64][65];
    const int64_t n0 = (int64_t)blockIdx.y * 64, kb = (int64_t)blockIdx.x * 64;
    const int64_t t0 = (int64_t)blockIdx.z * chunk, t1 = std::min<int64_t>(M, t0 + chunk);
    const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
    float acc[4][4] = {};
    for (int64_t tb = t0; tb < t1; tb += 16) {
        for (int i = threadIdx.x; i < 64 * 16; i += 256) {
            const int r = i % 64, tt = i / 64;
            const int64_t t = tb + tt;
            As[tt][r] = (t < t1 && n0 + r < N) ? load1(dY, DT, t * N + n0 + r) : 0.0f;
            Bs[tt][r] = (t < t1 && kb + r < K) ? load1(X, DT, t * K + kb + r) : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int tt = 0; tt < 16; tt++) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                a[i] = As[tt][ty * 4 + i];
                b[i] = Bs[tt][tx * 4 + i];
            }
#pragma unroll
            for (int i = 0; i < 4; i++)
#pragma unroll
                for (int j = 0; j < 4; j++) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
    const float alpha = FMT == kFmtNV ? *alpha_ptr : 1.0f;
    const int64_t nb = K / B, ns = K / sb;
    bool bad = false;
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const int64_t n = n0 + ty * 4 + i;
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int64_t k = kb + tx * 4 + j;
            float tc = 0.0f, ts = 0.0f;
            if (n < N && k < K) {
                if (G_out) G_out[n * K + k] = acc[i][j];
                uint32_t byte;
                const float sdq = weight_sdq(FMT, s_fp[n * nb + k / B], alpha, e8m0_floor, byte, bad);
                const float cv = c ? c[n * ns + k / sb] : 1.0f;
                bad |= bad_coeff(cv);
                ste_terms(acc[i][j], load1(W, WDT, n * K + k), sdq, cv, ste_clip != 0, tc, ts);
            }
            Tc[ty * 4 + i][tx * 4 + j] = tc;
            Ts[ty * 4 + i][tx * 4 + j] = ts;
        }
    }
    __syncthreads();
    const int nsub = 64 / sb;
    for (int e = threadIdx.x; e < 64 * nsub; e += 256) {
        const int r = e / nsub, s = e % nsub;
        const int64_t n = n0 + r, k = kb + (int64_t)s * sb;
        if (n < N && k < K) {
            float sum = 0.0f;
            for (int x = 0; x < sb; x++) sum += Tc[r][s * sb + x];
            part_c[((int64_t)blockIdx.z * N + n) * ns + k / sb] = sum;
        }
    }
    constexpr int nblk = 64 / B;
    for (int e = threadIdx.x; e < 64 * nblk; e += 256) {
        const int r = e / nblk, s = e % nblk;
        const int64_t n = n0 + r, k = kb + (int64_t)s * B;
        if (n < N && k < K) {
            float sum = 0.0f;
            for (int x = 0; x < B; x++) sum += Ts[r][s * B + x];
            part_s[((int64_t)blockIdx.z * N + n) * nb + k / B] = sum;
        }
    }
    if (bad) raise_domain_flag(flag);
}

// ------------------------------------------------------------------------------------------------
// Deterministic finishing reductions (fixed summation order, no atomics).

// col_sq[n] = sum over m-tiles of colpart[mt][n] in a fixed order: 16 row groups (mt mod 16, each
// summed in ascending mt), then a fixed pairwise tree over the groups. A workgroup covers 16
// columns, so even a narrow layer spreads over many workgroups.
__global__ void __launch_bounds__(256)
colsum_kernel(const double *__restrict__ colpart, int64_t mtiles, int64_t N, double *__restrict__ col_sq) {
    __shared__ double red[16][16];
    const int cx = threadIdx.x & 15, grp = threadIdx.x >> 4;
    const int64_t n = (int64_t)blockIdx.x * 16 + cx;
    double s = 0.0;
    if (n < N)
        for (int64_t mt = grp; mt < mtiles; mt += 16) s += colpart[mt * N + n];
    red[grp][cx] = s;
    __syncthreads();
    for (int w = 8; w > 0; w >>= 1) {
        if (grp < w) red[grp][cx] += red[grp + w][cx];
        __syncthreads();
    }
    if (grp == 0 && n < N) col_sq[n] = red[0][cx];
}

// loss = (sum over n of col_sq[n]) / (M N); one workgroup, strided partial sums then a fixed tree
__global__ void __launch_bounds__(256)
loss_kernel(const double *__restrict__ col_sq, int64_t N, double inv_mn, double *__restrict__ loss) {
    __shared__ double red[256];
    double s = 0.0;
    for (int64_t n = threadIdx.x; n < N; n += 256) s += col_sq[n];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = red[0] * inv_mn;
}

// grad_c = -(sum over splits of part_c) / c^2 ; grad_s = f * (sum over splits of part_s)
__global__ void __launch_bounds__(256)
bwd_finish_kernel(const float *__restrict__ part_s, const float *__restrict__ part_c, int64_t splits,
                  int64_t n_s, int64_t n_c, const float *__restrict__ c, const float *__restrict__ alpha_ptr,
                  int fmt, float *__restrict__ grad_s, float *__restrict__ grad_c) {
    const float f = fmt == kFmtNV ? *alpha_ptr : 1.0f;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n_s + n_c; i += (int64_t)gridDim.x * 256) {
        if (i < n_c) {
            float s = 0.0f;
            for (int64_t z = 0; z < splits; z++) s += part_c[z * n_c + i];
            const float cv = c ? c[i] : 1.0f;
            grad_c[i] = -s / (cv * cv);
        } else {
            const int64_t j = i - n_c;
            float s = 0.0f;
            for (int64_t z = 0; z < splits; z++) s += part_s[z * n_s + j];
            grad_s[j] = fmt == kFmtNV ? s * f : s;
        }
    }
}

// ================================================================================================
// Planning and dispatch
// ================================================================================================

static int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

FwdPlan plan_fwd(int op_dt, int64_t M, int64_t N, int64_t K) {
    FwdPlan p;
    p.path = (op_dt == kBF16 && mfma_fwd_supported(M, N, K)) ? 1 : 0;
    const int64_t tm = p.path == 1 ? kMfmaTileM : 64;
    p.mtiles = cdiv(M, tm);
    p.ws_bytes = kWsHeader + (size_t)(p.mtiles * N + N) * sizeof(double);
    return p;
}

BwdPlan plan_bwd(int op_dt, int fmt, int sb, int64_t M, int64_t N, int64_t K, bool want_G) {
    BwdPlan p;
    p.path = (op_dt == kBF16 && !want_G && mfma_bwd_supported(M, N, K)) ? 1 : 0;
    const int64_t tn = p.path == 1 ? kMfmaTileN : 64, tk = p.path == 1 ? kMfmaTileK : 64;
    const int64_t step = p.path == 1 ? kMfmaTokenStep : 16;
    const int64_t tiles = cdiv(N, tn) * cdiv(K, tk);
    const int64_t steps_total = cdiv(std::max<int64_t>(M, 1), step);
    int64_t splits = 1;
    if (!want_G) {
        // The token range is split so that tiles * splits workgroups fill the chip in whole rounds
        // (one 256 x 256 workgroup per CU on the MFMA path, several 64 x 64 ones on the VALU path):
        // minimise rounds * (steps per split + epilogue), each split keeping >= 4 steps. The MFMA
        // path's straight-through epilogue (a 256 x 256 tile at one wave per SIMD) costs about as
        // much as 36 of its 64-token steps, as measured on MI355X.
        const int64_t slots = p.path == 1 ? kMfmaConcurrentWgs : 2048;
        const int64_t epilogue_steps = p.path == 1 ? 36 : 4;
        const int64_t max_splits = std::max<int64_t>(1, std::min<int64_t>(steps_total / 4, 4096));
        int64_t best = -1;
        for (int64_t s = 1; s <= max_splits; s++) {
            const int64_t rounds = cdiv(tiles * s, slots);
            const int64_t cost = rounds * (cdiv(steps_total, s) + epilogue_steps);
            if (best < 0 || cost < best) {
                best = cost;
                splits = s;
            }
        }
    }
    p.chunk = cdiv(steps_total, splits) * step;
    p.splits = std::max<int64_t>(1, cdiv(M, p.chunk));
    const int64_t nb = K / block_of(fmt), ns = K / sb;
    p.ws_bytes = kWsHeader + (size_t)(p.splits * N * (nb + ns)) * sizeof(float);
    return p;
}

hipError_t launch_recon_fwd(const FwdPlan &p, int op_dt, const void *X, const void *W, int64_t M,
                            int64_t N, int64_t K, const void *Yref, void *dY, double *loss_out,
                            double *col_sq_opt, void *ws, hipStream_t st) {
    double *colpart = reinterpret_cast<double *>(reinterpret_cast<char *>(ws) + kWsHeader);
    double *col_sq = col_sq_opt ? col_sq_opt : colpart + p.mtiles * N;
    const float dscale = (float)(2.0 / ((double)M * (double)N));
    if (p.path == 1) {
        hipError_t e = launch_fwd_mfma(X, W, M, N, K, Yref, dY, dscale, colpart, st);
        if (e != hipSuccess) return e;
    } else {
        dim3 grid((unsigned)cdiv(N, 64), (unsigned)cdiv(M, 64));
        if (op_dt == kBF16) fwd_valu_kernel<kBF16><<<grid, 256, 0, st>>>(X, W, M, N, K, Yref, dY, dscale, colpart);
        else fwd_valu_kernel<kF32><<<grid, 256, 0, st>>>(X, W, M, N, K, Yref, dY, dscale, colpart);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (!Yref) return hipSuccess;
    return launch_fwd_finish(p.mtiles, M, N, colpart, col_sq, loss_out, st);
}

hipError_t launch_fwd_finish(int64_t mtiles, int64_t M, int64_t N, const double *colpart, double *col_sq,
                             double *loss_out, hipStream_t st) {
    colsum_kernel<<<(unsigned)cdiv(N, 16), 256, 0, st>>>(colpart, mtiles, N, col_sq);
    if (loss_out) loss_kernel<<<1, 256, 0, st>>>(col_sq, N, 1.0 / ((double)M * (double)N), loss_out);
    return hipGetLastError();
}

hipError_t launch_recon_fwd_mx(const void *Xc, const void *Xs, const void *Wc, const void *Ws, int64_t M, int64_t N,
                               int64_t K, const void *Yref, void *dY, double *loss_out, double *col_sq_opt, void *ws,
                               hipStream_t st) {
    const int64_t mtiles = cdiv(M, kMfmaTileM);
    double *colpart = reinterpret_cast<double *>(reinterpret_cast<char *>(ws) + kWsHeader);
    double *col_sq = col_sq_opt ? col_sq_opt : colpart + mtiles * N;
    const float dscale = (float)(2.0 / ((double)M * (double)N));
    hipError_t e = launch_fwd_mfma_mx(Xc, Xs, Wc, Ws, M, N, K, Yref, dY, dscale, colpart, st);
    if (e != hipSuccess || !Yref) return e;
    return launch_fwd_finish(mtiles, M, N, colpart, col_sq, loss_out, st);
}

hipError_t launch_recon_bwd(const BwdPlan &p, int op_dt, int fmt, int sb, int ste_clip, int e8m0_floor, const void *dY,
                            const void *X, int64_t M, int64_t N, int64_t K, const void *W, int w_dt,
                            const float *s_fp, const float *c, const float *alpha, float *grad_s,
                            float *grad_c, float *G_out, void *ws, uint32_t *flag, hipStream_t st) {
    const int64_t nb = K / block_of(fmt), ns = K / sb;
    float *part_s = reinterpret_cast<float *>(reinterpret_cast<char *>(ws) + kWsHeader);
    float *part_c = part_s + p.splits * N * nb;
    if (p.path == 1) {
        hipError_t e = launch_bwd_mfma(fmt, w_dt, dY, X, M, N, K, p.chunk, p.splits, W, s_fp, c, sb,
                                       alpha, ste_clip, e8m0_floor, part_s, part_c, flag, st);
        if (e != hipSuccess) return e;
    } else {
        dim3 grid((unsigned)cdiv(K, 64), (unsigned)cdiv(N, 64), (unsigned)p.splits);
#define BV(D, F, WD) bwd_valu_kernel<D, F, WD><<<grid, 256, 0, st>>>(dY, X, M, N, K, p.chunk, W, s_fp, c, sb, alpha, ste_clip, e8m0_floor, part_s, part_c, G_out, flag)
        if (op_dt == kBF16) {
            if (fmt == kFmtMX) { if (w_dt == kBF16) BV(kBF16, kFmtMX, kBF16); else BV(kBF16, kFmtMX, kF32); }
            else { if (w_dt == kBF16) BV(kBF16, kFmtNV, kBF16); else BV(kBF16, kFmtNV, kF32); }
        } else {
            if (fmt == kFmtMX) { if (w_dt == kBF16) BV(kF32, kFmtMX, kBF16); else BV(kF32, kFmtMX, kF32); }
            else { if (w_dt == kBF16) BV(kF32, kFmtNV, kBF16); else BV(kF32, kFmtNV, kF32); }
        }
#undef BV
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t total = N * (nb + ns);
    const unsigned g = (unsigned)std::min<int64_t>(std::max<int64_t>(cdiv(total, 256), 1), kStreamGridCap);
    bwd_finish_kernel<<<g, 256, 0, st>>>(part_s, part_c, p.splits, N * nb, N * ns, c, alpha, fmt, grad_s, grad_c);
    return hipGetLastError();
}

hipError_t launch_recon_bwd_mx(const BwdPlan &p, int sb, int ste_clip, int e8m0_floor, const void *dY, const void *Xc,
                               const void *Xs, int64_t M, int64_t N, int64_t K, const void *W, int w_dt,
                               const float *s_fp, const float *c, float *grad_s, float *grad_c, void *ws,
                               uint32_t *flag, hipStream_t st) {
    const int64_t nb = K / 32, ns = K / sb;
    float *part_s = reinterpret_cast<float *>(reinterpret_cast<char *>(ws) + kWsHeader);
    float *part_c = part_s + p.splits * N * nb;
    hipError_t e = launch_bwd_mfma_mx(w_dt, dY, Xc, Xs, M, N, K, p.chunk, p.splits, W, s_fp, c, sb, ste_clip,
                                      e8m0_floor, part_s, part_c, flag, st);
    if (e != hipSuccess) return e;
    const int64_t total = N * (nb + ns);
    const unsigned g = (unsigned)std::min<int64_t>(std::max<int64_t>(cdiv(total, 256), 1), kStreamGridCap);
    bwd_finish_kernel<<<g, 256, 0, st>>>(part_s, part_c, p.splits, N * nb, N * ns, c, nullptr, kFmtMX, grad_s, grad_c);
    return hipGetLastError();
}

}  // namespace focus
