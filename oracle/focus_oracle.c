/*
 * CPU oracle for the FOCUS scale-learning step -- TEST INFRASTRUCTURE ONLY.
 *
 * This file is the plain, slow reference that the HIP library is checked against. Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load it; the product path never
 * does. It shares no code, header, table or constant generator with the HIP library.
 *
 * Everything here is written from the definitions in the FOCUS paper (arXiv 2608.01847):
 *   - E2M1 element quantisation, block scales and the NVFP4 / MXFP4 scale rules: Sec. 3.1, Eq. (1)-(3)
 *   - the learnable full-precision scale copy quantised on the fly: Sec. 3.2, Eq. (4)
 *   - the quantisation / dequantisation scale split: Sec. 3.2, Eq. (5)
 *   - Coupled-Relaxation Scaling S_q = S_dq * c: Sec. 3.3, Eq. (6)-(7)
 *   - Dual-Granularity Scaling (one coefficient per sub-block): Sec. 3.4, Eq. (8)
 *   - export of FP4 codes plus dequantisation scales only: Fig. 3(d), Sec. 3.4
 * and from the public format definitions (OCP E4M3FN and E8M0, bfloat16) that the paper relies on.
 *
 * Every codec is the definition written out: "nearest representable value, ties to the even
 * code", found by comparing exact distances in double precision, not by bit tricks. The fp32
 * operations of the method are written as single fp32 operations in the order the equations give
 * them; build with -O2 -fno-fast-math -ffp-contract=off so the compiler keeps them that way.
 *
 * Readings of points the paper leaves open (listed with reasons in the design notes):
 *   R1  Q_E8M0 rounds up (smallest power of two >= s), the "ceiling in practice" of Eq. (3).
 *   R2  Q_E2M1 ties go to the even code; magnitudes above 6 saturate to 6.
 *   R3  a zero code keeps the sign of its input.
 *   R4  Q_E4M3 is round-to-nearest-even onto OCP E4M3FN, saturating at 448; x <= 0 gives 0.
 *       A block whose dequantisation (or quantisation) scale is 0 has signed-zero codes.
 *   R5  MXFP4 learns S_fp in the linear domain; NVFP4 learns Delta_fp (E4M3 domain), alpha frozen.
 *   R6  blocks and sub-blocks run along K (the contiguous, reduction dimension); sub-blocks are
 *       contiguous runs of sb elements inside a block.
 *   R7  NVFP4 activations: alpha from the max over the whole tensor passed in; alpha = 1 if it is 0.
 *   R8  S_dq(NVFP4) = fl32(alpha * Delta); S_q = fl32(S_dq * c); u = fl32(w / S_q); w_hat = fl32(q * S_dq).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define FMT_MXFP4 0
#define FMT_NVFP4 1

/* ------------------------------------------------------------------------------------------ */
/* E2M1 element grid (Sec. 3.1, Eq. 1): magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6; code = sign<<3 | index */
static const double E2M1_MAGNITUDE[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

/* index of the E2M1 magnitude nearest to a >= 0; ties go to the even index (R2); beyond 6 the
   nearest representable magnitude is 6 (saturation), which also covers +inf */
static int e2m1_nearest_index(double a) {
    if (a > 6.0) return 7;
    int best = 0;
    double best_d = fabs(a - E2M1_MAGNITUDE[0]);
    for (int i = 1; i < 8; i++) {
        double d = fabs(a - E2M1_MAGNITUDE[i]);
        /* a tie can only be between neighbours i-1 and i: keep whichever index is even */
        if (d < best_d || (d == best_d && (i % 2) == 0)) {
            best = i;
            best_d = d;
        }
    }
    return best;
}

/* Q_E2M1 of Eq. (1): returns the signed E2M1 value, writes the 4-bit code (R3 keeps the sign) */
static float e2m1_quantize(float u, uint8_t *code) {
    int negative = signbit(u) ? 1 : 0;
    int idx = e2m1_nearest_index(fabs((double)u));
    *code = (uint8_t)((negative << 3) | idx);
    double v = negative ? -E2M1_MAGNITUDE[idx] : E2M1_MAGNITUDE[idx];
    return (float)v;
}

static float e2m1_decode(uint8_t code) {
    double v = E2M1_MAGNITUDE[code & 7];
    return (float)((code & 8) ? -v : v);
}

/* ------------------------------------------------------------------------------------------ */
/* Q_E8M0 (Sec. 3.1, Eq. 3; R1): the smallest e in [-127, 127] with 2^e >= s. Non-positive s takes
   the smallest scale 2^-127. frexp gives s = m * 2^E with m in [0.5, 1): then s <= 2^E, and
   s <= 2^(E-1) only when m is exactly 0.5. NaN is a domain error. */
static int e8m0_ceil_exponent(float s, int *domain_error) {
    if (isnan(s)) {
        *domain_error = 1;
        return -127;
    }
    if (!(s > 0.0f)) return -127;
    if (isinf(s)) return 127;
    int E;
    double m = frexp((double)s, &E);
    int e = (m == 0.5) ? E - 1 : E;
    if (e < -127) e = -127;
    if (e > 127) e = 127;
    return e;
}

/* Q_E8M0 rounded down, the OCP MX rule: e = floor(log2 s) - drop clamped to [-127, 127] (drop = 2 for
   an activation block's amax, the exponent of E2M1's largest value 6 = 1.5 * 2^2; drop = 0 for a
   learned scale). frexp gives s = m * 2^E with m in [0.5, 1), so floor(log2 s) = E - 1 exactly, for
   subnormal s too. Non-positive s takes 2^-127, +inf 2^127; NaN is a domain error. */
static int e8m0_floor_exponent(float s, int drop, int *domain_error) {
    if (isnan(s)) {
        *domain_error = 1;
        return -127;
    }
    if (!(s > 0.0f)) return -127;
    if (isinf(s)) return 127;
    int E;
    (void)frexp((double)s, &E);
    int e = E - 1 - drop;
    if (e < -127) e = -127;
    if (e > 127) e = 127;
    return e;
}

/* 2^e as an fp32 value; 2^-127 is an fp32 subnormal and is represented exactly */
static float pow2f(int e) { return (float)ldexp(1.0, e); }

/* ------------------------------------------------------------------------------------------ */
/* OCP E4M3FN: 1 sign, 4 exponent (bias 7), 3 mantissa bits, no infinities, 0x7F is NaN.
   Non-negative finite codes 0x00..0x7E increase monotonically in value. */
static double e4m3_value(int byte) {
    int E = (byte >> 3) & 15, m = byte & 7;
    if (E == 0) return (m / 8.0) * ldexp(1.0, -6); /* subnormals: m/8 * 2^-6 */
    return (1.0 + m / 8.0) * ldexp(1.0, E - 7);
}

static double E4M3_TABLE[127];
static int e4m3_table_ready = 0;

static void e4m3_table_init(void) {
    if (e4m3_table_ready) return;
    for (int b = 0; b < 127; b++) E4M3_TABLE[b] = e4m3_value(b);
    e4m3_table_ready = 1;
}

/* Q_E4M3 (Sec. 3.1, Eq. 2; R4): nearest non-negative finite E4M3 value, ties to the even code,
   x > 448 saturates to 448, x <= 0 gives 0. Returns the code byte. */
static int e4m3_nearest_code(float x, int *domain_error) {
    if (isnan(x)) {
        *domain_error = 1;
        return 0;
    }
    if (!(x > 0.0f)) return 0;
    if ((double)x >= E4M3_TABLE[126]) return 126; /* 0x7E = 448, the largest finite value */
    double dx = (double)x;
    /* binary search: the largest code lo with value(lo) <= x; then x lies in [value(lo), value(lo+1)) */
    int lo = 0, hi = 126;
    while (hi - lo > 1) {
        int mid = (lo + hi) / 2;
        if (E4M3_TABLE[mid] <= dx) lo = mid; else hi = mid;
    }
    double dlo = dx - E4M3_TABLE[lo], dhi = E4M3_TABLE[lo + 1] - dx;
    if (dlo < dhi) return lo;
    if (dhi < dlo) return lo + 1;
    return (lo % 2 == 0) ? lo : lo + 1;
}

/* ------------------------------------------------------------------------------------------ */
/* bfloat16 round to nearest, ties to even mantissa: the two bf16 neighbours of x are the value
   truncated toward zero and the next one away from zero; pick the closer one exactly. */
static float bf16_nearest(float x) {
    if (isnan(x) || isinf(x)) return x;
    uint32_t bits, lo_bits, hi_bits;
    memcpy(&bits, &x, 4);
    lo_bits = bits & 0xFFFF0000u;
    hi_bits = lo_bits + 0x10000u;
    float lo, hi;
    memcpy(&lo, &lo_bits, 4);
    memcpy(&hi, &hi_bits, 4);
    /* above the largest finite bf16 the next neighbour is 2^128, which rounds to infinity */
    double ax = fabs((double)x);
    double mag_lo = fabs((double)lo);
    double mag_hi = isinf(hi) ? ldexp(1.0, 128) : fabs((double)hi);
    double dlo = ax - mag_lo, dhi = mag_hi - ax;
    if (dlo < dhi) return lo;
    if (dhi < dlo) return hi;
    return ((lo_bits >> 16) & 1u) ? hi : lo;
}

/* ========================================================================================== */
/* Exported array entry points                                                                 */
/* ========================================================================================== */

void oracle_e2m1_array(const float *u, int64_t n, float *q, uint8_t *code) {
    for (int64_t i = 0; i < n; i++) q[i] = e2m1_quantize(u[i], &code[i]);
}

void oracle_e2m1_decode_array(const uint8_t *code, int64_t n, float *v) {
    for (int64_t i = 0; i < n; i++) v[i] = e2m1_decode(code[i]);
}

/* writes the E8M0 byte e + 127 */
int oracle_e8m0_ceil_array(const float *s, int64_t n, uint8_t *byte) {
    int err = 0;
    for (int64_t i = 0; i < n; i++) byte[i] = (uint8_t)(e8m0_ceil_exponent(s[i], &err) + 127);
    return err;
}

int oracle_e8m0_floor_array(const float *s, int64_t n, uint8_t *byte) {
    int err = 0;
    for (int64_t i = 0; i < n; i++) byte[i] = (uint8_t)(e8m0_floor_exponent(s[i], 0, &err) + 127);
    return err;
}

int oracle_e4m3_array(const float *x, int64_t n, uint8_t *byte) {
    int err = 0;
    e4m3_table_init();
    for (int64_t i = 0; i < n; i++) byte[i] = (uint8_t)e4m3_nearest_code(x[i], &err);
    return err;
}

void oracle_e4m3_decode_array(const uint8_t *byte, int64_t n, float *v) {
    for (int64_t i = 0; i < n; i++) v[i] = (float)e4m3_value(byte[i] & 0x7F);
}

void oracle_bf16_round_array(const float *x, int64_t n, float *y) {
    for (int64_t i = 0; i < n; i++) y[i] = bf16_nearest(x[i]);
}

static int block_size_of(int fmt) { return fmt == FMT_MXFP4 ? 32 : 16; }

/* ------------------------------------------------------------------------------------------ */
/* Scale initialisation by absmax (Sec. 3.2: "initialized via absmax"; Eq. 2 and Eq. 3).
   MXFP4: S_fp = fl32(amax / 6), or fl32(amax / 4) under the OCP floor rule (whose E8M0 is then the
   OCP exponent floor(log2 amax) - 2).  NVFP4: alpha = fl32(max|W| / (6 * 448)) (alpha = 1 if W == 0),
   Delta_fp = fl32(amax / fl32(alpha * 6)). Coefficients c start at 1 (Sec. 3.3, Sec. 3.4). */
int oracle_init_scales(int fmt, int sb, int e8m0_floor, const float *W, int64_t rows, int64_t K,
                       float *s_fp, float *c, float *alpha_out) {
    int B = block_size_of(fmt);
    int64_t nb = K / B, ns = K / sb;
    float alpha = 1.0f;
    if (fmt == FMT_NVFP4) {
        float A = 0.0f;
        for (int64_t i = 0; i < rows * K; i++) A = fmaxf(A, fabsf(W[i]));
        alpha = (A > 0.0f) ? A / 2688.0f : 1.0f; /* 2688 = M_FP4 * M_FP8 = 6 * 448 */
        *alpha_out = alpha;
    }
    for (int64_t r = 0; r < rows; r++) {
        for (int64_t b = 0; b < nb; b++) {
            float amax = 0.0f;
            for (int j = 0; j < B; j++) amax = fmaxf(amax, fabsf(W[r * K + b * B + j]));
            if (fmt == FMT_MXFP4) s_fp[r * nb + b] = e8m0_floor ? amax / 4.0f : amax / 6.0f;
            else s_fp[r * nb + b] = amax / (alpha * 6.0f);
        }
        for (int64_t k = 0; k < ns; k++) c[r * ns + k] = 1.0f;
    }
    return 0;
}

/* ------------------------------------------------------------------------------------------ */
/* Learned-scale fake quantisation of a weight tensor [rows][K] (Eq. 4, 6-8, 1):
     S_dq = Q_fmt(S_fp)            MXFP4: 2^E8M0(S_fp)          NVFP4: fl32(alpha * Q_E4M3(Delta_fp))
     S_q  = fl32(S_dq * c_k)       one coefficient per sub-block of sb elements (sb == B is CRS)
     u    = fl32(w / S_q);  code = Q_E2M1(u);  w_hat = fl32(q * S_dq)
   Also returns what the straight-through backward needs: u, the clamp mask m = [|u| <= 6]
   (m = 1 everywhere when ste_clip == 0), S_dq per block and S_q per sub-block.
   Optional outputs may be NULL. Returns nonzero if a NaN scale or c <= 0 / non-finite c was seen. */
int oracle_fq_weight(int fmt, int sb, int ste_clip, int e8m0_floor, const float *W, int64_t rows, int64_t K,
                     const float *s_fp, const float *c, float alpha,
                     float *w_hat, uint8_t *codes, uint8_t *scale_bytes,
                     float *u_out, uint8_t *m_out, float *sdq_out, float *sq_out) {
    int B = block_size_of(fmt);
    int64_t nb = K / B, ns = K / sb;
    int err = 0;
    e4m3_table_init();
    for (int64_t r = 0; r < rows; r++) {
        for (int64_t b = 0; b < nb; b++) {
            float sdq;
            int byte;
            if (fmt == FMT_MXFP4) {
                int e = e8m0_floor ? e8m0_floor_exponent(s_fp[r * nb + b], 0, &err)
                                   : e8m0_ceil_exponent(s_fp[r * nb + b], &err);
                sdq = pow2f(e);
                byte = e + 127;
            } else {
                byte = e4m3_nearest_code(s_fp[r * nb + b], &err);
                sdq = alpha * (float)e4m3_value(byte);
            }
            if (scale_bytes) scale_bytes[r * nb + b] = (uint8_t)byte;
            if (sdq_out) sdq_out[r * nb + b] = sdq;
            for (int j = 0; j < B; j++) {
                int64_t k = b * B + j;
                int64_t sub = k / sb;
                float ck = c ? c[r * ns + sub] : 1.0f;
                if (!(ck > 0.0f) || isinf(ck)) err = 1;
                float sq = sdq * ck;
                if (sq_out && (k % sb) == 0) sq_out[r * ns + sub] = sq;
                float w = W[r * K + k];
                float u, q;
                uint8_t code, m;
                if (sdq == 0.0f || sq == 0.0f) {
                    /* R4: a zero scale quantises the whole block to signed zeros */
                    u = 0.0f;
                    q = signbit(w) ? -0.0f : 0.0f;
                    code = (uint8_t)(signbit(w) ? 8 : 0);
                    m = 0;
                } else {
                    u = w / sq;
                    q = e2m1_quantize(u, &code);
                    m = ste_clip ? (uint8_t)(fabsf(u) <= 6.0f) : (uint8_t)1;
                }
                float wh = q * sdq;
                if (w_hat) w_hat[r * K + k] = wh;
                if (codes) codes[r * K + k] = code;
                if (u_out) u_out[r * K + k] = u;
                if (m_out) m_out[r * K + k] = m;
            }
        }
    }
    return err;
}

/* ------------------------------------------------------------------------------------------ */
/* Dynamic activation fake quantisation of X [rows][K] (Sec. 3.2: activation quantisation stays
   fully dynamic; Sec. 4.1: weights and activations of all linear layers are quantised). The
   scales are recomputed from X by the absmax rules of Eq. (2)-(3) with no coefficients (c = 1):
     MXFP4: S = 2^E8M0(fl32(amax / 6)), or under the OCP floor rule S = 2^(floor(log2 amax) - 2)
     NVFP4: alpha = fl32(max|X| / 2688) over the whole X (R7); Delta = Q_E4M3(fl32(amax / fl32(alpha*6)));
            S = fl32(alpha * Delta)
   then u = fl32(x / S), code = Q_E2M1(u), x_hat = fl32(q * S). Multithreaded over rows. */
int oracle_fq_act(int fmt, int e8m0_floor, const float *X, int64_t rows, int64_t K,
                  float *x_hat, uint8_t *codes, uint8_t *scale_bytes, float *alpha_out) {
    int B = block_size_of(fmt);
    int64_t nb = K / B;
    float alpha = 1.0f;
    int err = 0;
    e4m3_table_init();
    if (fmt == FMT_NVFP4) {
        float A = 0.0f;
#pragma omp parallel for reduction(max : A) schedule(static)
        for (int64_t i = 0; i < rows * K; i++) A = fmaxf(A, fabsf(X[i]));
        alpha = (A > 0.0f) ? A / 2688.0f : 1.0f;
        if (alpha_out) *alpha_out = alpha;
    }
#pragma omp parallel for schedule(static) reduction(| : err)
    for (int64_t r = 0; r < rows; r++) {
        for (int64_t b = 0; b < nb; b++) {
            const float *xb = X + r * K + b * B;
            float amax = 0.0f;
            for (int j = 0; j < B; j++) amax = fmaxf(amax, fabsf(xb[j]));
            float S;
            int byte;
            if (fmt == FMT_MXFP4) {
                int e = e8m0_floor ? e8m0_floor_exponent(amax, 2, &err) : e8m0_ceil_exponent(amax / 6.0f, &err);
                S = pow2f(e);
                byte = e + 127;
            } else {
                byte = e4m3_nearest_code(amax / (alpha * 6.0f), &err);
                S = alpha * (float)e4m3_value(byte);
            }
            if (scale_bytes) scale_bytes[r * nb + b] = (uint8_t)byte;
            for (int j = 0; j < B; j++) {
                float x = xb[j], q;
                uint8_t code;
                if (S == 0.0f) {
                    q = signbit(x) ? -0.0f : 0.0f;
                    code = (uint8_t)(signbit(x) ? 8 : 0);
                } else {
                    q = e2m1_quantize(x / S, &code);
                }
                if (x_hat) x_hat[r * K + b * B + j] = q * S;
                if (codes) codes[r * K + b * B + j] = code;
            }
        }
    }
    return err;
}

/* ------------------------------------------------------------------------------------------ */
/* Export (Fig. 3(d): only FP4 codes and dequantisation scales are kept). Two codes per byte, the
   even-k code in the low nibble; rows stay row-major. */
void oracle_pack_codes(const uint8_t *codes, int64_t rows, int64_t K, uint8_t *packed) {
    for (int64_t r = 0; r < rows; r++)
        for (int64_t j = 0; j < K / 2; j++)
            packed[r * (K / 2) + j] =
                (uint8_t)((codes[r * K + 2 * j] & 15) | ((codes[r * K + 2 * j + 1] & 15) << 4));
}

void oracle_unpack_codes(const uint8_t *packed, int64_t rows, int64_t K, uint8_t *codes) {
    for (int64_t r = 0; r < rows; r++)
        for (int64_t j = 0; j < K / 2; j++) {
            codes[r * K + 2 * j] = packed[r * (K / 2) + j] & 15;
            codes[r * K + 2 * j + 1] = (packed[r * (K / 2) + j] >> 4) & 15;
        }
}

/* dequantise an exported tensor: w_hat = fl32(E2M1(code) * S_dq), S_dq from the stored byte */
void oracle_decode_packed(int fmt, const uint8_t *packed, const uint8_t *scale_bytes, float alpha,
                          int64_t rows, int64_t K, float *out) {
    int B = block_size_of(fmt);
    int64_t nb = K / B;
    for (int64_t r = 0; r < rows; r++)
        for (int64_t k = 0; k < K; k++) {
            uint8_t byte = scale_bytes[r * nb + k / B];
            float sdq = (fmt == FMT_MXFP4) ? pow2f((int)byte - 127) : alpha * (float)e4m3_value(byte);
            uint8_t p = packed[r * (K / 2) + k / 2];
            uint8_t code = (k % 2 == 0) ? (p & 15) : (p >> 4);
            out[r * K + k] = e2m1_decode(code) * sdq;
        }
}
