// Device-side FP4 / scale codecs and small helpers shared by the FOCUS kernels (gfx950).
//
// The element format is E2M1 (Sec. 3.1, Eq. 1): magnitudes {0, .5, 1, 1.5, 2, 3, 4, 6}; a code is
// sign << 3 | magnitude index. Scales are E8M0 (MXFP4, Eq. 3, rounded up to a power of two) or
// OCP E4M3FN (NVFP4, Eq. 2). All decisions are taken on fp32 values produced by single, correctly
// rounded fp32 operations; the library is built with -ffp-contract=off so none is fused.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace focus {

constexpr int kFmtMX = 0;
constexpr int kFmtNV = 1;
constexpr int kF32 = 0;
constexpr int kBF16 = 1;

__host__ __device__ constexpr int block_of(int fmt) { return fmt == kFmtMX ? 32 : 16; }

// ---- E2M1 --------------------------------------------------------------------------------------
// A code is sign << 3 | magnitude index (grid 0, 0.5, 1, 1.5, 2, 3, 4, 6). Q_E2M1 rounds |u| to the
// nearest grid value, a midpoint (0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5) going to the even index, and
// saturates at 6; a NaN takes index 0 with its sign bit. gfx950's FP4 conversion rounds and
// saturates exactly so (pinned against the threshold form over every bf16 value and the fp32
// neighbourhoods of every midpoint by a GPU test); it gives a NaN the largest magnitude, so NaNs are
// replaced by a signed zero first.
__device__ __forceinline__ float e2m1_nan_to_zero(float u) {
    return u == u ? u : __uint_as_float(__float_as_uint(u) & 0x80000000u);
}

// Codes of u0, u1 written into byte `sel` of `word` (u0 in the low nibble).
template <int SEL>
__device__ __forceinline__ uint32_t e2m1_code2(uint32_t word, float u0, float u1) {
    return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(word, e2m1_nan_to_zero(u0), e2m1_nan_to_zero(u1), 1.0f, SEL);
}

__device__ __forceinline__ uint32_t e2m1_code(float u) { return e2m1_code2<0>(0u, u, 0.0f) & 0xFu; }

// Grid values of the two codes in byte SEL of `word` (low nibble first), signed.
template <int SEL>
__device__ __forceinline__ void e2m1_value2(uint32_t word, float &v0, float &v1) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const f32x2 v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(word, 1.0f, SEL);
    v0 = v.x;
    v1 = v.y;
}

__device__ __forceinline__ float e2m1_value(uint32_t code) {
    float v0, v1;
    e2m1_value2<0>(code, v0, v1);
    return v0;
}

// ---- E8M0 (scale rounded up to a power of two) ---------------------------------------------------
// Smallest e in [-127, 127] with 2^e >= s. Non-positive s (and -0) -> -127; +inf -> 127;
// NaN sets *nan_seen and gives -127.
__device__ __forceinline__ int e8m0_ceil_exp(float s, bool &nan_seen) {
    // every case computed, the result selected (no divergent branches)
    const uint32_t b = __float_as_uint(s);
    const bool nan = (b & 0x7FFFFFFFu) > 0x7F800000u;
    const uint32_t E = b >> 23, man = b & 0x7FFFFFu;
    int e = (int)E - 127 + (man != 0u);
    e = E == 0u ? (man > 0x400000u ? -126 : -127) : e;  // subnormal s < 2^-126; 2^-127 is man 0x400000
    e = e > 127 ? 127 : e;
    e = (nan || (int32_t)b <= 0) ? -127 : e;
    nan_seen = nan_seen || nan;
    return e;
}

// E8M0 rounded down, the OCP MX rule: e = floor(log2 s) - drop, clamped to [-127, 127] (drop = 2 for an
// activation block's amax, the exponent of E2M1's largest value; drop = 0 for a learned scale).
// Non-positive s (and -0) -> -127; +inf -> 127; NaN sets *nan_seen and gives -127. floor(log2 s) is
// exact for subnormal s too (from the position of the leading mantissa bit).
__device__ __forceinline__ int e8m0_floor_exp(float s, int drop, bool &nan_seen) {
    const uint32_t b = __float_as_uint(s);
    const bool nan = (b & 0x7FFFFFFFu) > 0x7F800000u;
    const uint32_t E = b >> 23, man = b & 0x7FFFFFu;
    int e = E != 0u ? (int)E - 127 : (31 - __builtin_clz(man | 1u)) - 149;
    e -= drop;
    e = e < -127 ? -127 : e;
    e = e > 127 ? 127 : e;
    e = (nan || (int32_t)b <= 0) ? -127 : e;
    nan_seen = nan_seen || nan;
    return e;
}

// 2^e as fp32 for e in [-127, 127]; 2^-127 is the subnormal 0x00400000.
__device__ __forceinline__ float exp2i(int e) {
    return e >= -126 ? __uint_as_float((uint32_t)(e + 127) << 23) : __uint_as_float(0x00400000u);
}

// ---- E4M3 (OCP E4M3FN: bias 7, max 448, subnormals m * 2^-9, no infinities) -----------------------
// Round to nearest, ties to even, saturating at 448; x <= 0 -> 0; NaN sets *nan_seen.
__device__ __forceinline__ uint32_t e4m3_code(float x, bool &nan_seen) {
    // every case computed, the result selected (no divergent branches)
    const uint32_t b = __float_as_uint(x);
    const bool nan = (b & 0x7FFFFFFFu) > 0x7F800000u;
    // normal E4M3 range [2^-6, 448): keep 3 mantissa bits with round-half-even
    const uint32_t r = b + 0x7FFFFu + ((b >> 20) & 1u);
    uint32_t normal = (((r >> 23) - 120u) << 3) | ((r >> 20) & 7u);
    normal = normal > 0x7Eu ? 0x7Eu : normal;
    // subnormal range: the nearest multiple of 2^-9, ties to even (x * 512 is exact); the clamp
    // only keeps the conversion defined for inputs the selects below discard
    const float t = __builtin_fminf(__builtin_fmaxf(x * 512.0f, 0.0f), 512.0f);
    const uint32_t sub = (uint32_t)__builtin_rintf(t);
    uint32_t code = x >= 0.015625f ? normal : sub;
    code = x >= 448.0f ? 0x7Eu : code;
    code = (nan || (int32_t)b <= 0) ? 0u : code;
    nan_seen = nan_seen || nan;
    return code;
}

__device__ __forceinline__ float e4m3_value(uint32_t code) {
    uint32_t E = code >> 3, M = code & 7u;
    return E == 0u ? (float)M * 0.001953125f : __uint_as_float(((E + 120u) << 23) | (M << 20));
}

// ---- bf16 ---------------------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// round to nearest even (NaN kept quiet)
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t b = __float_as_uint(f);
    if ((b & 0x7FFFFFFFu) > 0x7F800000u) return (b >> 16) | 0x40u;
    return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// ---- 8-element vector I/O ---------------------------------------------------------------------
// Loads 8 consecutive values of a bf16 or fp32 row as fp32 (16- or 32-byte vector loads).
__device__ __forceinline__ void load8(const void *base, int dtype, int64_t idx, float v[8]) {
    if (dtype == kBF16) {
        uint4 p = *reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(base) + idx);
        uint32_t w[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
    } else {
        const float4 *p = reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(base) + idx);
        float4 a = p[0], b = p[1];
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
}

__device__ __forceinline__ void store8(void *base, int dtype, int64_t idx, const float v[8]) {
    if (dtype == kBF16) {
        uint4 p;
        p.x = f32_to_bf16_bits(v[0]) | (f32_to_bf16_bits(v[1]) << 16);
        p.y = f32_to_bf16_bits(v[2]) | (f32_to_bf16_bits(v[3]) << 16);
        p.z = f32_to_bf16_bits(v[4]) | (f32_to_bf16_bits(v[5]) << 16);
        p.w = f32_to_bf16_bits(v[6]) | (f32_to_bf16_bits(v[7]) << 16);
        *reinterpret_cast<uint4 *>(reinterpret_cast<uint16_t *>(base) + idx) = p;
    } else {
        float4 *p = reinterpret_cast<float4 *>(reinterpret_cast<float *>(base) + idx);
        p[0] = make_float4(v[0], v[1], v[2], v[3]);
        p[1] = make_float4(v[4], v[5], v[6], v[7]);
    }
}

// ---- the per-element quantiser shared by every weight / activation kernel ----------------------
// Quantises x with the quantisation scale sq and dequantisation scale sdq (Eq. 7 / Eq. 8):
// u = fl32(x / sq), q = Q_E2M1(u), x_hat = fl32(q * sdq). Returns the 4-bit code; writes x_hat and
// (for the backward) u and the straight-through mask. A zero scale gives a signed zero, u = 0, m = 0.
struct Quantized {
    float xhat;
    float u;
    float q;       // signed E2M1 value
    uint32_t code;
    bool m;
};

__device__ __forceinline__ Quantized quantize_element(float x, float sq, float sdq, bool ste_clip) {
    // both cases are computed and the result masked: no divergent branch per element
    Quantized r;
    const uint32_t keep = 0u - (uint32_t)!(sdq == 0.0f || sq == 0.0f);  // all ones unless a scale is zero
    const float u = x / (keep ? sq : 1.0f);
    const uint32_t sign = __float_as_uint(x) & 0x80000000u;
    // a zero scale gives index 0: the code keeps only the sign
    const uint32_t code = e2m1_code(u) & (keep | 8u);
    r.u = __uint_as_float(__float_as_uint(u) & keep);
    r.code = (code & 7u) | (sign >> 28);
    r.q = __uint_as_float(__float_as_uint(e2m1_value(r.code & 7u)) | sign);
    r.m = keep && (ste_clip ? (__builtin_fabsf(u) <= 6.0f) : true);
    r.xhat = r.q * sdq;
    return r;
}

// ---- division by a quantisation scale without a per-element divide -----------------------------
// u = fl32(a / b) from y = fl32(1 / b), one correctly rounded division per scale, by Markstein's
// method (P. Markstein, IBM J. Res. Dev. 34(1), 1990): q0 = fl(a y), then twice q <- fl(q - r y) with
// the residual r = q b - a formed exactly by an FMA. The first correction leaves a quotient within one
// unit in the last place of a / b; from such a quotient and the correctly rounded reciprocal, the second
// gives the correctly rounded quotient (Markstein's theorem). That needs every intermediate away from
// overflow and underflow, which holds when 2^-40 <= b <= 2^40, |a| <= 2^80 and |a / b| >= 2^-4. Below
// 2^-4 the result stays within a few units of the last place of a / b, far under the smallest E2M1
// midpoint (0.25), with the sign of a; zeros keep their sign. Callers take this path only when every
// lane's operands are in that range (scale_in_fast_range, and a finite bf16 weight of at most 2^80).
__device__ __forceinline__ float div_by_scale(float a, float b, float y) {
    const float q0 = a * y;
    const float r0 = __builtin_fmaf(q0, b, -a);
    const float q1 = __builtin_fmaf(-r0, y, q0);
    const float r1 = __builtin_fmaf(q1, b, -a);
    return __builtin_fmaf(-r1, y, q1);
}

__device__ __forceinline__ bool scale_in_fast_range(float b) { return b >= 0x1p-40f && b <= 0x1p40f; }

// Nonzero when one of 8 bf16 values (four packed pairs) is not finite or exceeds 2^80 in magnitude
// (bits 0x6780): adding 0x187F to a 15-bit magnitude sets its bit 15 exactly when the magnitude
// exceeds 0x6780, and both halves of a word are tested at once (no carry crosses them).
__device__ __forceinline__ uint32_t bf16x8_over_2p80(uint4 p) {
    constexpr uint32_t M = 0x7FFF7FFFu, C = 0x187F187Fu;
    return (((p.x & M) + C) | ((p.y & M) + C) | ((p.z & M) + C) | ((p.w & M) + C)) & 0x80008000u;
}

// Dequantisation scale of one weight block from its learnable copy (Eq. 4): MXFP4 2^E8M0(s), rounded
// up (default) or down (e8m0_floor, the OCP rule), NVFP4 fl32(alpha * Q_E4M3(s)). Also returns the
// exported scale byte.
__device__ __forceinline__ float weight_sdq(int fmt, float s, float alpha, int e8m0_floor, uint32_t &byte,
                                            bool &nan_seen) {
    if (fmt == kFmtMX) {
        int e = e8m0_floor ? e8m0_floor_exp(s, 0, nan_seen) : e8m0_ceil_exp(s, nan_seen);
        byte = (uint32_t)(e + 127);
        return exp2i(e);
    }
    byte = e4m3_code(s, nan_seen);
    return alpha * e4m3_value(byte);
}

// a coefficient outside the domain (c <= 0, NaN or inf)
__device__ __forceinline__ bool bad_coeff(float c) {
    return !(c > 0.0f) || __float_as_uint(c) == 0x7F800000u;
}

// Sticky flag in the first word of the workspace. Plain stores of the same value from many lanes
// are benign; nothing on the hot path writes it unless an input is outside the domain.
__device__ __forceinline__ void raise_domain_flag(uint32_t *flag) { *reinterpret_cast<volatile uint32_t *>(flag) = 1u; }

}  // namespace focus
