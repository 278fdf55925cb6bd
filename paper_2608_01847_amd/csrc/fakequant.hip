// Streaming fake-quantisation kernels of the FOCUS step for gfx950 (HBM-bound).
//
// Work unit: a "chunk" of 8 consecutive elements along K, one per thread per loop trip (one
// 16-byte bf16 or 32-byte fp32 vector load). K is a multiple of the block size (16 or 32), so a
// block is 2 or 4 adjacent lanes and its absmax / gradient sums are formed with quad shuffles,
// never with atomics. Grids are capped and grid-stride; every lane of a block runs the same trips.
#include "focus_device.h"
#include "internal.h"

namespace focus {

// xor-shuffle within groups of `width` lanes (width <= 4 here); every lane of the group is active
__device__ __forceinline__ float shfl_xor_f(float v, int mask) { return __shfl_xor(v, mask, 64); }

__device__ __forceinline__ float group_max(float v, int lanes) {
    if (lanes >= 2) v = fmaxf(v, shfl_xor_f(v, 1));
    if (lanes >= 4) v = fmaxf(v, shfl_xor_f(v, 2));
    return v;
}

__device__ __forceinline__ float group_sum(float v, int lanes) {
    // fixed pairing order: (l ^ 1) then (l ^ 2); every lane ends with the same bits
    if (lanes >= 2) v = v + shfl_xor_f(v, 1);
    if (lanes >= 4) v = v + shfl_xor_f(v, 2);
    return v;
}

// ------------------------------------------------------------------------------------------------
// Tiles of the streaming fake-quant kernels. A workgroup covers 64 rows x 256 elements of a
// [rows][K] tensor; thread t takes 8-element chunk (t % 32) of rows t/32, t/32 + 8, ..., t/32 + 56, so
// each wave reads two 512-byte row pieces per load instruction and a block (32 or 16 elements) is 4
// or 2 adjacent lanes. (Wider tiles of 512 or 1024 elements and 32 or 16 rows, whose waves read 1 or
// 2 KB of one row per load, gave the same outputs and measured no faster.) All 8 chunks of a thread are loaded before any is used. The tile's scale
// bytes are staged in LDS and leave as 4-byte words: in the block-major layout [K/B][rows] a block's
// 64 rows are one contiguous 64-byte run, in the row-major layout [rows][K/B] a row's 8 (16) blocks
// are 2 (4) words.
constexpr int kTileRows = 64;
constexpr int kTileCols = 256;
constexpr int kRowStep = 8;   // rows between a thread's chunks (256 threads / 32 chunks per row)
constexpr int kChunks = 8;    // chunks per thread

struct Tile {
    int64_t row;       // row of the thread's first chunk (chunk i is row + 8 i)
    int64_t col;       // first element of the thread's chunks
    int64_t tile_row;  // first row of the tile
    int64_t row_end;   // one past the last row of the launch
    int64_t kb;        // first block of the tile
    int nrows;         // valid rows of the tile
    int nblk;          // valid blocks of the tile
    bool col_ok;
};

// Workgroups are handed to the 8 XCDs in turn (workgroup b to XCD b % 8); tile numbers are assigned so
// that each XCD takes one contiguous eighth of the tiles, so neighbouring column tiles, which share the
// 128-byte lines of a row's learnable scales, meet in one L2.
__device__ __forceinline__ uint32_t xcd_contiguous_tile() {
    const uint32_t G = gridDim.x, per = G / 8, rem = G % 8;
    const uint32_t x = blockIdx.x % 8, i = blockIdx.x / 8;
    return x < rem ? x * (per + 1) + i : rem * (per + 1) + (x - rem) * per + i;
}

template <int B>
__device__ __forceinline__ Tile tile_of(int64_t row0, int64_t rows, int64_t K, uint32_t ctiles,
                                        uint32_t tile = xcd_contiguous_tile()) {
    Tile t;
    const uint32_t rt = tile / ctiles, ct = tile - rt * ctiles;
    t.tile_row = row0 + (int64_t)rt * kTileRows;
    t.row_end = row0 + rows;
    t.row = t.tile_row + (threadIdx.x >> 5);
    t.col = (int64_t)ct * kTileCols + (threadIdx.x & 31) * 8;
    t.col_ok = t.col < K;
    t.kb = (int64_t)ct * (kTileCols / B);
    const int64_t nr = t.row_end - t.tile_row;
    t.nrows = nr < kTileRows ? (int)nr : kTileRows;
    const int64_t nb = (K - (int64_t)ct * kTileCols) / B;
    t.nblk = nb < kTileCols / B ? (int)nb : kTileCols / B;
    return t;
}

// Raw 16 bytes of chunk i (8 bf16 values), zero where the chunk lies outside the tensor. The weights
// and activations are read once per pass and the packed codes and fake-quantised tensors written once
// (store_code_word, store8_stream), so all of them go with the non-temporal cache policy: on the
// hidden-8192 block's tensors that made the packed activation pass 2-10% and the grouped weight pass
// 5-6% faster, with bf16 outputs (the NVFP4 block) 3% and 13%, with the same output bits and no change
// to the GEMMs that read the outputs next. (The small per-block S_fp and c loads keep the default
// policy: streamed as well they made the weight pass slower.)
__device__ __forceinline__ uint4 load_chunk_bf16(const void *X, const Tile &t, int64_t K, int i) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const int64_t r = t.row + (int64_t)i * kRowStep;
    if (!t.col_ok || r >= t.row_end) return make_uint4(0u, 0u, 0u, 0u);
    const u32x4 v = __builtin_nontemporal_load(
        reinterpret_cast<const u32x4 *>(reinterpret_cast<const uint16_t *>(X) + r * K + t.col));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// store8 with the non-temporal cache policy
__device__ __forceinline__ void store8_stream(void *base, int dtype, int64_t idx, const float v[8]) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    if (dtype == kBF16) {
        u32x4 p;
        p.x = f32_to_bf16_bits(v[0]) | (f32_to_bf16_bits(v[1]) << 16);
        p.y = f32_to_bf16_bits(v[2]) | (f32_to_bf16_bits(v[3]) << 16);
        p.z = f32_to_bf16_bits(v[4]) | (f32_to_bf16_bits(v[5]) << 16);
        p.w = f32_to_bf16_bits(v[6]) | (f32_to_bf16_bits(v[7]) << 16);
        __builtin_nontemporal_store(p, reinterpret_cast<u32x4 *>(reinterpret_cast<uint16_t *>(base) + idx));
    } else {
        u32x4 *p = reinterpret_cast<u32x4 *>(reinterpret_cast<float *>(base) + idx);
        __builtin_nontemporal_store(u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                                          __float_as_uint(v[3])}, p);
        __builtin_nontemporal_store(u32x4{__float_as_uint(v[4]), __float_as_uint(v[5]), __float_as_uint(v[6]),
                                          __float_as_uint(v[7])}, p + 1);
    }
}

__device__ __forceinline__ void store_code_word(uint8_t *dst, uint32_t packed) {
    __builtin_nontemporal_store(packed, reinterpret_cast<uint32_t *>(dst));
}

__device__ __forceinline__ void unpack_bf16(const uint4 p, float v[8]) {
    const uint32_t w[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
    for (int i = 0; i < 4; i++) {
        v[2 * i] = __uint_as_float(w[i] << 16);
        v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}

// Writes the staged scale bytes sb[j][r] (block kb + j, row tile_row + r) to a [rows_total][nb_total]
// (row-major) or [nb_total][rows_total] (block-major) array; one item per thread, 4-byte words where
// the four bytes are valid and the address is word aligned, single bytes otherwise.
template <int NBLK>
__device__ __forceinline__ void store_tile_scales(const uint8_t (&sb)[NBLK][kTileRows], const Tile &t,
                                                  uint8_t *out, int64_t rows_total, int64_t nb_total,
                                                  int block_major) {
    const int item = threadIdx.x;
    if (block_major) {
        // item -> block j = item / 16, rows 4 q .. 4 q + 3 with q = item % 16
        if (item >= NBLK * 16) return;
        const int j = item >> 4, r = (item & 15) * 4;
        if (j >= t.nblk || r >= t.nrows) return;
        uint8_t *dst = out + (t.kb + j) * rows_total + t.tile_row + r;
        if (r + 4 <= t.nrows && (reinterpret_cast<uintptr_t>(dst) & 3u) == 0) {
            *reinterpret_cast<uint32_t *>(dst) = *reinterpret_cast<const uint32_t *>(&sb[j][r]);
        } else {
            for (int k = 0; k < 4 && r + k < t.nrows; k++) dst[k] = sb[j][r + k];
        }
    } else {
        // item -> row r = item / (NBLK / 4), blocks 4 w .. 4 w + 3
        constexpr int WPR = NBLK / 4;
        if (item >= kTileRows * WPR) return;
        const int r = item / WPR, j = (item % WPR) * 4;
        if (r >= t.nrows || j >= t.nblk) return;
        uint8_t *dst = out + (t.tile_row + r) * nb_total + t.kb + j;
        if (j + 4 <= t.nblk && (reinterpret_cast<uintptr_t>(dst) & 3u) == 0) {
            const uint32_t w = (uint32_t)sb[j][r] | ((uint32_t)sb[j + 1][r] << 8) | ((uint32_t)sb[j + 2][r] << 16) |
                               ((uint32_t)sb[j + 3][r] << 24);
            *reinterpret_cast<uint32_t *>(dst) = w;
        } else {
            for (int k = 0; k < 4 && j + k < t.nblk; k++) dst[k] = sb[j + k][r];
        }
    }
}

// Grid of a tiled launch: row tiles x column tiles.
__host__ __device__ inline uint32_t col_tiles(int64_t K) { return (uint32_t)((K + kTileCols - 1) / kTileCols); }
constexpr uint32_t kMaxTiledGrid = 1u << 23;

// Byte offset of the 4-byte word of packed codes holding elements col .. col + 7 of row r (col % 8 == 0)
// of a [rows][K] tensor: row-major [rows][K/2], or K-slabs [K/128][rows][64] (code_slab).
__device__ __forceinline__ int64_t code_word_off(int64_t r, int64_t col, int64_t K, int64_t rows, int code_slab) {
    return code_slab ? ((col >> 7) * rows + r) * 64 + ((col & 127) >> 1) : (r * K + col) >> 1;
}

// Arguments of the tiled weight kernels for one layer: rows [row0, row0 + nrows) of a [rows][K] tensor
// (a launch may cover part of a tensor) with its scales, coefficients and outputs.
struct WeightJob {
    const void *W;
    const float *s_fp, *c, *alpha;
    void *w_hat;
    uint8_t *codes, *scale_bytes;
    int64_t row0, nrows, rows, K;
    uint32_t ctiles;
};
// Several layers of one launch (passed by value in the kernel arguments), layer l's tiles numbered
// from first[l].
struct WeightGroup {
    WeightJob job[kMaxWeightLayers];
    uint32_t first[kMaxWeightLayers];
    int n;
};

// ------------------------------------------------------------------------------------------------
// K1 / K7: weight fake quantisation with learned scales (Eq. 4, 6-8) and export (Fig. 3(d)), bf16
// weights. Per sub-block one correctly rounded reciprocal of S_q; u = W / S_q by div_by_scale when the
// whole wave's operands are in its range (always, for weights and scales of realistic size), by true
// division otherwise. Either way u is fl32(W / S_q) wherever the E2M1 rounding depends on it.
// (one coefficient per chunk fits 96 VGPRs: five waves per SIMD keep more loads in flight)
template <int FMT, int OUT, int NCOEF>
__device__ __forceinline__ void fq_weight_tile(const WeightJob &j, uint32_t tile, int sb_log2, int e8m0_floor,
                                               int block_major, int code_slab, uint32_t *flag) {
    const void *__restrict__ W = j.W;
    const float *__restrict__ s_fp = j.s_fp;
    const float *__restrict__ c = j.c;
    void *__restrict__ w_hat = j.w_hat;
    uint8_t *__restrict__ codes = j.codes;
    uint8_t *__restrict__ scale_bytes = j.scale_bytes;
    const int64_t K = j.K, rows_total = j.rows;
    constexpr int B = block_of(FMT);
    constexpr int NBLK = kTileCols / B;
    __shared__ uint8_t sbuf[NBLK][kTileRows];
    const Tile t = tile_of<B>(j.row0, j.nrows, K, j.ctiles, tile);
    // packed-code word of the thread's chunk 0, and the step to its next chunk (8 rows further)
    const int64_t cw0 = code_word_off(t.row, t.col, K, rows_total, code_slab);
    const int64_t cws = code_slab ? (int64_t)kRowStep * 64 : (int64_t)kRowStep * K / 2;
    // NCOEF coefficients per 8-element chunk: 1 for sub-blocks of 8 or more, 2 or 4 for 4 or 2
    constexpr int EPC = 8 / NCOEF;  // elements per coefficient within a chunk
    const float alpha = FMT == kFmtNV ? *j.alpha : 1.0f;
    const int64_t nb = K / B, ns = K >> sb_log2;
    bool bad = false;
    uint4 raw[kChunks];
#pragma unroll
    for (int i = 0; i < kChunks; i++) raw[i] = load_chunk_bf16(W, t, K, i);
    float sv[kChunks], cv[kChunks][NCOEF];
#pragma unroll
    for (int i = 0; i < kChunks; i++) {
        const int64_t r = t.row + (int64_t)i * kRowStep;
        const bool ok = t.col_ok && r < t.row_end;
        sv[i] = ok ? s_fp[r * nb + t.col / B] : 0.0f;
#pragma unroll
        for (int k = 0; k < NCOEF; k++) cv[i][k] = (c && ok) ? c[r * ns + (t.col >> sb_log2) + k] : 1.0f;
    }
#pragma unroll
    for (int i = 0; i < kChunks; i++) {
        const int64_t r = t.row + (int64_t)i * kRowStep;
        const bool ok = t.col_ok && r < t.row_end;
        uint32_t byte;
        bool nan_seen = false;
        const float sdq = weight_sdq(FMT, sv[i], alpha, e8m0_floor, byte, nan_seen);
        float sq[NCOEF], y[NCOEF];
        bool fast = bf16x8_over_2p80(raw[i]) == 0u;
#pragma unroll
        for (int k = 0; k < NCOEF; k++) {
            nan_seen |= bad_coeff(cv[i][k]);
            sq[k] = sdq * cv[i][k];
            y[k] = 1.0f / sq[k];
            fast = fast && scale_in_fast_range(sq[k]);
        }
        if (ok) bad |= nan_seen;
        float v[8], u[8];
        unpack_bf16(raw[i], v);
        uint32_t packed;
        if (__all(fast || !ok)) {
            // every lane in range: the codes of u straight from the FP4 conversion (u is finite and
            // carries the sign of w)
#pragma unroll
            for (int e = 0; e < 8; e++) u[e] = div_by_scale(v[e], sq[e / EPC], y[e / EPC]);
            packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, u[0], u[1], 1.0f, 0);
            packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, u[2], u[3], 1.0f, 1);
            packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, u[4], u[5], 1.0f, 2);
            packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, u[6], u[7], 1.0f, 3);
            // a zero-scale block never takes this path (its S_q is out of range)
        } else {
            packed = 0u;
#pragma unroll
            for (int e = 0; e < 8; e++) packed |= quantize_element(v[e], sq[e / EPC], sdq, true).code << (4 * e);
        }
        if (ok) {
            const int64_t e0 = r * K + t.col;
            if (w_hat) {
                float out[8];
                e2m1_value2<0>(packed, out[0], out[1]);
                e2m1_value2<1>(packed, out[2], out[3]);
                e2m1_value2<2>(packed, out[4], out[5]);
                e2m1_value2<3>(packed, out[6], out[7]);
#pragma unroll
                for (int e = 0; e < 8; e++) out[e] *= sdq;
                store8_stream(w_hat, OUT, e0, out);
            }
            if (codes) store_code_word(codes + cw0 + i * cws, packed);
            if (scale_bytes && (t.col % B) == 0) sbuf[(t.col % kTileCols) / B][(int)(r - t.tile_row)] = (uint8_t)byte;
        }
    }
    if (scale_bytes) {
        __syncthreads();
        store_tile_scales<NBLK>(sbuf, t, scale_bytes, rows_total, nb, block_major);
    }
    if (bad) raise_domain_flag(flag);
}


template <int FMT, int OUT, int NCOEF>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NCOEF == 1 ? 5 : 4)))
fq_weight_kernel(WeightJob j, int sb_log2, int e8m0_floor, int block_major, int code_slab, uint32_t *flag) {
    fq_weight_tile<FMT, OUT, NCOEF>(j, xcd_contiguous_tile(), sb_log2, e8m0_floor, block_major, code_slab, flag);
}

// The same for several layers in one launch: their tiles are numbered one layer after the other
// (layer l's from g.first[l]), so one grid covers them all.
template <int FMT, int OUT, int NCOEF>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NCOEF == 1 ? 5 : 4)))
fq_weight_group_kernel(WeightGroup g, int sb_log2, int e8m0_floor, int block_major, int code_slab, uint32_t *flag) {
    const uint32_t tile = xcd_contiguous_tile();
    int l = 0;
    for (int i = 1; i < g.n; i++) l = tile >= g.first[i] ? i : l;
    fq_weight_tile<FMT, OUT, NCOEF>(g.job[l], tile - g.first[l], sb_log2, e8m0_floor, block_major, code_slab, flag);
}

// fp32 weights (the 256-wide fp32 layer): one chunk per thread, true division per element.
template <int FMT, int OUT>
__global__ void __launch_bounds__(256)
fq_weight_f32_kernel(const void *__restrict__ W, uint32_t nchunks, int64_t row0, int64_t K,
                 const float *__restrict__ s_fp, const float *__restrict__ c, int sb_log2,
                 const float *__restrict__ alpha_ptr, int e8m0_floor, void *__restrict__ w_hat,
                 uint8_t *__restrict__ codes, uint8_t *__restrict__ scale_bytes, int64_t rows_total,
                 int block_major, int code_slab, uint32_t *flag) {
    constexpr int B = block_of(FMT);
    const float alpha = FMT == kFmtNV ? *alpha_ptr : 1.0f;
    const int sb = 1 << sb_log2;
    const int64_t nb = K / B;
    bool bad = false;
    const int64_t e_row0 = row0 * K;  // rows are contiguous: chunk t starts at element row0 K + 8 t
    for (uint32_t t = blockIdx.x * 256u + threadIdx.x; t < nchunks; t += gridDim.x * 256u) {
        const int64_t e0 = e_row0 + (int64_t)t * 8;
        float v[8];
        load8(W, kF32, e0, v);
        uint32_t byte;
        const float sdq = weight_sdq(FMT, s_fp[e0 / B], alpha, e8m0_floor, byte, bad);
        float cv[4] = {1.0f, 1.0f, 1.0f, 1.0f};
        const int ncoef = sb >= 8 ? 1 : 8 >> sb_log2;
        if (c) {
            for (int i = 0; i < ncoef; i++) {
                cv[i] = c[(e0 >> sb_log2) + i];
                bad |= bad_coeff(cv[i]);
            }
        }
        float out[8];
        uint32_t packed = 0;
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const float ci = sb >= 8 ? cv[0] : cv[i >> sb_log2];
            const float sq = sdq * ci;
            Quantized z = quantize_element(v[i], sq, sdq, true);
            out[i] = z.xhat;
            packed |= z.code << (4 * i);
        }
        if (w_hat) store8(w_hat, OUT, e0, out);
        if (codes) *reinterpret_cast<uint32_t *>(codes + (code_slab ? code_word_off(e0 / K, e0 % K, K, rows_total, 1) : e0 / 2)) = packed;
        if (scale_bytes && (e0 % B) == 0) {
            const int64_t row = e0 / K, blk = (e0 - row * K) / B;
            scale_bytes[block_major ? blk * rows_total + row : row * nb + blk] = (uint8_t)byte;
        }
    }
    if (bad) raise_domain_flag(flag);
}

// ------------------------------------------------------------------------------------------------
// K2 (MXFP4): dynamic activation fake quantisation, one pass. Block of 32 = 4 lanes.
// S = 2^e with e = E8M0_up(fl32(amax / 6)), or with e8m0_floor the OCP rule e = floor(log2 amax) - 2;
// u = x / S is computed as x * 2^-e, which is the same correctly rounded value because 2^-e is exact
// for every e in [-127, 127].
template <int OUT>
__global__ void __launch_bounds__(256)
fq_act_mx_kernel(const void *__restrict__ X, int64_t row0, int64_t rows, int64_t K, uint32_t ctiles,
                      void *__restrict__ x_hat, uint8_t *__restrict__ codes, uint8_t *__restrict__ scale_bytes,
                      int64_t rows_total, int block_major, int code_slab, int e8m0_floor, uint32_t *flag) {
    constexpr int NBLK = kTileCols / 32;
    __shared__ uint8_t sbuf[NBLK][kTileRows];
    const Tile t = tile_of<32>(row0, rows, K, ctiles);
    // packed-code word of the thread's chunk 0, and the step to its next chunk (8 rows further)
    const int64_t cw0 = code_word_off(t.row, t.col, K, rows_total, code_slab);
    const int64_t cws = code_slab ? (int64_t)kRowStep * 64 : (int64_t)kRowStep * K / 2;
    bool bad = false;
    uint4 raw[kChunks];
#pragma unroll
    for (int i = 0; i < kChunks; i++) raw[i] = load_chunk_bf16(X, t, K, i);
#pragma unroll
    for (int i = 0; i < kChunks; i++) {
        const int64_t r = t.row + (int64_t)i * kRowStep;
        const bool ok = t.col_ok && r < t.row_end;
        float v[8];
        unpack_bf16(raw[i], v);
        float amax = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; e++) amax = fmaxf(amax, __builtin_fabsf(v[e]));
        amax = group_max(amax, 4);
        bool nan_seen = false;
        const int e = e8m0_floor ? e8m0_floor_exp(amax, 2, nan_seen) : e8m0_ceil_exp(amax / 6.0f, nan_seen);
        if (ok) bad |= nan_seen;
        const float S = exp2i(e), inv = exp2i(-e);
        // u = x 2^-e has the sign of x, so the hardware code's sign bit is the code's; element i
        // lands in nibble i
        uint32_t packed = e2m1_code2<0>(0u, v[0] * inv, v[1] * inv);
        packed = e2m1_code2<1>(packed, v[2] * inv, v[3] * inv);
        packed = e2m1_code2<2>(packed, v[4] * inv, v[5] * inv);
        packed = e2m1_code2<3>(packed, v[6] * inv, v[7] * inv);
        if (ok) {
            const int64_t e0 = r * K + t.col;
            if (x_hat) {
                float out[8];
                e2m1_value2<0>(packed, out[0], out[1]);
                e2m1_value2<1>(packed, out[2], out[3]);
                e2m1_value2<2>(packed, out[4], out[5]);
                e2m1_value2<3>(packed, out[6], out[7]);
#pragma unroll
                for (int k = 0; k < 8; k++) out[k] *= S;
                store8_stream(x_hat, OUT, e0, out);
            }
            if (codes) store_code_word(codes + cw0 + i * cws, packed);
            if (scale_bytes && (t.col % 32) == 0) sbuf[(t.col % kTileCols) / 32][(int)(r - t.tile_row)] = (uint8_t)(e + 127);
        }
    }
    if (scale_bytes) {
        __syncthreads();
        store_tile_scales<NBLK>(sbuf, t, scale_bytes, rows_total, K / 32, block_major);
    }
    if (bad) raise_domain_flag(flag);
}

// fp32 activations: one chunk per thread (the same arithmetic).
template <int OUT>
__global__ void __launch_bounds__(256)
fq_act_mx_f32_kernel(const void *__restrict__ X, uint32_t nchunks, int64_t row0, int64_t K,
                 void *__restrict__ x_hat, uint8_t *__restrict__ codes, uint8_t *__restrict__ scale_bytes,
                 int64_t rows_total, int block_major, int code_slab, int e8m0_floor, uint32_t *flag) {
    const int64_t e_row0 = row0 * K;
    bool bad = false;
    for (uint32_t t = blockIdx.x * 256u + threadIdx.x; t < nchunks; t += gridDim.x * 256u) {
        const int64_t e0 = e_row0 + (int64_t)t * 8;
        float v[8];
        load8(X, kF32, e0, v);
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = fmaxf(amax, __builtin_fabsf(v[i]));
        amax = group_max(amax, 4);
        const int e = e8m0_floor ? e8m0_floor_exp(amax, 2, bad) : e8m0_ceil_exp(amax / 6.0f, bad);
        const float S = exp2i(e), inv = exp2i(-e);
        uint32_t packed = e2m1_code2<0>(0u, v[0] * inv, v[1] * inv);
        packed = e2m1_code2<1>(packed, v[2] * inv, v[3] * inv);
        packed = e2m1_code2<2>(packed, v[4] * inv, v[5] * inv);
        packed = e2m1_code2<3>(packed, v[6] * inv, v[7] * inv);
        float out[8];
        e2m1_value2<0>(packed, out[0], out[1]);
        e2m1_value2<1>(packed, out[2], out[3]);
        e2m1_value2<2>(packed, out[4], out[5]);
        e2m1_value2<3>(packed, out[6], out[7]);
#pragma unroll
        for (int i = 0; i < 8; i++) out[i] *= S;
        if (x_hat) store8(x_hat, OUT, e0, out);
        if (codes) *reinterpret_cast<uint32_t *>(codes + (code_slab ? code_word_off(e0 / K, e0 % K, K, rows_total, 1) : e0 / 2)) = packed;
        if (scale_bytes && (t & 3u) == 0) {
            const int64_t row = e0 / K, blk = (e0 - row * K) / 32;
            scale_bytes[block_major ? blk * rows_total + row : row * (K / 32) + blk] = (uint8_t)(e + 127);
        }
    }
    if (bad) raise_domain_flag(flag);
}

// ------------------------------------------------------------------------------------------------
// Absmax of a whole tensor, pass 1: one partial maximum per workgroup (max is order-free, so the
// result is exact and deterministic).
template <int IN>
__global__ void __launch_bounds__(256)
absmax_partial_kernel(const void *__restrict__ X, uint64_t nchunks, float *__restrict__ partial) {
    float m = 0.0f;
    for (uint64_t t = (uint64_t)blockIdx.x * 256u + threadIdx.x; t < nchunks; t += (uint64_t)gridDim.x * 256u) {
        float v[8];
        load8(X, IN, (int64_t)t * 8, v);
#pragma unroll
        for (int i = 0; i < 8; i++) m = fmaxf(m, __builtin_fabsf(v[i]));
    }
    __shared__ float red[256];
    red[threadIdx.x] = m;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    if (threadIdx.x == 0) partial[blockIdx.x] = red[0];
}

// pass 2 helper: every workgroup folds the partials into the tensor scale
// alpha = fl32(max|X| / (6 * 448)) (Eq. 2), or 1 for an all-zero tensor
__device__ float tensor_alpha_from_partials(const float *__restrict__ partial, int npart) {
    __shared__ float red[256];
    float m = 0.0f;
    for (int i = threadIdx.x; i < npart; i += 256) m = fmaxf(m, partial[i]);
    red[threadIdx.x] = m;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    const float A = red[0];
    return A > 0.0f ? A / 2688.0f : 1.0f;
}

// pass 2 of the NVFP4 tensor scale: one workgroup folds the partial maxima once, into a workspace
// slot that the elementwise kernels read (and into alpha_out when given)
__global__ void __launch_bounds__(256)
tensor_alpha_kernel(const float *__restrict__ partial, int npart, float *__restrict__ alpha_slot,
                    float *__restrict__ alpha_out) {
    const float a = tensor_alpha_from_partials(partial, npart);
    if (threadIdx.x == 0) {
        *alpha_slot = a;
        if (alpha_out) *alpha_out = a;
    }
}

// K2 (NVFP4) pass 2: block of 16 = 2 lanes; Delta = Q_E4M3(fl32(amax / fl32(alpha * 6))),
// S = fl32(alpha * Delta), u = fl32(x / S): S is not a power of two, so u comes from one correctly
// rounded reciprocal per block and div_by_scale when the wave's operands are in its range, else from a
// true division.
template <int OUT>
__global__ void __launch_bounds__(256)
fq_act_nv_kernel(const void *__restrict__ X, int64_t row0, int64_t rows, int64_t K, uint32_t ctiles,
                 const float *__restrict__ alpha_slot, void *__restrict__ x_hat, uint8_t *__restrict__ codes,
                 uint8_t *__restrict__ scale_bytes, int64_t rows_total, int block_major, int code_slab, uint32_t *flag) {
    constexpr int NBLK = kTileCols / 16;
    __shared__ uint8_t sbuf[NBLK][kTileRows];
    const Tile t = tile_of<16>(row0, rows, K, ctiles);
    // packed-code word of the thread's chunk 0, and the step to its next chunk (8 rows further)
    const int64_t cw0 = code_word_off(t.row, t.col, K, rows_total, code_slab);
    const int64_t cws = code_slab ? (int64_t)kRowStep * 64 : (int64_t)kRowStep * K / 2;
    const float alpha = *alpha_slot;
    const float alpha6 = alpha * 6.0f;
    bool bad = false;
    uint4 raw[kChunks];
#pragma unroll
    for (int i = 0; i < kChunks; i++) raw[i] = load_chunk_bf16(X, t, K, i);
#pragma unroll
    for (int i = 0; i < kChunks; i++) {
        const int64_t r = t.row + (int64_t)i * kRowStep;
        const bool ok = t.col_ok && r < t.row_end;
        float v[8];
        unpack_bf16(raw[i], v);
        float amax = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; e++) amax = fmaxf(amax, __builtin_fabsf(v[e]));
        amax = group_max(amax, 2);
        bool nan_seen = false;
        const uint32_t byte = e4m3_code(amax / alpha6, nan_seen);
        if (ok) bad |= nan_seen;
        const float S = alpha * e4m3_value(byte);
        const float y = 1.0f / S;
        const bool fast = bf16x8_over_2p80(raw[i]) == 0u && scale_in_fast_range(S);
        uint32_t packed;
        if (__all(fast || !ok)) {
            float u[8];
#pragma unroll
            for (int e = 0; e < 8; e++) u[e] = div_by_scale(v[e], S, y);
            packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, u[0], u[1], 1.0f, 0);
            packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, u[2], u[3], 1.0f, 1);
            packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, u[4], u[5], 1.0f, 2);
            packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, u[6], u[7], 1.0f, 3);
        } else {
            packed = 0u;
#pragma unroll
            for (int e = 0; e < 8; e++) packed |= quantize_element(v[e], S, S, true).code << (4 * e);
        }
        if (ok) {
            const int64_t e0 = r * K + t.col;
            if (x_hat) {
                float out[8];
                e2m1_value2<0>(packed, out[0], out[1]);
                e2m1_value2<1>(packed, out[2], out[3]);
                e2m1_value2<2>(packed, out[4], out[5]);
                e2m1_value2<3>(packed, out[6], out[7]);
#pragma unroll
                for (int e = 0; e < 8; e++) out[e] *= S;
                store8_stream(x_hat, OUT, e0, out);
            }
            if (codes) store_code_word(codes + cw0 + i * cws, packed);
            if (scale_bytes && (t.col % 16) == 0) sbuf[(t.col % kTileCols) / 16][(int)(r - t.tile_row)] = (uint8_t)byte;
        }
    }
    if (scale_bytes) {
        __syncthreads();
        store_tile_scales<NBLK>(sbuf, t, scale_bytes, rows_total, K / 16, block_major);
    }
    if (bad) raise_domain_flag(flag);
}

// fp32 activations: one chunk per thread, true division per element.
template <int OUT>
__global__ void __launch_bounds__(256)
fq_act_nv_f32_kernel(const void *__restrict__ X, uint32_t nchunks, int64_t row0, int64_t K,
                     const float *__restrict__ alpha_slot, void *__restrict__ x_hat, uint8_t *__restrict__ codes,
                     uint8_t *__restrict__ scale_bytes, int64_t rows_total, int block_major, int code_slab, uint32_t *flag) {
    const float alpha = *alpha_slot;
    const float alpha6 = alpha * 6.0f;
    const int64_t e_row0 = row0 * K;  // rows are contiguous: chunk t starts at e_row0 + 8 t
    bool bad = false;
    for (uint32_t t = blockIdx.x * 256u + threadIdx.x; t < nchunks; t += gridDim.x * 256u) {
        const int64_t e0 = e_row0 + (int64_t)t * 8;
        float v[8];
        load8(X, kF32, e0, v);
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = fmaxf(amax, __builtin_fabsf(v[i]));
        amax = group_max(amax, 2);
        const uint32_t byte = e4m3_code(amax / alpha6, bad);
        const float S = alpha * e4m3_value(byte);
        float out[8];
        uint32_t packed = 0;
#pragma unroll
        for (int i = 0; i < 8; i++) {
            Quantized z = quantize_element(v[i], S, S, true);
            out[i] = z.xhat;
            packed |= z.code << (4 * i);
        }
        if (x_hat) store8(x_hat, OUT, e0, out);
        if (codes) *reinterpret_cast<uint32_t *>(codes + (code_slab ? code_word_off(e0 / K, e0 % K, K, rows_total, 1) : e0 / 2)) = packed;
        if (scale_bytes && (t & 1u) == 0) {
            const int64_t row = e0 / K, blk = (e0 - row * K) / 16;
            scale_bytes[block_major ? blk * rows_total + row : row * (K / 16) + blk] = (uint8_t)byte;
        }
    }
    if (bad) raise_domain_flag(flag);
}

// ------------------------------------------------------------------------------------------------
// Straight-through backward of the dynamic activation fake quantisation (Sec. 3.2: STE on every
// non-differentiable operation): dX = m * dX_hat, m the clamp mask [|x / S| <= 6] (1 everywhere when
// ste_clip is 0; 0 in a block whose scale is zero), with the block scale S recomputed exactly as the
// forward forms it. The absmax scale passes no gradient. Under the paper's rounded-up E8M0, |x| <=
// amax <= 6 S, so every MXFP4 mask is 1; the OCP floor rule and NVFP4's rounded E4M3 scale can clip.
template <int FMT, int IN, int GD>
__global__ void __launch_bounds__(256)
fq_act_bwd_kernel(const void *__restrict__ X, uint32_t nchunks, int64_t row0, int64_t K,
                  const float *__restrict__ alpha_slot, int e8m0_floor, int ste_clip,
                  const void *__restrict__ dX_hat, void *__restrict__ dX) {
    constexpr int B = block_of(FMT);
    const float alpha = FMT == kFmtNV ? *alpha_slot : 1.0f;
    const int64_t e_row0 = row0 * K;
    for (uint32_t t = blockIdx.x * 256u + threadIdx.x; t < nchunks; t += gridDim.x * 256u) {
        const int64_t e0 = e_row0 + (int64_t)t * 8;
        float v[8], g[8];
        load8(X, IN, e0, v);
        load8(dX_hat, GD, e0, g);
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = fmaxf(amax, __builtin_fabsf(v[i]));
        amax = group_max(amax, B / 8);
        bool nan = false;
        float S;
        if (FMT == kFmtMX) {
            const int e = e8m0_floor ? e8m0_floor_exp(amax, 2, nan) : e8m0_ceil_exp(amax / 6.0f, nan);
            S = exp2i(e);
        } else {
            S = alpha * e4m3_value(e4m3_code(amax / (alpha * 6.0f), nan));
        }
        float out[8];
#pragma unroll
        for (int i = 0; i < 8; i++) out[i] = quantize_element(v[i], S, S, ste_clip != 0).m ? g[i] : 0.0f;
        store8(dX, GD, e0, out);
    }
}

// ------------------------------------------------------------------------------------------------
// K8: absmax initialisation (Sec. 3.2). MXFP4: s = fl32(amax / 6) (E8M0 rounded up), or fl32(amax / 4)
// with the OCP floor rule, whose E8M0 is then floor(log2 amax) - 2. NVFP4: Delta_fp =
// fl32(amax / fl32(alpha * 6)) with alpha from the partial maxima; c = 1.
template <int FMT, int IN>
__global__ void __launch_bounds__(256)
scales_init_kernel(const void *__restrict__ W, uint32_t nchunks, uint32_t cpr, int64_t row0, int64_t K,
                   const float *__restrict__ alpha_slot, float *__restrict__ s_fp, float *__restrict__ c,
                   int sb_log2, int e8m0_floor, float *__restrict__ alpha_out) {
    constexpr int B = block_of(FMT);
    float alpha = 1.0f;
    if (FMT == kFmtNV) alpha = *alpha_slot;  // alpha_out was written with the slot
    else if (alpha_out && blockIdx.x == 0 && threadIdx.x == 0) *alpha_out = 1.0f;
    const int sb = 1 << sb_log2;
    (void)cpr;
    const int64_t e_row0 = row0 * K;  // rows are contiguous: chunk t starts at e_row0 + 8 t
    for (uint32_t t = blockIdx.x * 256u + threadIdx.x; t < nchunks; t += gridDim.x * 256u) {
        const int64_t e0 = e_row0 + (int64_t)t * 8;
        float v[8];
        load8(W, IN, e0, v);
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = fmaxf(amax, __builtin_fabsf(v[i]));
        amax = group_max(amax, B / 8);
        if ((e0 % B) == 0)
            s_fp[e0 / B] = FMT == kFmtMX ? (e8m0_floor ? amax / 4.0f : amax / 6.0f) : amax / (alpha * 6.0f);
        if (sb >= 8) {
            if ((e0 % sb) == 0) c[e0 >> sb_log2] = 1.0f;
        } else {
            for (int i = 0; i < (8 >> sb_log2); i++) c[(e0 >> sb_log2) + i] = 1.0f;
        }
    }
}

// ------------------------------------------------------------------------------------------------
// K3: straight-through backward from a given G = dL/dW_hat (fp32).
//   grad_c = -(1/c^2) sum_sub G m w ;  grad_s = f * sum_block G (q - m u)
template <int FMT, int WDT>
__global__ void __launch_bounds__(256)
fq_bwd_kernel(const float *__restrict__ G, uint32_t nchunks, uint32_t cpr, int64_t row0, int64_t K,
              const void *__restrict__ W, const float *__restrict__ s_fp, const float *__restrict__ c,
              int sb_log2, const float *__restrict__ alpha_ptr, int ste_clip, int e8m0_floor,
              float *__restrict__ grad_s, float *__restrict__ grad_c, uint32_t *flag) {
    constexpr int B = block_of(FMT);
    const float alpha = FMT == kFmtNV ? *alpha_ptr : 1.0f;
    const int sb = 1 << sb_log2;
    const int64_t nb = K / B, ns = K >> sb_log2;
    bool bad = false;
    (void)cpr, (void)nb, (void)ns;
    const int64_t e_row0 = row0 * K;  // rows are contiguous: chunk t starts at e_row0 + 8 t
    for (uint32_t t = blockIdx.x * 256u + threadIdx.x; t < nchunks; t += gridDim.x * 256u) {
        const int64_t e0 = e_row0 + (int64_t)t * 8;
        float w[8], g[8];
        load8(W, WDT, e0, w);
        load8(G, kF32, e0, g);
        uint32_t byte;
        const float sdq = weight_sdq(FMT, s_fp[e0 / B], alpha, e8m0_floor, byte, bad);
        float cv[4] = {1.0f, 1.0f, 1.0f, 1.0f};
        const int ncoef = sb >= 8 ? 1 : 8 >> sb_log2;
        if (c) {
            for (int i = 0; i < ncoef; i++) {
                cv[i] = c[(e0 >> sb_log2) + i];
                bad |= bad_coeff(cv[i]);
            }
        }
        float tc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        float ts = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const int ci = sb >= 8 ? 0 : (i >> sb_log2);
            const float sq = sdq * cv[ci];
            Quantized z = quantize_element(w[i], sq, sdq, ste_clip != 0);
            const float mw = z.m ? w[i] : 0.0f;
            const float mu = z.m ? z.u : 0.0f;
            tc[ci] += g[i] * mw;
            ts += g[i] * (z.q - mu);
        }
        if (sb >= 8) {
            const float s = group_sum(tc[0], sb / 8);
            if ((e0 % sb) == 0) grad_c[e0 >> sb_log2] = -s / (cv[0] * cv[0]);
        } else {
            for (int i = 0; i < ncoef; i++) grad_c[(e0 >> sb_log2) + i] = -tc[i] / (cv[i] * cv[i]);
        }
        const float s = group_sum(ts, B / 8);
        if ((e0 % B) == 0) grad_s[e0 / B] = FMT == kFmtNV ? s * alpha : s;
    }
    if (bad) raise_domain_flag(flag);
}

// ================================================================================================
// Host launchers
// ================================================================================================

// The chunk index of one launch stays below 2^31; longer tensors are launched in row ranges.
template <typename F>
static hipError_t for_row_ranges(int64_t rows, int64_t K, F &&launch) {
    const int64_t cpr = K / 8;
    const int64_t max_rows = std::max<int64_t>(1, (int64_t(1) << 30) / cpr);
    for (int64_t r0 = 0; r0 < rows; r0 += max_rows) {
        const int64_t nr = std::min(max_rows, rows - r0);
        const uint32_t nchunks = (uint32_t)(nr * cpr);
        // one chunk per thread: a full grid streams HBM faster than a capped grid-stride loop
        const uint32_t grid = (uint32_t)((nchunks + 255) / 256);
        launch(r0, nchunks, (uint32_t)cpr, grid);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

static int log2i(int v) {
    int l = 0;
    while ((1 << l) < v) l++;
    return l;
}

// Tiled launches: row ranges of whole 64-row tiles, each launch at most kMaxTiledGrid workgroups (its
// work-item count, 256 per workgroup, then stays below 2^32).
template <typename F>
static hipError_t for_tile_ranges(int64_t rows, int64_t K, F &&launch) {
    const uint32_t ct = col_tiles(K);
    const int64_t max_rows = std::max<int64_t>(1, (int64_t)kMaxTiledGrid / ct) * kTileRows;
    for (int64_t r0 = 0; r0 < rows; r0 += max_rows) {
        const int64_t nr = std::min(max_rows, rows - r0);
        const uint32_t grid = (uint32_t)((nr + kTileRows - 1) / kTileRows) * ct;
        launch(r0, nr, ct, grid);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_fq_weight(int fmt, int in_dt, int out_dt, const void *W, int64_t rows, int64_t K,
                            const float *s_fp, const float *c, int sb, const float *alpha, int e8m0_floor,
                            void *w_hat, uint8_t *codes, uint8_t *scale_bytes, int block_major, int code_slab,
                            uint32_t *flag, hipStream_t st) {
    const int sbl = log2i(sb);
    if (in_dt == kBF16) {
        return for_tile_ranges(rows, K, [&](int64_t r0, int64_t nr, uint32_t ct, uint32_t grid) {
            const WeightJob j{W, s_fp, c, alpha, w_hat, codes, scale_bytes, r0, nr, rows, K, ct};
#define FQW(F, O, NC) fq_weight_kernel<F, O, NC><<<grid, 256, 0, st>>>(j, sbl, e8m0_floor, block_major, code_slab, flag)
#define FQW_NC(F, O) if (sb >= 8) FQW(F, O, 1); else if (sb == 4) FQW(F, O, 2); else FQW(F, O, 4)
            if (fmt == kFmtMX) { if (out_dt == kBF16) FQW_NC(kFmtMX, kBF16); else FQW_NC(kFmtMX, kF32); }
            else { if (out_dt == kBF16) FQW_NC(kFmtNV, kBF16); else FQW_NC(kFmtNV, kF32); }
#undef FQW_NC
#undef FQW
        });
    }
    return for_row_ranges(rows, K, [&](int64_t r0, uint32_t n, uint32_t cpr, uint32_t grid) {
        (void)cpr;
#define FQW(F, O) fq_weight_f32_kernel<F, O><<<grid, 256, 0, st>>>(W, n, r0, K, s_fp, c, sbl, alpha, e8m0_floor, w_hat, codes, scale_bytes, rows, block_major, code_slab, flag)
        if (fmt == kFmtMX) { if (out_dt == kBF16) FQW(kFmtMX, kBF16); else FQW(kFmtMX, kF32); }
        else { if (out_dt == kBF16) FQW(kFmtNV, kBF16); else FQW(kFmtNV, kF32); }
#undef FQW
    });
}

hipError_t launch_fq_weight_group(int fmt, int in_dt, int out_dt, const WeightLayer *L, int n, int sb,
                                  int e8m0_floor, int block_major, int code_slab, uint32_t *flag, hipStream_t st) {
    auto one_by_one = [&]() {
        for (int i = 0; i < n; i++) {
            if (L[i].rows == 0 || L[i].K == 0) continue;
            const hipError_t e = launch_fq_weight(fmt, in_dt, out_dt, L[i].W, L[i].rows, L[i].K, L[i].s_fp, L[i].c, sb,
                                                  L[i].alpha, e8m0_floor, L[i].w_hat, L[i].codes, L[i].scale_bytes,
                                                  block_major, code_slab, flag, st);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    };
    if (in_dt != kBF16 || n > kMaxWeightLayers) return one_by_one();
    WeightGroup g{};
    int m = 0;
    uint64_t total = 0;
    for (int i = 0; i < n; i++) {
        if (L[i].rows == 0 || L[i].K == 0) continue;
        const uint32_t ct = col_tiles(L[i].K);
        g.job[m] = WeightJob{L[i].W, L[i].s_fp, L[i].c, L[i].alpha, L[i].w_hat, L[i].codes, L[i].scale_bytes,
                             0, L[i].rows, L[i].rows, L[i].K, ct};
        g.first[m] = (uint32_t)std::min<uint64_t>(total, kMaxTiledGrid);
        total += (uint64_t)((L[i].rows + kTileRows - 1) / kTileRows) * ct;
        m++;
    }
    if (m == 0) return hipSuccess;
    if (total > kMaxTiledGrid) return one_by_one();
    g.n = m;
    const uint32_t grid = (uint32_t)total;
    const int sbl = log2i(sb);
#define FQG(F, O, NC) fq_weight_group_kernel<F, O, NC><<<grid, 256, 0, st>>>(g, sbl, e8m0_floor, block_major, code_slab, flag)
#define FQG_NC(F, O) if (sb >= 8) FQG(F, O, 1); else if (sb == 4) FQG(F, O, 2); else FQG(F, O, 4)
    if (fmt == kFmtMX) { if (out_dt == kBF16) FQG_NC(kFmtMX, kBF16); else FQG_NC(kFmtMX, kF32); }
    else { if (out_dt == kBF16) FQG_NC(kFmtNV, kBF16); else FQG_NC(kFmtNV, kF32); }
#undef FQG_NC
#undef FQG
    return hipGetLastError();
}

// NVFP4 tensor scale: kAbsmaxParts partial maxima, then alpha into partial[kAbsmaxParts]
static hipError_t launch_tensor_alpha(int in_dt, const void *X, int64_t n, float *partial, float *alpha_out,
                                      hipStream_t st) {
    const uint64_t nchunks = (uint64_t)n / 8;
    if (in_dt == kBF16) absmax_partial_kernel<kBF16><<<kAbsmaxParts, 256, 0, st>>>(X, nchunks, partial);
    else absmax_partial_kernel<kF32><<<kAbsmaxParts, 256, 0, st>>>(X, nchunks, partial);
    tensor_alpha_kernel<<<1, 256, 0, st>>>(partial, kAbsmaxParts, partial + kAbsmaxParts, alpha_out);
    return hipGetLastError();
}

hipError_t launch_fq_act(int fmt, int in_dt, int out_dt, const void *X, int64_t rows, int64_t K,
                         void *x_hat, uint8_t *codes, uint8_t *scale_bytes, int block_major, int code_slab, int e8m0_floor,
                         float *alpha_out, float *partial, uint32_t *flag, hipStream_t st) {
    if (fmt == kFmtMX) {
        if (in_dt == kBF16)
            return for_tile_ranges(rows, K, [&](int64_t r0, int64_t nr, uint32_t ct, uint32_t grid) {
#define FQA(O) fq_act_mx_kernel<O><<<grid, 256, 0, st>>>(X, r0, nr, K, ct, x_hat, codes, scale_bytes, rows, block_major, code_slab, e8m0_floor, flag)
                if (out_dt == kBF16) FQA(kBF16); else FQA(kF32);
#undef FQA
            });
        return for_row_ranges(rows, K, [&](int64_t r0, uint32_t n, uint32_t cpr, uint32_t grid) {
            (void)cpr;
#define FQA(O) fq_act_mx_f32_kernel<O><<<grid, 256, 0, st>>>(X, n, r0, K, x_hat, codes, scale_bytes, rows, block_major, code_slab, e8m0_floor, flag)
            if (out_dt == kBF16) FQA(kBF16); else FQA(kF32);
#undef FQA
        });
    }
    hipError_t e = launch_tensor_alpha(in_dt, X, rows * K, partial, alpha_out, st);
    if (e != hipSuccess) return e;
    const float *slot = partial + kAbsmaxParts;
    if (in_dt == kBF16)
        return for_tile_ranges(rows, K, [&](int64_t r0, int64_t nr, uint32_t ct, uint32_t grid) {
#define FQN(O) fq_act_nv_kernel<O><<<grid, 256, 0, st>>>(X, r0, nr, K, ct, slot, x_hat, codes, scale_bytes, rows, block_major, code_slab, flag)
            if (out_dt == kBF16) FQN(kBF16); else FQN(kF32);
#undef FQN
        });
    return for_row_ranges(rows, K, [&](int64_t r0, uint32_t n, uint32_t cpr, uint32_t grid) {
        (void)cpr;
#define FQN(O) fq_act_nv_f32_kernel<O><<<grid, 256, 0, st>>>(X, n, r0, K, slot, x_hat, codes, scale_bytes, rows, block_major, code_slab, flag)
        if (out_dt == kBF16) FQN(kBF16); else FQN(kF32);
#undef FQN
    });
}

hipError_t launch_fq_act_bwd(int fmt, int in_dt, int g_dt, const void *X, int64_t rows, int64_t K, int e8m0_floor,
                             int ste_clip, const void *dX_hat, void *dX, float *partial, hipStream_t st) {
    const float *slot = partial + kAbsmaxParts;
    if (fmt == kFmtNV) {
        hipError_t e = launch_tensor_alpha(in_dt, X, rows * K, partial, nullptr, st);
        if (e != hipSuccess) return e;
    }
    return for_row_ranges(rows, K, [&](int64_t r0, uint32_t n, uint32_t cpr, uint32_t grid) {
        (void)cpr;
#define AB(F, I, G) fq_act_bwd_kernel<F, I, G><<<grid, 256, 0, st>>>(X, n, r0, K, slot, e8m0_floor, ste_clip, dX_hat, dX)
        if (fmt == kFmtMX) {
            if (in_dt == kBF16) { if (g_dt == kBF16) AB(kFmtMX, kBF16, kBF16); else AB(kFmtMX, kBF16, kF32); }
            else { if (g_dt == kBF16) AB(kFmtMX, kF32, kBF16); else AB(kFmtMX, kF32, kF32); }
        } else {
            if (in_dt == kBF16) { if (g_dt == kBF16) AB(kFmtNV, kBF16, kBF16); else AB(kFmtNV, kBF16, kF32); }
            else { if (g_dt == kBF16) AB(kFmtNV, kF32, kBF16); else AB(kFmtNV, kF32, kF32); }
        }
#undef AB
    });
}

hipError_t launch_scales_init(int fmt, int in_dt, const void *W, int64_t rows, int64_t K, float *s_fp,
                              float *c, int sb, int e8m0_floor, float *alpha_out, float *partial, hipStream_t st) {
    const int sbl = log2i(sb);
    if (fmt == kFmtNV) {
        hipError_t e = launch_tensor_alpha(in_dt, W, rows * K, partial, alpha_out, st);
        if (e != hipSuccess) return e;
    }
    const float *slot = partial + kAbsmaxParts;
    return for_row_ranges(rows, K, [&](int64_t r0, uint32_t n, uint32_t cpr, uint32_t grid) {
        float *ao = r0 == 0 && fmt == kFmtMX ? alpha_out : nullptr;
#define SI(F, I) scales_init_kernel<F, I><<<grid, 256, 0, st>>>(W, n, cpr, r0, K, slot, s_fp, c, sbl, e8m0_floor, ao)
        if (fmt == kFmtMX) { if (in_dt == kBF16) SI(kFmtMX, kBF16); else SI(kFmtMX, kF32); }
        else { if (in_dt == kBF16) SI(kFmtNV, kBF16); else SI(kFmtNV, kF32); }
#undef SI
    });
}

hipError_t launch_fq_bwd(int fmt, int w_dt, const float *G, int64_t rows, int64_t K, const void *W,
                         const float *s_fp, const float *c, int sb, const float *alpha, int ste_clip,
                         int e8m0_floor, float *grad_s, float *grad_c, uint32_t *flag, hipStream_t st) {
    const int sbl = log2i(sb);
    return for_row_ranges(rows, K, [&](int64_t r0, uint32_t n, uint32_t cpr, uint32_t grid) {
#define FQB(F, WD) fq_bwd_kernel<F, WD><<<grid, 256, 0, st>>>(G, n, cpr, r0, K, W, s_fp, c, sbl, alpha, ste_clip, e8m0_floor, grad_s, grad_c, flag)
        if (fmt == kFmtMX) { if (w_dt == kBF16) FQB(kFmtMX, kBF16); else FQB(kFmtMX, kF32); }
        else { if (w_dt == kBF16) FQB(kFmtNV, kBF16); else FQB(kFmtNV, kF32); }
#undef FQB
    });
}

}  // namespace focus
