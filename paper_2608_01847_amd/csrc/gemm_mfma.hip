// bf16 MFMA reconstruction GEMMs for gfx950 (v_mfma_f32_32x32x16_bf16, fp32 accumulation).
//
// Every kernel computes a 256 x 256 output tile per workgroup of 256 threads (four waves, 2 x 2,
// each owning 128 x 128 = 4 x 4 MFMA tiles of 32 x 32; one workgroup per CU), with one barrier per
// reduction step. Operand tiles go from memory straight into a ring of LDS stages with
// direct-to-LDS buffer loads (buffer_load ... lds), several steps ahead of the MFMAs:
//   forward : 32 of K per step (128 for packed MXFP4 operands) in 5 (4) stages;
//   backward: 32 tokens per step in 4 stages; with packed MXFP4 X_hat, 5 stages of dY, codes and
//             scale bytes, whose codes are converted to bf16 into 3 further stages.
// The fragments of each half-step (16 of the reduction) are read from LDS one whole step before
// their MFMAs, into one of three register sets that rotate over a three-step unrolled loop.
//
// MFMA operand layout (32x32x16): lane l holds 8 consecutive reduction values of row l % 32 of A
// (resp. column l % 32 of B), starting at reduction index 8 (l / 32). Accumulator register r of
// lane l holds C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].
//
// Forward:  C = X_hat W_hat^T (rows = tokens, columns = out features). X_hat [M][K] and
//           W_hat [N][K] are K-contiguous, so fragments are plain 16-byte LDS reads. The epilogue
//           forms D = C - Y_ref, dY = D * 2/(M N) and per-column sums of D^2: a lane owns one
//           column, so the column sums are in-lane plus one cross-lane add.
// Backward: C = X_hat^T dY (rows = in features k, columns = out features n), i.e. G^T with the
//           reduction over tokens. Both operands are token-major in memory and are staged as they
//           lie; transposing LDS reads (ds_read_b64_tr_b16) form the fragments. In the epilogue a
//           lane holds 4 consecutive k of one n per register group, so a sub-block of 8 is an
//           in-lane sum of 4 plus one exchange with lane l ^ 32, and a block of 32 is 16 in-lane
//           values plus the same exchange.
#include "gemm_common.h"

#include <utility>

namespace focus {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

namespace {

constexpr int kTile = 256;            // output tile edge
constexpr int kThreads = 256;         // four waves
constexpr int kLdsBytes = 160 * 1024; // LDS of one gfx950 CU

static_assert(kTile == kMfmaTileM && kTile == kMfmaTileN && kTile == kMfmaTileK, "tile geometry");

// Raw buffer resources: a load whose offset is at or past num_records returns zeros and a store
// there is dropped, so bounds are handled by the hardware range check instead of branches (an
// offset with bit 31 set is always past it, since num_records is kept below 2^31).
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, int64_t bytes) {
    const int64_t n = bytes < 0 ? 0 : (bytes > 0x7FFFFFFF ? 0x7FFFFFFF : bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)n, kRsrcWord3);
}



// ---- forward operand staging: direct-to-LDS buffer loads ---------------------------------------
// The forward operands are K-contiguous, so their tiles go from HBM / L2 straight into LDS with
// buffer_load_dwordx4 ... lds (no VGPR round trip, no LDS store instructions). A step covers 32
// of K; five 32 KB stages (the default) keep up to three steps' loads in flight while one step is
// computed and the next step's fragments are read.
constexpr int kFwdStep = 32;
constexpr int kFwdOpBytes = kTile * 64;   // 256 rows x 32 bf16 = 16 KB
constexpr int kFwdStageBytes = 2 * kFwdOpBytes;
#ifndef FOCUS_FWD_STAGES
#define FOCUS_FWD_STAGES 5
#endif
constexpr int kFwdStages = FOCUS_FWD_STAGES;
static_assert(kFwdStages >= 4 && kFwdStages * kFwdStageBytes <= kLdsBytes, "forward stages fit the LDS");

typedef __attribute__((address_space(3))) char lds_char;

// Row `row`'s xor key for the 64-byte-row tile: ((row >> 1) & 3) ^ ((row >> 3) & 1). A fragment
// read serves 8 or 16 consecutive rows of one logical chunk per cycle; with this key those rows
// land on distinct 16-byte slots of a 128- or 256-byte bank span.
__device__ __forceinline__ uint32_t fwd_key(uint32_t row) { return ((row >> 1) & 3u) ^ ((row >> 3) & 1u); }

// Byte offset of 16-byte chunk `chunk` (0..3) of row `row` in a 64-byte-row tile.
__device__ __forceinline__ uint32_t fwd_off(uint32_t row, uint32_t chunk) {
    return row * 64u + ((chunk ^ fwd_key(row)) << 4);
}

// A direct-to-LDS load writes lane L's 16 bytes at LDS byte 16 L from the instruction's base, so
// each wave fills 1 KB blocks: lane L of block q lands in row 16 q + L / 4, physical chunk L % 4,
// which must hold logical chunk (L % 4) ^ fwd_key(row). The key depends on row bits 1-3 only,
// i.e. on L alone, so one step offset serves all four blocks. Offsets are in bytes of a row of
// `pitch` bytes (2 K for bf16 operands, K / 2 for packed FP4 codes); each thread's offsets at the
// first step are fixed for the whole tile.
struct FwdDma {
    uint32_t lane_off[4];
    uint32_t cb;  // byte offset of this lane's chunk inside a step's 64 bytes of a row
    __device__ __forceinline__ void init(int64_t pitch, int wave, int lane) {
        cb = ((uint32_t)(lane & 3) ^ fwd_key((uint32_t)lane >> 2)) * 16u;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const uint32_t row = (wave * 4 + i) * 16 + (lane >> 2);
            lane_off[i] = row * (uint32_t)pitch + cb;
        }
    }
    // Offset bits of the step whose row bytes start at b0: chunks at or past the row end get bit
    // 31 set, so they are out of range and read as zeros (an arithmetic mask, not a branch).
    __device__ __forceinline__ uint32_t step_bad(int64_t pitch, int64_t b0) const {
        const int32_t lim = (int32_t)(pitch - b0);
        return ((uint32_t)(lim - 1 - (int32_t)cb) >> 31) << 31;
    }
    // Load i (0..3) of this wave for the step whose row bytes start at b0 = base.
    __device__ __forceinline__ void issue_one(__amdgpu_buffer_rsrc_t rs, uint32_t base, uint32_t bad,
                                              lds_char *dst, int wave, int i) const {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst + (wave * 4 + i) * 1024, 16,
                                                 (int)((lane_off[i] + base) | bad), 0, 0, 0);
    }
};

// Backward operands are token-major tiles, [32 tokens][256 columns] of bf16, staged as they lie
// in memory and transposed by the fragment reads. The 16-byte chunk index of a row is xor-ed with
// 4 (row & 3): a transposing read touches 4 rows x 64 contiguous bytes per 32 lanes, which then
// fall on 256 distinct bytes.
constexpr int kBwdStep = 32;                          // tokens per step
constexpr int kBwdRowBytes = kTile * 2;               // 256 columns of bf16
constexpr int kBwdOpBytes = kBwdStep * kBwdRowBytes;  // 16 KB
constexpr int kBwdStageBytes = 2 * kBwdOpBytes;
constexpr int kBwdStages = 4;
static_assert(kBwdStages * kBwdStageBytes <= kLdsBytes, "backward stages fit the LDS allocation");
static_assert(kMfmaTokenStep % kBwdStep == 0, "token ranges of a split are whole steps");

__device__ __forceinline__ uint32_t bwd_off(uint32_t r, uint32_t c) {
    return r * (uint32_t)kBwdRowBytes + (((c >> 3) ^ ((r & 3u) << 2)) << 4) + (c & 7u) * 2u;
}

// Block q (1 KB) of a backward tile holds token rows 2 q and 2 q + 1: lane L lands in row
// 2 q + L / 32, physical chunk L % 32, which holds logical chunk (L % 32) ^ (4 (row & 3)). A wave
// fills blocks 4 wave .. 4 wave + 3. Offsets are relative to the step's first token row and fixed
// for the whole tile; columns at or past C get bit 31 set and read as zeros, and rows at or past
// the end of the token range fall outside the step's resource.
struct BwdDma {
    uint32_t off[4];
    __device__ __forceinline__ void init(int64_t C, int64_t c0, int wave, int lane) {
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const uint32_t row = 2 * (wave * 4 + i) + (lane >> 5);
            const uint32_t chunk = (uint32_t)(lane & 31) ^ ((row & 3u) << 2);
            const uint32_t col = (uint32_t)c0 + chunk * 8;
            const uint32_t bad = ((uint32_t)((int32_t)C - 1 - (int32_t)col) >> 31) << 31;
            off[i] = ((row * (uint32_t)C + col) * 2u) | bad;
        }
    }
    // The resource of the step starting at token t0 of a [.., C] matrix (no rows past t_end).
    __device__ __forceinline__ static __amdgpu_buffer_rsrc_t step_rsrc(const uint16_t *base, int64_t C, int64_t t0,
                                                                     int64_t t_end) {
        const int64_t rows = t_end - t0 < kBwdStep ? t_end - t0 : kBwdStep;
        return make_rsrc(base + t0 * C, rows * C * 2);
    }
    __device__ __forceinline__ void issue_one(__amdgpu_buffer_rsrc_t rs, lds_char *dst, int wave, int i) const {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, dst + (wave * 4 + i) * 1024, 16, (int)off[i], 0, 0, 0);
    }
};

// s_waitcnt with vmcnt <= n (n < 64) and the LDS and export counters unconstrained
#define FOCUS_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (0x7 << 4) | (0xF << 8))

// Fragments of one k16 step: A rows / B columns of the wave's 128 x 128 sub-tile.
struct Frags {
    bf16x8_t a[4], b[4];
};

__device__ __forceinline__ void load_frags_fwd(Frags &f, const char *As, const char *Bs, int ks, int wm, int wn,
                                               int lane) {
    const uint32_t lr = lane & 31, lh = lane >> 5;
#pragma unroll
    for (int i = 0; i < 4; i++) {
        f.a[i] = *reinterpret_cast<const bf16x8_t *>(As + fwd_off(wm * 128 + i * 32 + lr, ks * 2 + lh));
        f.b[i] = *reinterpret_cast<const bf16x8_t *>(Bs + fwd_off(wn * 128 + i * 32 + lr, ks * 2 + lh));
    }
}

__device__ __forceinline__ void mma_frags(const Frags &f, f32x16_t (&acc)[4][4]) {
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
}

// Fragment of 32 operand rows (columns c .. c + 31 of a token-major tile) for the k16 step whose
// first token row is t0: lane l needs tokens t0 + 8 (l / 32) + 0..7 of column c + l % 32. A
// transposing read hands lane i of a 16-lane group element i % 4 of the 8-byte pieces addressed
// by lanes 4 e + i / 4 (e = 0..3); pointing lane j at row t0' + j / 4, columns c' + 4 (j % 4) .. + 3
// gives lane i tokens t0' .. t0' + 3 of column c' + i. Two reads (rows r and r + 4, the same
// swizzle) cover the 8 tokens.
//
// The reads are issued as inline assembly: the compiler's builtin for them carries no aliasing
// information, so the compiler would make every such read wait for all direct-to-LDS loads in
// flight (vmcnt(0)), draining the pipeline each step. The price is that the compiler does not
// track these reads: `tr_wait` must run before their registers are used, and it takes the
// fragments as operands so that no consumer can be scheduled above it.
typedef short i16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lds_addr(const char *p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char *)p;
}

template <int OFF>
__device__ __forceinline__ i16x4_t ds_read_tr(uint32_t addr) {
    i16x4_t r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}

// Two fp32 values rounded to bf16 (to nearest, ties to even) in one instruction: lo in bits 0-15,
// hi in bits 16-31. Written out because the toolchain in use miscompiles the two-element vector
// conversion for gfx950 (it converts the first element only).
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
    uint32_t r;
    asm("v_cvt_pk_bf16_f32 %0, %1, %2" : "=v"(r) : "v"(lo), "v"(hi));
    return r;
}

// Per-lane byte offset, inside a tile, of the lower read of the fragment at columns c (step 0).
__device__ __forceinline__ uint32_t tr_lane_off(uint32_t c, int lane) {
    const uint32_t j = lane & 15;
    const uint32_t cc = c + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
    const uint32_t r = 8 * (lane >> 5) + (j >> 2);
    return bwd_off(r, cc);
}

// Fragments of k16 step KS of a stage; a_off / b_off are the lanes' tr_lane_off of the four A
// and four B fragments (relative to the stage), base the stage's LDS address.
template <int KS>
__device__ __forceinline__ void load_frags_tr(Frags &f, uint32_t base, const uint32_t (&a_off)[4],
                                              const uint32_t (&b_off)[4]) {
    constexpr int kRow = KS * 16 * kBwdRowBytes;  // first token row of the k16 step
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const i16x4_t a_lo = ds_read_tr<kRow>(base + a_off[i]);
        const i16x4_t a_hi = ds_read_tr<kRow + 4 * kBwdRowBytes>(base + a_off[i]);
        const i16x4_t b_lo = ds_read_tr<kBwdOpBytes + kRow>(base + b_off[i]);
        const i16x4_t b_hi = ds_read_tr<kBwdOpBytes + kRow + 4 * kBwdRowBytes>(base + b_off[i]);
        const i16x4_t va[2] = {a_lo, a_hi}, vb[2] = {b_lo, b_hi};
        f.a[i] = __builtin_bit_cast(bf16x8_t, va);
        f.b[i] = __builtin_bit_cast(bf16x8_t, vb);
    }
}

__device__ __forceinline__ void tr_wait(Frags &f) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(f.a[0]), "+v"(f.a[1]), "+v"(f.a[2]), "+v"(f.a[3]), "+v"(f.b[0]), "+v"(f.b[1]),
                   "+v"(f.b[2]), "+v"(f.b[3]));
}

// The same for a set whose 16 reads were followed by other LDS operations: a wave's LDS operations
// complete in order, so once at most 15 are in flight the set has landed.
__device__ __forceinline__ void tr_wait15(Frags &f) {
    asm volatile("s_waitcnt lgkmcnt(15)"
                 : "+v"(f.a[0]), "+v"(f.a[1]), "+v"(f.a[2]), "+v"(f.a[3]), "+v"(f.b[0]), "+v"(f.b[1]),
                   "+v"(f.b[2]), "+v"(f.b[3]));
}

// Workgroups are dealt to the 8 XCDs round-robin (id % 8), each XCD with its own L2. Renumbering
// so that XCD x runs a contiguous block of tiles keeps tiles that share operand panels in one L2.
__device__ __forceinline__ uint32_t xcd_tile(uint32_t id, uint32_t count) {
    const uint32_t per = count / 8u;
    return id < per * 8u ? (id % 8u) * per + id / 8u : id;
}

// Position t of a rows x cols tile grid in grouped order: groups of `group` row-tiles (default 4)
// are walked column by column, so the ~32 workgroups an XCD runs at once cover about 4 x 8 tiles and
// share 4 row panels and 8 column panels instead of 1 and 32.
constexpr uint32_t kGroupRows = 4;
__device__ __forceinline__ void grouped_tile(uint32_t t, uint32_t rows, uint32_t cols, uint32_t &r, uint32_t &c,
                                             uint32_t group = kGroupRows) {
    const uint32_t per_group = group * cols;
    const uint32_t first = (t / per_group) * group;
    const uint32_t in_group = rows - first < group ? rows - first : group;
    const uint32_t u = t % per_group;
    r = first + u % in_group;
    c = u / in_group;
}

// Calls f(std::integral_constant<int, 0>) ... f(<N-1>): every accumulator index is then a
// compile-time constant, so the accumulators stay in registers.
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, Is...>) {
    (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

}  // namespace

// ------------------------------------------------------------------------------------------------
// Forward reconstruction GEMM, Y_hat = X_hat W_hat^T with the MSE epilogue (or the plain product).
// Operands are bf16 (MX == false) or packed MXFP4 (MX == true): codes (two per byte, even k in the low
// nibble; X row-major [M][K / 2], W in K-slabs [K / 128][N][64]) and block-major E8M0 scale bytes
// [K / 32][rows], exactly the values X_hat and W_hat hold under MXFP4, multiplied by the block-scaled
// FP4 MFMA. Both modes stage 64 bytes of each operand row per step (32 bf16 or 128 FP4 k), so the LDS
// geometry, swizzle, pipeline and epilogue are shared; in MX mode a step's W tile is one contiguous
// 16 KB run of its K-slab.
template <bool MSE, bool MX>
__global__ void __launch_bounds__(kThreads, 1)
fwd_mfma_kernel(const void *__restrict__ X, const void *__restrict__ W, const uint8_t *__restrict__ Xs,
                const uint8_t *__restrict__ Ws, int64_t M, int64_t N, int64_t K,
                const uint16_t *__restrict__ Yref, uint16_t *__restrict__ dY, float dscale,
                double *__restrict__ colpart, int tiles_n) {
    constexpr int S = MX ? 4 : kFwdStages;                          // LDS stages
    constexpr int kLoads = MX ? 10 : 8;                             // loads per slot per thread
    constexpr int kKStep = MX ? 128 : kFwdStep;                     // k per step
    constexpr int kScaleBytes = MX ? 2048 : 0;                      // per stage: [256][4] bytes X, then W
    constexpr int kStage = kFwdStageBytes + kScaleBytes;
    static_assert(S * kStage <= kLdsBytes, "forward stages fit the LDS");
    __shared__ __attribute__((aligned(16))) char smem[S * kStage];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6, wm = wave >> 1, wn = wave & 1;
    const int lr = lane & 31, lh = lane >> 5;
    uint32_t tm, tn;
    grouped_tile(xcd_tile(blockIdx.x, gridDim.x), gridDim.x / tiles_n, tiles_n, tm, tn);
    const int64_t m0 = (int64_t)tm * kTile, n0 = (int64_t)tn * kTile;

    f32x16_t acc[4][4];
    const f32x16_t zero = {};
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) acc[i][j] = zero;

    // S LDS stages, one step each. Load "slot" j fills stage j % S: for j < nk it is step j of the
    // operands; slots nk .. nk + 3 bring the four 64-row quarters of the Y_ref tile (zeros in the
    // plain mode), so the epilogue's input arrives while the last steps' MFMAs run. Every slot is
    // kLoads loads per thread, which is what the vmcnt waits below count on.
    lds_char *const lsm = (lds_char *)smem;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const int64_t pitch = MX ? K / 2 : K * 2;  // bytes of an operand row
    // MX scale loads: lane L brings rows 128 (L / 32) + 32 (L % 4) + 4 ((L / 4) % 8) .. + 3 of its wave's
    // block (a permutation of the 64 four-row words), see load_scales; sc_sel picks byte lr % 4 of a
    // word of the first block into byte 0 and of the second block into byte 2 (0x0c: a zero byte)
    const uint32_t sc_row = ((uint32_t)lane >> 5) * 128u + ((uint32_t)lane & 3u) * 32u + (((uint32_t)lane >> 2) & 7u) * 4u;
    const uint32_t sc_b = (uint32_t)lr & 3u;
    const uint32_t sc_sel = sc_b | 0x0C00u | ((4u + sc_b) << 16) | 0x0C000000u;
    FwdDma dma;  // X and W rows have the same length, so one set of offsets serves both (bf16; X codes)
    dma.init(pitch, wave_u, lane);
    // MX: step j's W tile is rows n0 .. n0 + 255 of K-slab j, 64 bytes each, one contiguous run; rows
    // past N are outside the resource and read as zeros
    FwdDma dmaw;
    dmaw.init(64, wave_u, lane);
    const char *const ws_base = static_cast<const char *>(W) + n0 * 64;
    const int64_t w_slab = N * 64;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(static_cast<const char *>(X) + m0 * pitch, (M - m0) * pitch);
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(static_cast<const char *>(W) + n0 * pitch, (N - n0) * pitch);
    // block-major scale bytes [K/32][rows]: a step's 4 blocks of the tile's 256 rows are 4 runs of 256
    // contiguous bytes per operand
    const __amdgpu_buffer_rsrc_t rxs = make_rsrc(Xs, MX ? (K / 32) * M : 0);
    const __amdgpu_buffer_rsrc_t rws = make_rsrc(Ws, MX ? (K / 32) * N : 0);
    const __amdgpu_buffer_rsrc_t r_none = make_rsrc(dY, 0);
    const __amdgpu_buffer_rsrc_t rs_y = make_rsrc(MSE ? Yref + m0 * N : dY, MSE ? (M - m0) * N * 2 : 0);
    const __amdgpu_buffer_rsrc_t rs_d = make_rsrc(dY + m0 * N, (M - m0) * N * 2);
    const uint32_t N32 = (uint32_t)N;  // offsets are below 256 * N * 2 < 2^31 (checked when chosen)
    const int64_t nk = (K + kKStep - 1) / kKStep;
    // Quarter q of the output tile holds tile rows q*32 + 0..31 and 128 + q*32 + 0..31 (local rows
    // 0..63), i.e. accumulator block i == q of every wave. In LDS a quarter is 64 rows of 512 bytes;
    // the 16-byte chunk index of row r is xor-ed with 2 (r % 4) ^ 4 ((r / 4) % 2): the transposing
    // reads of the epilogue (4 consecutive rows x 32 bytes per 16 lanes) then touch 8 distinct
    // chunk slots, and the 2-byte writes of rows r and r + 4 (the two lane halves) different banks.
    auto q_row = [](uint32_t rl, uint32_t q) { return (rl >> 5) * 128u + q * 32u + (rl & 31u); };
    auto q_key = [](uint32_t rl) { return ((rl & 3u) << 1) ^ (((rl >> 2) & 1u) << 2); };
    auto q_off = [&](uint32_t rl, uint32_t chunk) { return rl * 512u + ((chunk ^ q_key(rl)) << 4); };
    auto stage = [&](int sidx) { return lsm + sidx * kStage; };
    // Load i of slot j into stage st: loads 0-3 bring X rows, 4-7 W rows of an operand step, and in
    // MX mode 8 / 9 the scale bytes of block 4 j + wave of the tile's 256 X / W rows (a [4][256]
    // byte array per operand in the stage; lane L's 4 bytes, rows 4 L .. 4 L + 3, land at byte 4 L
    // of the wave's run). A Y_ref quarter is 32 one-KB blocks of two rows each, this wave filling
    // blocks 8 wave .. 8 wave + 7 (lane L of block b lands in local row 2 b + L / 32, physical chunk
    // L % 32); in MX mode its loads 8 and 9 are empty and only write zeros into the stage's scale
    // bytes. Scale rows past M or N belong to the next block (or past the array) and meet zero codes.
    auto issue_op = [&](lds_char *st, int64_t j, int i) {
        const uint32_t base = (uint32_t)j * 64u, bad = dma.step_bad(pitch, base);  // 64 row bytes per step
        if (i < 4) dma.issue_one(ra, base, bad, st, wave_u, i);
        else if (MX && i < 8)
            dmaw.issue_one(make_rsrc(ws_base + j * w_slab, (N - n0) * 64), 0u, 0u, st + kFwdOpBytes, wave_u, i - 4);
        else if (i < 8) dma.issue_one(rb, base, bad, st + kFwdOpBytes, wave_u, i - 4);
        else {
            const uint32_t blk = (uint32_t)j * 4u + wave_u;
            const uint32_t so = blk * (uint32_t)(i == 8 ? M : N) + (uint32_t)(i == 8 ? m0 : n0) + sc_row;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(i == 8 ? rxs : rws, st + kFwdStageBytes + (i - 8) * 1024 + wave_u * 256, 4,
                                                     (int)so, 0, 0, 0);
        }
    };
    auto issue_y = [&](lds_char *st, int64_t j, int i) {
        if (MX && i >= 8) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(r_none, st + kFwdStageBytes + (i - 8) * 1024 + wave_u * 256, 4, 0, 0, 0, 0);
            return;
        }
        const uint32_t q = (uint32_t)((j - nk) & 3);
        const uint32_t blk = wave_u * 8 + i, rl = 2 * blk + (lane >> 5);
        const uint32_t chunk = (uint32_t)(lane & 31) ^ q_key(rl);
        const uint32_t col = (uint32_t)n0 + chunk * 8;
        const uint32_t bad = ((uint32_t)((int32_t)N32 - 1 - (int32_t)col) >> 31) << 31;  // col >= N
        const uint32_t off = ((q_row(rl, q) * N32 + col) * 2u) | bad;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_y, st + blk * 1024, 16, (int)off, 0, 0, 0);
    };
    auto issue_slot = [&](int64_t j) {
        lds_char *st = stage((int)(j % S));
        if (j < nk) {
#pragma unroll
            for (int i = 0; i < kLoads; i++) issue_op(st, j, i);
        } else {
#pragma unroll
            for (int i = 0; i < kLoads; i++) issue_y(st, j, i);
        }
    };
    // MX mode: this lane's scales (rows of its X / W fragments) of a stage, byte 0 / 2 holding the
    // scale of the first / second 64 k it covers (lane half lh takes the odd 32-k block of each 64).
    // A fragment row is 32 h + 32 i + lr (h the wave's half of the tile, i = 0..3), and the scale
    // loads place the 4-byte words (4 consecutive rows of a block) so that the words of rows
    // 128 h + 32 i + 4 a .. + 3, i = 0..3, are adjacent: 16 bytes at (8 h + a) 16. A lane reads
    // those 16 bytes of its two blocks and picks byte lr % 4 of each word.
    auto load_scales = [&](const char *st, uint32_t (&sa)[4], uint32_t (&sb)[4]) {
        typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
        const char *sx = st + kFwdStageBytes + lh * 256;
        const char *sw = sx + 1024;
        const uint32_t qa = (uint32_t)(wm * 8 + (lr >> 2)) * 16u, qb = (uint32_t)(wn * 8 + (lr >> 2)) * 16u;
        const u32x4v xa = *reinterpret_cast<const u32x4v *>(sx + qa), xc = *reinterpret_cast<const u32x4v *>(sx + 512 + qa);
        const u32x4v wa = *reinterpret_cast<const u32x4v *>(sw + qb), wc = *reinterpret_cast<const u32x4v *>(sw + 512 + qb);
#pragma unroll
        for (int i = 0; i < 4; i++) {
            sa[i] = __builtin_amdgcn_perm(xc[i], xa[i], sc_sel);
            sb[i] = __builtin_amdgcn_perm(wc[i], wa[i], sc_sel);
        }
    };
    auto mfma = [&](auto i, auto j, const Frags &fr, const uint32_t (&sa)[4], const uint32_t (&sb)[4], auto half) {
        if constexpr (MX) {
            typedef int v4i __attribute__((ext_vector_type(4)));
            typedef int v8i __attribute__((ext_vector_type(8)));
            const v4i a4 = __builtin_bit_cast(v4i, fr.a[i]), b4 = __builtin_bit_cast(v4i, fr.b[j]);
            const v8i a8 = {a4[0], a4[1], a4[2], a4[3], 0, 0, 0, 0}, b8 = {b4[0], b4[1], b4[2], b4[3], 0, 0, 0, 0};
            constexpr int ops = decltype(half)::value * 2;
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, acc[i][j], 4, 4, ops, (int)sa[i], ops,
                                                                        (int)sb[j]);
        } else {
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr.a[i], fr.b[j], acc[i][j], 0, 0, 0);
        }
    };
#pragma unroll
    for (int s0 = 0; s0 < S - 1; s0++) issue_slot(s0);
    // Before the barrier of step kt, this thread's loads of slots up to kt + 1 have landed (only
    // slots kt + 2 .. kt + S - 2 may still be in flight); after it, everyone's have, so the first
    // fragments of step kt + 1 can be read while step kt's MFMAs run, and stage (kt - 1) % S,
    // whose fragments every wave read during step kt - 2 and used in step kt - 1, can be refilled
    // with slot kt + S - 1. A bare s_barrier:
    // __syncthreads would also wait for the loads still in flight.
    FOCUS_WAIT_VMCNT(kLoads * (S - 3));
    asm volatile("s_barrier" ::: "memory");
    // Fragments are read a whole step ahead, in three sets: step kt's two halves use sets X and Y,
    // both read during step kt - 1; after the barrier the free set Z takes step kt + 1's first half
    // (and MX its scales), and X, once its MFMAs are issued, step kt + 1's second half. Read half a
    // step ahead (two sets), the MFMAs waited for their fragments: three sets are 2-6% faster on the
    // hidden-8192 layers, bit-identical. The sets rotate with a period of three steps.
    Frags f, g, h;
    uint32_t sa[4], sb[4], na[4], nb[4];
    load_frags_fwd(f, smem, smem + kFwdOpBytes, 0, wm, wn, lane);
    load_frags_fwd(g, smem, smem + kFwdOpBytes, 1, wm, wn, lane);
    if constexpr (MX) load_scales(smem, na, nb);
    // One step (sc = kt % S). The loads of slot kt + S - 1 go out spread over the step's 32 MFMAs:
    // one after every fourth (operand loads 0-3 in the first half, 4-7 in the second; MX's scale
    // loads after the fourth MFMA of each half). Issued closer together they fill the texture
    // unit's queue, and a wave stalled on a full queue issues no MFMA (loads after every second
    // MFMA of the first half only: 4-7% slower). The scheduling barriers keep the compiler from
    // regrouping them. Stage (kt - 1) % S, which they fill, was last read in step kt - 2.
    auto issue_at = [&](lds_char *st, int64_t kt, int li, auto y_slot) {
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (decltype(y_slot)::value) issue_y(st, kt + S - 1, li);
        else issue_op(st, kt + S - 1, li);
        __builtin_amdgcn_sched_barrier(0);
    };
    auto step = [&](int64_t kt, int sc, auto y_slot, Frags &X, Frags &Y, Frags &Z) {
        FOCUS_WAIT_VMCNT(kLoads * (S - 3));
        asm volatile("s_barrier" ::: "memory");
        const int sn = sc == S - 1 ? 0 : sc + 1, sl = sc == 0 ? S - 1 : sc - 1;
        const char *An = smem + sn * kStage, *Bn = An + kFwdOpBytes;
        lds_char *st = stage(sl);
        if constexpr (MX) {
#pragma unroll
            for (int i = 0; i < 4; i++) sa[i] = na[i], sb[i] = nb[i];
        }
        load_frags_fwd(Z, An, Bn, 0, wm, wn, lane);
        if constexpr (MX) load_scales(An, na, nb);
        static_for<16>([&](auto idx) {
            constexpr int i = idx / 4, jj = idx % 4;
            mfma(std::integral_constant<int, i>{}, std::integral_constant<int, jj>{}, X, sa, sb, std::integral_constant<int, 0>{});
            if constexpr (idx % 4 == 1) issue_at(st, kt, idx / 4, y_slot);
            if constexpr (MX && idx == 3) issue_at(st, kt, 8, y_slot);
        });
        load_frags_fwd(X, An, Bn, 1, wm, wn, lane);
        static_for<16>([&](auto idx) {
            constexpr int i = idx / 4, jj = idx % 4;
            mfma(std::integral_constant<int, i>{}, std::integral_constant<int, jj>{}, Y, sa, sb, std::integral_constant<int, 1>{});
            if constexpr (idx % 4 == 1) issue_at(st, kt, 4 + idx / 4, y_slot);
            if constexpr (MX && idx == 3) issue_at(st, kt, 9, y_slot);
        });
    };
    auto nxt = [](int sc) { return sc == S - 1 ? 0 : sc + 1; };
    const int64_t n_op = nk > S - 1 ? nk - (S - 1) : 0;  // steps whose slot kt + S - 1 is an operand step
    int64_t kt = 0;
    int sc = 0;
    for (; kt + 3 <= n_op; kt += 3) {
        step(kt, sc, std::false_type{}, f, g, h);
        sc = nxt(sc);
        step(kt + 1, sc, std::false_type{}, h, f, g);
        sc = nxt(sc);
        step(kt + 2, sc, std::false_type{}, g, h, f);
        sc = nxt(sc);
    }
    // the last operand steps, then the sets renamed once so that the Y_ref steps (at most S - 1)
    // start from the loop's rotation and run as straight-line code (a rotation chosen at run time
    // in each of them made the compiler spill)
    if (kt < n_op) {
        step(kt, sc, std::false_type{}, f, g, h);
        sc = nxt(sc);
        kt++;
    }
    if (kt < n_op) {
        step(kt, sc, std::false_type{}, h, f, g);
        sc = nxt(sc);
        kt++;
        Frags t = f;  // (g, h, f) becomes (f, g, h)
        f = g, g = h, h = t;
    } else if (n_op % 3 == 1) {
        Frags t = f;  // (h, f, g) becomes (f, g, h)
        f = h, h = g, g = t;
    }
    static_for<S - 1>([&](auto r) {
        if (kt < nk) {
            constexpr int q = decltype(r)::value % 3;
            if constexpr (q == 0) step(kt, sc, std::true_type{}, f, g, h);
            else if constexpr (q == 1) step(kt, sc, std::true_type{}, h, f, g);
            else step(kt, sc, std::true_type{}, g, h, f);
            sc = nxt(sc);
            kt++;
        }
    });
    // quarters not yet issued (S == 4: the last one) go into stages whose steps every wave is done with
    if constexpr (S < 5) {
        asm volatile("s_barrier" ::: "memory");
        for (int64_t j = nk + S - 1; j <= nk + 3; j++) issue_slot(j);
    }

    // ---- epilogue, one quarter at a time: D = Y_hat - Y_ref, dY = D * dscale, column sums of D^2
    // Each lane reads its 16 Y values of an accumulator tile from LDS with four transposing reads
    // (4 consecutive rows of its column each), then writes the 16 dY values over them; the quarter
    // then leaves with coalesced 16-byte stores, which drain while the next quarter is processed.
    // Rows past M and columns past N hold zero accumulators and read Y_ref as zero, so they add
    // nothing to the column sums; their stores fall outside the resource and are dropped. D^2 is
    // summed per accumulator tile in fp32 (16 terms), then into the column's fp64 total. dY is
    // rounded to bf16 by the hardware conversion (round to nearest even).
    double csum[4] = {0.0, 0.0, 0.0, 0.0};
    // The epilogue is bound by vector instructions, so every LDS address is a per-lane offset
    // computed once here plus the quarter's base and a constant: q_key(rl) depends on rl % 8 only,
    // so 8 more rows are 4096 bytes further, and two accumulator tiles further right (64 columns,
    // 8 chunks, which the key's 3 bits leave alone) are 128 bytes further.
    //  * dY writes of accumulator tile j, register r: row wm 32 + 8 (r / 4) + 4 lh + r % 4, column
    //    wn 128 + 32 j + lr: w_off[j % 2][r % 4] + 4096 (r / 4) + 128 (j / 2).
    //  * transposing Y_ref reads of tile j, row group g: the 16-lane group g16 covers rows
    //    4 (g16 / 2) .. + 3 of an 8-row group and columns 16 (g16 % 2) .. + 15 of the tile's 32;
    //    lane j16 of it points at row j16 / 4, columns 4 (j16 % 4) .. + 3 (see the backward's
    //    fragment reads): y_off[j % 2] + 4096 g + 128 (j / 2).
    //  * the quarter's coalesced stores: thread t moves chunk t % 32 of local rows t / 32 + 8 i
    //    (i = 0..7): LDS st_lds + 4096 i; memory st_mem + (q_row(8 i, q) - q_row(0, 0)) 2 N, the
    //    column bound folded into st_mem's bit 31 (rows past M fall outside the resource).
    const uint32_t g16 = (uint32_t)lane >> 4, j16 = (uint32_t)lane & 15u;
    uint32_t w_off[2][4], y_off[2];
#pragma unroll
    for (int jb = 0; jb < 2; jb++) {
        const uint32_t n = wn * 128 + jb * 32 + lr;
#pragma unroll
        for (int rr = 0; rr < 4; rr++) w_off[jb][rr] = q_off(wm * 32 + 4 * lh + rr, n >> 3) + (n & 7u) * 2u;
        const uint32_t col = wn * 128 + jb * 32 + 16 * (g16 & 1u) + 4 * (j16 & 3u);
        y_off[jb] = q_off(wm * 32 + 4 * (g16 >> 1) + (j16 >> 2), col >> 3) + (col & 7u) * 2u;
    }
    const uint32_t st_lds = q_off((uint32_t)t >> 5, (uint32_t)t & 31u);
    const uint32_t st_col = (uint32_t)n0 + ((uint32_t)t & 31u) * 8u;
    const uint32_t st_mem = (((uint32_t)t >> 5) * N32 + st_col) * 2u |
                            ((uint32_t)((int32_t)N32 - 1 - (int32_t)st_col) >> 31) << 31;  // col >= N
    typedef __attribute__((address_space(3))) uint16_t lds_u16;
    auto lds16 = [](uint32_t addr) { return reinterpret_cast<lds_u16 *>((uintptr_t)addr); };
    static_for<4>([&](auto q) {
        if (q == 0) {
            FOCUS_WAIT_VMCNT(3 * kLoads);  // this thread's loads of quarter 0 have landed
            asm volatile("s_barrier" ::: "memory");
        }
        const uint32_t qa = (uint32_t)(uintptr_t)stage((int)((nk + q) % S));  // the quarter's LDS address
        uint32_t wa[2][4];
#pragma unroll
        for (int jb = 0; jb < 2; jb++)
#pragma unroll
            for (int rr = 0; rr < 4; rr++) wa[jb][rr] = qa + w_off[jb][rr];
        static_for<4>([&](auto j) {
            constexpr uint32_t jo = 128u * (j / 2);
            float y[16];
            if constexpr (MSE) {
                const uint32_t ya = qa + y_off[j % 2];
                i16x4_t yv[4];
                static_for<4>([&](auto g) { yv[g] = ds_read_tr<4096 * g + jo>(ya); });
                asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(yv[0]), "+v"(yv[1]), "+v"(yv[2]), "+v"(yv[3]));
                static_for<16>([&](auto r) {
                    y[r] = __uint_as_float((uint32_t)(uint16_t)yv[r >> 2][r & 3] << 16);
                });
            }
            float sq = 0.0f;
            // two rows per conversion (round to nearest even, the low half from the first operand),
            // the halves stored by separate 2-byte writes
            static_for<8>([&](auto h) {
                constexpr int r0 = 2 * h, r1 = 2 * h + 1;
                float o0 = acc[q][j][r0], o1 = acc[q][j][r1];
                if constexpr (MSE) {
                    const float d0 = o0 - y[r0], d1 = o1 - y[r1];
                    sq = __builtin_fmaf(d0, d0, sq);
                    sq = __builtin_fmaf(d1, d1, sq);
                    o0 = d0 * dscale;
                    o1 = d1 * dscale;
                }
                const uint32_t pk = cvt_pk_bf16(o0, o1);
                *(lds16(wa[j % 2][r0 & 3]) + (4096u * (r0 >> 2) + jo) / 2) = (uint16_t)pk;
                *(lds16(wa[j % 2][r1 & 3]) + (4096u * (r1 >> 2) + jo) / 2) = (uint16_t)(pk >> 16);
            });
            csum[j] += (double)sq;
        });
        // After quarter 0 every thread waits for its remaining loads (no store has been issued
        // yet, so the count is exact); the barrier then makes all four quarters visible.
        if (q == 0) FOCUS_WAIT_VMCNT(0);
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 8; i++) {
            typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
            const u32x4 w = *reinterpret_cast<const __attribute__((address_space(3))) u32x4 *>(
                (uintptr_t)(qa + st_lds + 4096u * i));
            const uint32_t rows = (uint32_t)(i / 4) * 128u + (uint32_t)(i % 4) * 8u + (uint32_t)q * 32u;
            __builtin_amdgcn_raw_buffer_store_b128(w, rs_d, (int)(st_mem + rows * N32 * 2u), 0, 0);
        }
    });
    if (!MSE) return;
#pragma unroll
    for (int j = 0; j < 4; j++) csum[j] += __shfl_xor(csum[j], 32, 64);  // lanes l and l ^ 32 share a column
    double *red = reinterpret_cast<double *>(smem);                     // [2 waves along M][256 columns]
    __syncthreads();                                                    // every quarter has left LDS
    if (lh == 0) {
#pragma unroll
        for (int j = 0; j < 4; j++) red[wm * kTile + wn * 128 + j * 32 + lr] = csum[j];
    }
    __syncthreads();
    if (n0 + t < N) colpart[(int64_t)tm * N + n0 + t] = red[t] + red[kTile + t];
}

// Fused straight-through epilogue of the backward kernels on G^T = acc (a 256 k x 256 n tile):
// per-split partial sums of G m w per sub-block and of G (q - m u) per block.
// acc[i][j][r] is G[n][k] for n = n0 + 128 wn + 32 j + (lane % 32) and
// k = k0 + 128 wm + 32 i + 8 (r / 4) + 4 (lane / 32) + r % 4: lane l holds, for each group g of
// 8 k, the 4 consecutive k 4 (l / 32) .. + 3, and lanes l, l ^ 32 together hold the whole group.
template <int FMT, int WDT>
__device__ __forceinline__ void ste_epilogue(const f32x16_t (&acc)[4][4], int64_t k0, int64_t n0, int64_t split,
                                             int64_t N, int64_t K, const void *__restrict__ W,
                                             const float *__restrict__ s_fp, const float *__restrict__ c, int sb_log2,
                                             const float *__restrict__ alpha_ptr, int ste_clip, int e8m0_floor,
                                             float *__restrict__ part_s, float *__restrict__ part_c, uint32_t *flag,
                                             int wm, int wn, int lane) {
    constexpr int B = block_of(FMT);
    constexpr int NBI = 32 / B;                   // blocks per 32 k (1 MXFP4, 2 NVFP4)
    constexpr int WB = WDT == kBF16 ? 2 : 4;      // bytes per weight element
    const float alpha = FMT == kFmtNV ? *alpha_ptr : 1.0f;
    const int sb = 1 << sb_log2;
    const int64_t nb = K / B, ns = K >> sb_log2;
    const int lr = lane & 31, lh = lane >> 5;
    const bool has_c = c != nullptr;
    bool bad = false;
    // W, S_fp and c of the tile's rows come through range-checked buffer loads: rows past N read
    // as zeros, and so do columns past K (bit 31 of the offset). Out-of-range elements have G = 0
    // and w = 0 and add exactly zero to every sum; they are kept out of the domain check, and
    // their partial sums are not stored (bit 31 again: the store is dropped). All offsets are
    // 32-bit: a tile spans 256 rows of W (checked when the path is chosen).
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(reinterpret_cast<const char *>(W) + n0 * K * WB, (N - n0) * K * WB);
    const __amdgpu_buffer_rsrc_t rsf = make_rsrc(s_fp + n0 * nb, (N - n0) * nb * 4);
    const __amdgpu_buffer_rsrc_t rc = make_rsrc(has_c ? c + n0 * ns : s_fp, has_c ? (N - n0) * ns * 4 : 0);
    const __amdgpu_buffer_rsrc_t rps = make_rsrc(part_s + (split * N + n0) * nb, (N - n0) * nb * 4);
    const __amdgpu_buffer_rsrc_t rpc = make_rsrc(part_c + (split * N + n0) * ns, (N - n0) * ns * 4);
    const uint32_t K32 = (uint32_t)K, nb32 = (uint32_t)nb, ns32 = (uint32_t)ns;
    auto past = [&](uint32_t k) { return (uint32_t)(k >= K32) << 31; };  // k < 2^31 (K is)
    const uint32_t lh_drop = (uint32_t)lh << 31;  // stores made by the lane pair's lower lane only
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    static_for<4>([&](auto j) {
        const uint32_t nl = wn * 128 + j * 32 + lr;  // row of W inside the tile (< 256)
        const bool n_ok = n0 + nl < N;
        const uint32_t n_drop = (uint32_t)!n_ok << 31;
        // all loads of this column first
        float wv[4][4][4];   // [i][g][e]
        float sv[4][NBI];    // [i][block]
        float cv[4][4][2];   // [i][g][elements 0-1 / 2-3]
        static_for<4>([&](auto i) {
            const uint32_t kb = (uint32_t)k0 + wm * 128 + i * 32;
            static_for<4>([&](auto g) {
                const uint32_t k = kb + 8 * g + 4 * lh;  // this lane's 4 consecutive k
                const uint32_t wo = ((nl * K32 + k) * WB) | past(k);
                if constexpr (WDT == kBF16) {
                    const u32x2 p = __builtin_amdgcn_raw_buffer_load_b64(rw, (int)wo, 0, 0);
                    wv[i][g][0] = __uint_as_float(p.x << 16);
                    wv[i][g][1] = __uint_as_float(p.x & 0xFFFF0000u);
                    wv[i][g][2] = __uint_as_float(p.y << 16);
                    wv[i][g][3] = __uint_as_float(p.y & 0xFFFF0000u);
                } else {
                    const u32x4 p = __builtin_amdgcn_raw_buffer_load_b128(rw, (int)wo, 0, 0);
                    wv[i][g][0] = __uint_as_float(p.x);
                    wv[i][g][1] = __uint_as_float(p.y);
                    wv[i][g][2] = __uint_as_float(p.z);
                    wv[i][g][3] = __uint_as_float(p.w);
                }
                // coefficients of elements 0-1 and 2-3 (the same sub-block unless sb == 2); without
                // c the resource is empty and the select makes them 1
                const uint32_t c0 = ((nl * ns32 + (k >> sb_log2)) * 4u) | past(k);
                const float l0 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rc, (int)c0, 0, 0));
                float l1 = l0;  // a sub-block of 4 or more holds all four k (sb_log2 is uniform)
                if (sb_log2 == 1) {
                    const uint32_t c1 = ((nl * ns32 + ((k + 2) >> sb_log2)) * 4u) | past(k);
                    l1 = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rc, (int)c1, 0, 0));
                }
                cv[i][g][0] = has_c ? l0 : 1.0f;
                cv[i][g][1] = has_c ? l1 : 1.0f;
            });
            static_for<NBI>([&](auto h) {
                const uint32_t kh = kb + h * B;
                const uint32_t so = ((nl * nb32 + kh / B) * 4u) | past(kh);
                sv[i][h] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsf, (int)so, 0, 0));
            });
        });
        static_for<4>([&](auto i) {
            const uint32_t kb = (uint32_t)k0 + wm * 128 + i * 32;  // one MXFP4 / two NVFP4 blocks
            float sdq[NBI];
            static_for<NBI>([&](auto h) {
                bool nan = false;
                uint32_t byte;
                sdq[h] = weight_sdq(FMT, sv[i][h], alpha, e8m0_floor, byte, nan);
                bad = bad || (n_ok && kb + h * B < K32 && nan);
            });
            float tc[4][2];  // per group of 8 k: this lane's sums of G m w over elements 0-1 / 2-3
            float ts[4];     // per group of 8 k: this lane's sum of G (q - m u)
            static_for<4>([&](auto g) {
                const float sd = sdq[(8 * g) / B];
                const float cv0 = cv[i][g][0], cv1 = cv[i][g][1];
                bad = bad || (n_ok && kb + 8 * g < K32 && has_c && (bad_coeff(cv0) || bad_coeff(cv1)));
                tc[g][0] = tc[g][1] = ts[g] = 0.0f;
                static_for<4>([&](auto e) {
                    float a1, a2;
                    ste_terms(acc[i][j][(int)(4 * g + e)], wv[i][g][e], sd, e < 2 ? cv0 : cv1, ste_clip != 0, a1, a2);
                    tc[g][e >> 1] += a1;
                    ts[g] += a2;
                });
            });
            // ---- sub-block sums of G m w (scaled by -1/c^2 after the split reduction) ----
            if (sb <= 4) {
                // a sub-block lies inside one lane's 4 consecutive k
                static_for<4>([&](auto g) {
                    const uint32_t k = kb + 8 * g + 4 * lh;
                    const uint32_t drop = n_drop | past(k);
                    if (sb == 4) {
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(tc[g][0] + tc[g][1]), rpc,
                                                              (int)(((nl * ns32 + (k >> 2)) * 4u) | drop), 0, 0);
                    } else {
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(tc[g][0]), rpc,
                                                              (int)(((nl * ns32 + (k >> 1)) * 4u) | drop), 0, 0);
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(tc[g][1]), rpc,
                                                              (int)(((nl * ns32 + (k >> 1) + 1) * 4u) | drop), 0, 0);
                    }
                });
            } else {
                float s8[4];
                static_for<4>([&](auto g) {
                    s8[g] = tc[g][0] + tc[g][1];
                    s8[g] += __shfl_xor(s8[g], 32, 64);
                });
                const uint32_t drop = n_drop | lh_drop;
                if (sb == 8) {
                    static_for<4>([&](auto g) {
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(s8[g]), rpc,
                                                              (int)(((nl * ns32 + (kb >> 3) + g) * 4u) | drop | past(kb + 8 * g)), 0, 0);
                    });
                } else if (sb == 16) {
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(s8[0] + s8[1]), rpc,
                                                          (int)(((nl * ns32 + (kb >> 4)) * 4u) | drop | past(kb)), 0, 0);
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(s8[2] + s8[3]), rpc,
                                                          (int)(((nl * ns32 + (kb >> 4) + 1) * 4u) | drop | past(kb + 16)), 0, 0);
                } else {
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint((s8[0] + s8[1]) + (s8[2] + s8[3])), rpc,
                                                          (int)(((nl * ns32 + (kb >> 5)) * 4u) | drop | past(kb)), 0, 0);
                }
            }
            // ---- block sums of G (q - m u) ----
            float h0 = ts[0] + ts[1], h1 = ts[2] + ts[3];
            h0 += __shfl_xor(h0, 32, 64);
            h1 += __shfl_xor(h1, 32, 64);
            const uint32_t drop = n_drop | lh_drop;
            if constexpr (B == 32) {
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(h0 + h1), rps,
                                                      (int)(((nl * nb32 + (kb >> 5)) * 4u) | drop | past(kb)), 0, 0);
            } else {
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(h0), rps,
                                                      (int)(((nl * nb32 + (kb >> 4)) * 4u) | drop | past(kb)), 0, 0);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(h1), rps,
                                                      (int)(((nl * nb32 + (kb >> 4) + 1) * 4u) | drop | past(kb + 16)), 0, 0);
            }
        });
    });
    if (bad) raise_domain_flag(flag);
}

// ------------------------------------------------------------------------------------------------
template <int FMT, int WDT>
__global__ void __launch_bounds__(kThreads, 1)
bwd_mfma_kernel(const uint16_t *__restrict__ dY, const uint16_t *__restrict__ X, int64_t M, int64_t N, int64_t K,
                int64_t chunk, const void *__restrict__ W, const float *__restrict__ s_fp,
                const float *__restrict__ c, int sb_log2, const float *__restrict__ alpha_ptr, int ste_clip,
                int e8m0_floor, float *__restrict__ part_s, float *__restrict__ part_c, uint32_t *flag, int tiles_n) {
    __shared__ __attribute__((aligned(16))) char smem[kBwdStages * kBwdStageBytes];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6, wm = wave >> 1, wn = wave & 1;
    // linear id -> (split, tile): splits outermost, tiles of one split in grouped order, so that an
    // XCD's concurrent workgroups share the operand panels of one token range
    const uint32_t id = xcd_tile(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
    uint32_t tk, tn;
    grouped_tile(id % gridDim.x, gridDim.x / tiles_n, tiles_n, tk, tn);
    const int64_t k0 = (int64_t)tk * kTile, n0 = (int64_t)tn * kTile;
    const int64_t split = id / gridDim.x;
    const int64_t t_begin = split * chunk, t_end = std::min<int64_t>(M, t_begin + chunk);

    f32x16_t acc[4][4];
    const f32x16_t zero = {};
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) acc[i][j] = zero;

    // A = X_hat^T (rows = in features k), B = dY (columns = out features n), both staged as
    // token-major tiles. Four stages of 32 tokens, pipelined as in the forward kernel: slot j
    // (8 loads per thread) fills stage j % 4 with step j; slots past the token range are empty
    // resources whose loads only write zeros, which keeps every slot at 8 loads for the waits.
    lds_char *const lsm = (lds_char *)smem;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    BwdDma pa, pb;
    pa.init(K, k0, wave_u, lane);
    pb.init(N, n0, wave_u, lane);
    const int64_t nk = t_end > t_begin ? (t_end - t_begin + kBwdStep - 1) / kBwdStep : 0;
#pragma unroll
    for (int s0 = 0; s0 < kBwdStages - 1; s0++) {
        const int64_t t0 = t_begin + s0 * kBwdStep;
        const __amdgpu_buffer_rsrc_t ra = BwdDma::step_rsrc(X, K, t0, t_end), rb = BwdDma::step_rsrc(dY, N, t0, t_end);
        lds_char *st = lsm + s0 * kBwdStageBytes;
#pragma unroll
        for (int i = 0; i < 4; i++) pa.issue_one(ra, st, wave_u, i);
#pragma unroll
        for (int i = 0; i < 4; i++) pb.issue_one(rb, st + kBwdOpBytes, wave_u, i);
    }
    uint32_t a_off[4], b_off[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
        a_off[i] = tr_lane_off(wm * 128 + i * 32, lane);
        b_off[i] = tr_lane_off(wn * 128 + i * 32, lane);
    }
    const uint32_t lds0 = lds_addr(smem);
    FOCUS_WAIT_VMCNT(8);
    asm volatile("s_barrier" ::: "memory");
    // Fragments are read a whole step ahead in three rotating sets, as in bwd_mfma_mx_kernel: step
    // kt multiplies sets P and Q, filled during step kt - 1, and refills R and then P with step
    // kt + 1's halves.
    Frags f, g, h;
    load_frags_tr<0>(f, lds0, a_off, b_off);
    load_frags_tr<1>(g, lds0, a_off, b_off);
    auto step = [&](int64_t kt, Frags &P, Frags &Q, Frags &R) {
        const uint32_t nxt = lds0 + (uint32_t)((kt + 1) & 3) * kBwdStageBytes;
        const int64_t t0 = t_begin + (kt + 3) * kBwdStep;
        const __amdgpu_buffer_rsrc_t ra = BwdDma::step_rsrc(X, K, t0, t_end), rb = BwdDma::step_rsrc(dY, N, t0, t_end);
        lds_char *st = lsm + (int)((kt + 3) & 3) * kBwdStageBytes;
        // slot kt + 1 and this thread's reads of P have landed (only reads of Q may be in flight);
        // after the barrier everyone's have, and stage (kt - 1) % 4 is free for slot kt + 3
        FOCUS_WAIT_VMCNT(8);
        tr_wait15(P);
        asm volatile("s_barrier" ::: "memory");
        load_frags_tr<0>(R, nxt, a_off, b_off);
        // the 8 loads of slot kt + 3 go out one after every second MFMA (see the forward kernel)
        static_for<16>([&](auto idx) {
            constexpr int i = idx / 4, jj = idx % 4;
            acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(P.a[i], P.b[jj], acc[i][jj], 0, 0, 0);
            if constexpr (idx % 2 == 1) {
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (idx / 2 < 4) pa.issue_one(ra, st, wave_u, idx / 2);
                else pb.issue_one(rb, st + kBwdOpBytes, wave_u, idx / 2 - 4);
                __builtin_amdgcn_sched_barrier(0);
            }
        });
        tr_wait15(Q);  // read during step kt - 1
        load_frags_tr<1>(P, nxt, a_off, b_off);
        mma_frags(Q, acc);
    };
    int64_t kt = 0;
    for (; kt + 3 <= nk; kt += 3) {
        step(kt, f, g, h);
        step(kt + 1, h, f, g);
        step(kt + 2, g, h, f);
    }
    if (kt < nk) step(kt, f, g, h);
    if (kt + 1 < nk) step(kt + 1, h, f, g);
    tr_wait(f);  // no read may still be in flight when the workgroup ends
    // the empty slots' zero writes must land before the workgroup's LDS is handed on
    FOCUS_WAIT_VMCNT(0);
    ste_epilogue<FMT, WDT>(acc, k0, n0, split, N, K, W, s_fp, c, sb_log2, alpha_ptr, ste_clip, e8m0_floor, part_s,
                           part_c, flag, wm, wn, lane);
}

// ------------------------------------------------------------------------------------------------
// Backward reconstruction GEMM with X_hat given as packed MXFP4 (codes [M][K / 2], even k in the low
// nibble, and E8M0 bytes block-major [K / 32][M], the arrays focus_fakequant_fwd writes). Under
// MXFP4 X_hat is exactly an E2M1 code times its block's power of two (Eq. 1, 3), so the bf16 operand
// is rebuilt in LDS without loss, reading a quarter of the bytes of the bf16 X_hat. Same tile, MFMA
// and fused epilogue as bwd_mfma_kernel.
//
// Per 32-token step a DMA slot brings the dY tile (16 KB, the bf16 kernel's token-major layout), the
// step's codes ([32 tokens][128 bytes]) and its scale bytes ([8 blocks][32 tokens], one copy per
// wave so that every thread issues the same number of loads). Two steps after a slot's loads are
// issued, each thread converts one token's 32 codes of one block (16 bytes, one scale) into 32 bf16
// with the scaled FP4 conversion and writes them into one of three bf16 A stages, in the layout the
// transposing fragment reads expect. Step kt issues slot kt + 4, converts slot kt + 2, reads the
// fragments of step kt + 1 and multiplies step kt: 5 DMA stages + 3 A stages = 153 KB of LDS.
constexpr int kMxDmaStages = 5;
constexpr int kMxCodeOff = kBwdOpBytes;            // codes after the dY tile
constexpr int kMxScaleOff = kMxCodeOff + 32 * 128; // then 4 per-wave copies of the scale bytes
constexpr int kMxDmaStageBytes = kMxScaleOff + 4 * 256;
constexpr int kMxAStages = 3;
constexpr int kMxAOff = kMxDmaStages * kMxDmaStageBytes;
constexpr int kMxLdsBytes = kMxAOff + kMxAStages * kBwdOpBytes;
constexpr int kMxLoads = 6;  // loads per slot per thread: dY 4, codes 1, scales 1
static_assert(kMxLdsBytes <= kLdsBytes, "MXFP4 backward stages fit the LDS");

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <int OFF>
__device__ __forceinline__ u32x4_t ds_read_b128(uint32_t addr) {
    u32x4_t r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}

template <int OFF>
__device__ __forceinline__ uint32_t ds_read_u8(uint32_t addr) {
    uint32_t r;
    asm volatile("ds_read_u8 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}

__device__ __forceinline__ void ds_write_b128(uint32_t addr, u32x4_t v) {
    asm volatile("ds_write_b128 %0, %1" : : "v"(addr), "v"(v) : "memory");
}

// Waits until at most N LDS operations of this wave are in flight; the values read by the earlier
// ones are passed through so that no consumer is scheduled above the wait.
template <int N>
__device__ __forceinline__ void lds_wait(u32x4_t &a, uint32_t &b) {
    static_assert(N >= 0 && N < 16, "lgkmcnt is a 4-bit field");
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "i"(N));
}

// Byte offset of (token row r, column c) in an A stage of the MXFP4 backward: the bf16 kernel's
// token-major layout with one more xor on the 16-byte chunk index, by its 32-column block b:
// (b ^ b / 4) % 4. Within a block that is a fixed permutation of its 4 chunks, so the transposing
// fragment reads stay conflict-free; the conversion's 16-byte writes (8 lanes of one row, blocks
// 0-7, the same chunk of each block) then fall on 8 distinct 16-byte bank groups instead of 2.
__device__ __forceinline__ uint32_t mx_a_off(uint32_t r, uint32_t c) {
    const uint32_t ch = c >> 3, b = ch >> 2;
    return r * (uint32_t)kBwdRowBytes + ((ch ^ ((r & 3u) << 2) ^ ((b ^ (b >> 2)) & 3u)) << 4) + (c & 7u) * 2u;
}

// tr_lane_off for the A stages of the MXFP4 backward
__device__ __forceinline__ uint32_t mx_tr_lane_off(uint32_t c, int lane) {
    const uint32_t j = lane & 15;
    const uint32_t cc = c + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
    const uint32_t r = 8 * (lane >> 5) + (j >> 2);
    return mx_a_off(r, cc);
}

// a buffer resource of `bytes` (< 2^31) bytes
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc_u32(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRsrcWord3);
}

// buffer resources of one DMA slot of the MXFP4 backward
struct MxSlot {
    __amdgpu_buffer_rsrc_t rd, rc, rs;  // dY rows, code rows, scale bytes
    uint32_t t0;                        // the slot's first token
};

template <int WDT>
__global__ void __launch_bounds__(kThreads, 1)
bwd_mfma_mx_kernel(const uint16_t *__restrict__ dY, const uint8_t *__restrict__ Xc, const uint8_t *__restrict__ Xs,
                   int64_t M, int64_t N, int64_t K, int64_t chunk, const void *__restrict__ W,
                   const float *__restrict__ s_fp, const float *__restrict__ c, int sb_log2, int ste_clip,
                   int e8m0_floor, float *__restrict__ part_s, float *__restrict__ part_c, uint32_t *flag,
                   int tiles_n) {
    __shared__ __attribute__((aligned(16))) char smem[kMxLdsBytes];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6, wm = wave >> 1, wn = wave & 1;
    // groups of up to 10 k-tiles of equal size: the ~32 workgroups an XCD runs at once cover about
    // 8-10 k-tiles x 3-4 out-feature tiles, so each dY panel (four times the bytes of a packed X_hat
    // panel) is shared by 8-10 of them and each X_hat panel by 3-4
    const uint32_t id = xcd_tile(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
    const uint32_t tiles_k = gridDim.x / tiles_n, ngroups = (tiles_k + 9) / 10;
    uint32_t tk, tn;
    grouped_tile(id % gridDim.x, tiles_k, tiles_n, tk, tn, (tiles_k + ngroups - 1) / ngroups);
    const int64_t k0 = (int64_t)tk * kTile, n0 = (int64_t)tn * kTile;
    const int64_t split = id / gridDim.x;
    const int64_t t_begin = split * chunk, t_end = std::min<int64_t>(M, t_begin + chunk);

    f32x16_t acc[4][4];
    const f32x16_t zero = {};
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) acc[i][j] = zero;

    lds_char *const lsm = (lds_char *)smem;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    BwdDma pb;
    pb.init(N, n0, wave_u, lane);
    const int64_t kc = K / 2;  // code bytes per token row
    // this lane's code chunk: token row 8 wave + lane / 8 of the step, 16 bytes = block lane % 8 of the tile
    const uint32_t c_row = 8u * wave_u + ((uint32_t)lane >> 3), c_blk = (uint32_t)lane & 7u;
    const uint32_t c_col = (uint32_t)(k0 / 2) + 16u * c_blk;
    const uint32_t c_off = (c_row * (uint32_t)kc + c_col) | ((uint32_t)((int32_t)kc - 1 - (int32_t)c_col) >> 31 << 31);
    // this lane's 4 scale bytes: block lane / 8 of the tile, tokens 4 (lane % 8) .. + 3 of the step
    const uint32_t s_blk = (uint32_t)(k0 / 32) + ((uint32_t)lane >> 3);
    const uint32_t s_bad = (uint32_t)((int32_t)(K / 32) - 1 - (int32_t)s_blk) >> 31 << 31;
    const uint32_t s_off = s_blk * (uint32_t)M + 4u * ((uint32_t)lane & 7u);
    const __amdgpu_buffer_rsrc_t rs_all = make_rsrc(Xs, (K / 32) * M), rs_none = make_rsrc(Xs, 0);
    const int64_t nk = t_end > t_begin ? (t_end - t_begin + kBwdStep - 1) / kBwdStep : 0;

    // The resources of the slot whose first token is t: the dY rows and code rows of its 32 tokens
    // (rows past the token range read as zeros; a slot past the range has empty resources, whose
    // loads write zeros) and the scale bytes (all blocks; offsets carry the slot's first token).
    auto slot_at = [&](int64_t t) {
        MxSlot sl;
        const int64_t rem = t_end - t;
        const uint32_t rows = rem <= 0 ? 0u : (rem < kBwdStep ? (uint32_t)rem : (uint32_t)kBwdStep);
        sl.rd = make_rsrc_u32(dY + t * N, rows * (uint32_t)N * 2u);
        sl.rc = make_rsrc_u32(Xc + t * kc, rows * (uint32_t)kc);
        sl.rs = rows ? rs_all : rs_none;
        sl.t0 = (uint32_t)t;
        return sl;
    };
    // load i (0..5) of a slot into the DMA stage at st: 0 the codes, 1 the scale bytes, 2-5 the dY
    // tile. The codes go first: loads complete in issue order, so waiting for a slot's codes leaves
    // its dY loads in flight (they are needed two steps later than the codes).
    auto issue = [&](lds_char *st, const MxSlot &sl, int i) {
        if (i == 0) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(sl.rc, st + kMxCodeOff + wave_u * 1024, 16, (int)c_off, 0, 0, 0);
        } else if (i == 1) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(sl.rs, st + kMxScaleOff + wave_u * 256, 4,
                                                     (int)((s_off + sl.t0) | s_bad), 0, 0, 0);
        } else {
            pb.issue_one(sl.rd, st, wave_u, i - 2);
        }
    };
    const uint32_t lds0 = lds_addr(smem);
    // conversion: this thread's 16 code bytes and scale byte of a DMA stage, 32 bf16 into an A stage
    const uint32_t cv_code = (uint32_t)kMxCodeOff + (uint32_t)wave_u * 1024u + 16u * (uint32_t)lane;
    const uint32_t cv_scale = (uint32_t)kMxScaleOff + (uint32_t)wave_u * 256u + 32u * c_blk + c_row;
    // write j: chunk j (k 8 j .. 8 j + 7) of this thread's block
    uint32_t cv_dst[4];
#pragma unroll
    for (int j = 0; j < 4; j++) cv_dst[j] = mx_a_off(c_row, 8u * (4u * c_blk + j));
    auto cvt_chunk = [&](uint32_t word, float sc, uint32_t dst) {
        u32x4_t v;
        v.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, sc, 0));
        v.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, sc, 1));
        v.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, sc, 2));
        v.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(word, sc, 3));
        ds_write_b128(dst, v);
    };
    auto scale_of = [](uint32_t byte) { return exp2i((int)(byte & 0xFFu) - 127); };
    auto d_addr = [&](int i) { return lds0 + (uint32_t)(i * kMxDmaStageBytes); };
    auto a_addr = [&](int i) { return lds0 + (uint32_t)(kMxAOff + i * kBwdOpBytes); };

    // prologue: slots 0-3 in flight, slots 0 and 1 converted into A stages 0 and 1
#pragma unroll
    for (int s0 = 0; s0 < 4; s0++) {
        const MxSlot sl = slot_at(t_begin + s0 * kBwdStep);
#pragma unroll
        for (int i = 0; i < kMxLoads; i++) issue(lsm + s0 * kMxDmaStageBytes, sl, i);
    }
    FOCUS_WAIT_VMCNT(2 * kMxLoads);
    asm volatile("s_barrier" ::: "memory");
#pragma unroll
    for (int s0 = 0; s0 < 2; s0++) {
        u32x4_t w = ds_read_b128<0>(d_addr(s0) + cv_code);
        uint32_t sb = ds_read_u8<0>(d_addr(s0) + cv_scale);
        lds_wait<0>(w, sb);
        const float sc = scale_of(sb);
        cvt_chunk(w.x, sc, a_addr(s0) + cv_dst[0]);
        cvt_chunk(w.y, sc, a_addr(s0) + cv_dst[1]);
        cvt_chunk(w.z, sc, a_addr(s0) + cv_dst[2]);
        cvt_chunk(w.w, sc, a_addr(s0) + cv_dst[3]);
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");

    uint32_t a_off[4], b_off[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
        a_off[i] = mx_tr_lane_off(wm * 128 + i * 32, lane);
        b_off[i] = tr_lane_off(wn * 128 + i * 32, lane);  // the dY tile opens its DMA stage
    }
    // A fragments live in an A stage, B fragments in a DMA stage: one base per operand
    auto frags = [&](auto ks, Frags &fr, uint32_t abase, uint32_t bbase) {
        constexpr int kRow = decltype(ks)::value * 16 * kBwdRowBytes;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const i16x4_t a_lo = ds_read_tr<kRow>(abase + a_off[i]);
            const i16x4_t a_hi = ds_read_tr<kRow + 4 * kBwdRowBytes>(abase + a_off[i]);
            const i16x4_t b_lo = ds_read_tr<kRow>(bbase + b_off[i]);
            const i16x4_t b_hi = ds_read_tr<kRow + 4 * kBwdRowBytes>(bbase + b_off[i]);
            const i16x4_t va[2] = {a_lo, a_hi}, vb[2] = {b_lo, b_hi};
            fr.a[i] = __builtin_bit_cast(bf16x8_t, va);
            fr.b[i] = __builtin_bit_cast(bf16x8_t, vb);
        }
    };
    // LDS offsets of the stages, rotated each step (no divisions in the loop): DMA stages of slots kt,
    // kt + 2 and kt + 4, A stages of steps kt and kt + 2
    uint32_t o_cur = 0, o_cv = 2 * kMxDmaStageBytes, o_is = 4 * kMxDmaStageBytes;
    uint32_t a_cur = kMxAOff, a_cv = kMxAOff + 2 * kBwdOpBytes;
    auto next_d = [](uint32_t o) { return o == (kMxDmaStages - 1) * kMxDmaStageBytes ? 0u : o + kMxDmaStageBytes; };
    auto next_a = [](uint32_t o) {
        return o == kMxAOff + (kMxAStages - 1) * kBwdOpBytes ? (uint32_t)kMxAOff : o + kBwdOpBytes;
    };
    // Fragments are read a whole step ahead, in three sets: step kt's two k16 halves use sets X and
    // Y, both filled during step kt - 1; after the barrier the free set Z takes step kt + 1's first
    // half, and X, once its MFMAs are issued, step kt + 1's second half. Read only half a step ahead
    // (two sets), the waits for the fragments stalled the matrix units: three sets are 5-7% faster
    // on the hidden-8192 layers, bit-identical. The sets rotate with a period of three steps, so the
    // loop is unrolled three times.
    Frags f, g, h;
    frags(std::integral_constant<int, 0>{}, f, a_addr(0), d_addr(0));
    frags(std::integral_constant<int, 1>{}, g, a_addr(0), d_addr(0));
    auto step = [&](int64_t kt, Frags &X, Frags &Y, Frags &Z) {
        const MxSlot sl = slot_at(t_begin + (kt + 4) * kBwdStep);
        lds_char *st = lsm + o_is;
        const uint32_t cds = lds0 + o_cv, cas = lds0 + a_cv;
        const uint32_t a_nx = lds0 + next_a(a_cur), o_nx = lds0 + next_d(o_cur);
        // this thread's codes and scale bytes of slot kt + 2 and all of slot kt + 1 have landed (slot
        // kt + 3 and the dY loads of slot kt + 2 may be in flight), and so have its reads of X and
        // its conversion writes of step kt - 1 (only reads of Y may be in flight); after the barrier
        // everyone's have, and every wave is done with step kt - 1's stages
        FOCUS_WAIT_VMCNT(kMxLoads + 4);
        tr_wait15(X);
        asm volatile("s_barrier" ::: "memory");
        // the conversion's two reads go first, then the 16 fragment reads of step kt + 1's first
        // half: lgkmcnt(15) then means that the first two have landed
        u32x4_t w = ds_read_b128<0>(cds + cv_code);
        uint32_t sb = ds_read_u8<0>(cds + cv_scale);
        frags(std::integral_constant<int, 0>{}, Z, a_nx, o_nx);
        float sc = 0.0f;
        static_for<16>([&](auto idx) {
            constexpr int i = idx / 4, jj = idx % 4;
            acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(X.a[i], X.b[jj], acc[i][jj], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            // slot kt + 4: one load after every second MFMA; the conversion of slot kt + 2 after
            // MFMAs 4, 6, 8, 10 (one 16-byte chunk each), starting with the wait for its reads
            if constexpr (idx % 2 == 1 && idx / 2 < kMxLoads) issue(st, sl, idx / 2);
            if constexpr (idx == 4) {
                lds_wait<15>(w, sb);
                sc = scale_of(sb);
            }
            if constexpr (idx >= 4 && idx <= 10 && idx % 2 == 0) {
                constexpr int ch = (idx - 4) / 2;
                cvt_chunk(w[ch], sc, cas + cv_dst[ch]);
            }
            __builtin_amdgcn_sched_barrier(0);
        });
        tr_wait15(Y);  // read during step kt - 1
        frags(std::integral_constant<int, 1>{}, X, a_nx, o_nx);
        mma_frags(Y, acc);
        o_cur = next_d(o_cur), o_cv = next_d(o_cv), o_is = next_d(o_is);
        a_cur = next_a(a_cur), a_cv = next_a(a_cv);
    };
    int64_t kt = 0;
    for (; kt + 3 <= nk; kt += 3) {
        step(kt, f, g, h);
        step(kt + 1, h, f, g);
        step(kt + 2, g, h, f);
    }
    if (kt < nk) step(kt, f, g, h);
    if (kt + 1 < nk) step(kt + 1, h, f, g);
    tr_wait(f);  // no read may still be in flight when the workgroup ends
    FOCUS_WAIT_VMCNT(0);
    ste_epilogue<kFmtMX, WDT>(acc, k0, n0, split, N, K, W, s_fp, c, sb_log2, nullptr, ste_clip, e8m0_floor, part_s,
                              part_c, flag, wm, wn, lane);
}

// ================================================================================================

// Buffer offsets are 32-bit: a tile's rows must span less than 2^31 bytes.
bool mfma_fwd_supported(int64_t M, int64_t N, int64_t K) {
    return M > 0 && N > 0 && N % 8 == 0 && K % 16 == 0 && int64_t(kTile) * K * 2 < (int64_t(1) << 31) &&
           int64_t(kTile) * N * 2 < (int64_t(1) << 31) &&
           (M + kTile - 1) / kTile * ((N + kTile - 1) / kTile) < (int64_t(1) << 31);
}

bool mfma_bwd_supported(int64_t M, int64_t N, int64_t K) {
    return N % 8 == 0 && K % 16 == 0 && N > 0 && K > 0 && M >= 0 && int64_t(kBwdStep) * N * 2 < (int64_t(1) << 31) &&
           int64_t(kBwdStep) * K * 2 < (int64_t(1) << 31) && int64_t(kTile) * K * 4 < (int64_t(1) << 31);
}

hipError_t launch_fwd_mfma(const void *X, const void *W, int64_t M, int64_t N, int64_t K, const void *Yref, void *dY,
                           float dscale, double *colpart, hipStream_t st) {
    const int tiles_m = (int)((M + kTile - 1) / kTile), tiles_n = (int)((N + kTile - 1) / kTile);
    const dim3 grid((unsigned)tiles_m * tiles_n);
    const uint16_t *y = static_cast<const uint16_t *>(Yref);
    uint16_t *d = static_cast<uint16_t *>(dY);
    if (Yref) fwd_mfma_kernel<true, false><<<grid, kThreads, 0, st>>>(X, W, nullptr, nullptr, M, N, K, y, d, dscale, colpart, tiles_n);
    else fwd_mfma_kernel<false, false><<<grid, kThreads, 0, st>>>(X, W, nullptr, nullptr, M, N, K, y, d, dscale, colpart, tiles_n);
    return hipGetLastError();
}

bool mfma_fwd_mx_supported(int64_t M, int64_t N, int64_t K) {
    return M > 0 && N > 0 && N % 8 == 0 && M % 4 == 0 && K % 128 == 0 && int64_t(kTile) * K / 2 < (int64_t(1) << 31) &&
           (K / 32) * std::max(M, N) < (int64_t(1) << 31) &&
           int64_t(kTile) * N * 2 < (int64_t(1) << 31) &&
           (M + kTile - 1) / kTile * ((N + kTile - 1) / kTile) < (int64_t(1) << 31);
}

hipError_t launch_fwd_mfma_mx(const void *Xc, const void *Xs, const void *Wc, const void *Ws, int64_t M, int64_t N,
                              int64_t K, const void *Yref, void *dY, float dscale, double *colpart, hipStream_t st) {
    const int tiles_m = (int)((M + kTile - 1) / kTile), tiles_n = (int)((N + kTile - 1) / kTile);
    const dim3 grid((unsigned)tiles_m * tiles_n);
    const uint8_t *xs = static_cast<const uint8_t *>(Xs), *ws = static_cast<const uint8_t *>(Ws);
    const uint16_t *y = static_cast<const uint16_t *>(Yref);
    uint16_t *d = static_cast<uint16_t *>(dY);
    if (Yref) fwd_mfma_kernel<true, true><<<grid, kThreads, 0, st>>>(Xc, Wc, xs, ws, M, N, K, y, d, dscale, colpart, tiles_n);
    else fwd_mfma_kernel<false, true><<<grid, kThreads, 0, st>>>(Xc, Wc, xs, ws, M, N, K, y, d, dscale, colpart, tiles_n);
    return hipGetLastError();
}

bool mfma_bwd_mx_supported(int64_t M, int64_t N, int64_t K) {
    return N > 0 && K > 0 && M >= 0 && N % 8 == 0 && K % 32 == 0 && M % 4 == 0 &&
           int64_t(kBwdStep) * N * 2 < (int64_t(1) << 31) && (K / 32) * M < (int64_t(1) << 31) - 64 &&
           int64_t(kTile) * K * 4 < (int64_t(1) << 31);
}

hipError_t launch_bwd_mfma_mx(int w_dt, const void *dY, const void *Xc, const void *Xs, int64_t M, int64_t N,
                              int64_t K, int64_t chunk, int64_t splits, const void *W, const float *s_fp,
                              const float *c, int sb, int ste_clip, int e8m0_floor, float *part_s, float *part_c,
                              uint32_t *flag, hipStream_t st) {
    const int tiles_k = (int)((K + kTile - 1) / kTile), tiles_n = (int)((N + kTile - 1) / kTile);
    int sbl = 0;
    while ((1 << sbl) < sb) sbl++;
    const dim3 grid((unsigned)tiles_k * tiles_n, (unsigned)splits);
    const uint16_t *dy = static_cast<const uint16_t *>(dY);
    const uint8_t *xc = static_cast<const uint8_t *>(Xc), *xs = static_cast<const uint8_t *>(Xs);
    if (w_dt == kBF16)
        bwd_mfma_mx_kernel<kBF16><<<grid, kThreads, 0, st>>>(dy, xc, xs, M, N, K, chunk, W, s_fp, c, sbl, ste_clip,
                                                             e8m0_floor, part_s, part_c, flag, tiles_n);
    else
        bwd_mfma_mx_kernel<kF32><<<grid, kThreads, 0, st>>>(dy, xc, xs, M, N, K, chunk, W, s_fp, c, sbl, ste_clip,
                                                            e8m0_floor, part_s, part_c, flag, tiles_n);
    return hipGetLastError();
}

hipError_t launch_bwd_mfma(int fmt, int w_dt, const void *dY, const void *X, int64_t M, int64_t N, int64_t K,
                           int64_t chunk, int64_t splits, const void *W, const float *s_fp, const float *c, int sb,
                           const float *alpha, int ste_clip, int e8m0_floor, float *part_s, float *part_c,
                           uint32_t *flag, hipStream_t st) {
    const int tiles_k = (int)((K + kTile - 1) / kTile), tiles_n = (int)((N + kTile - 1) / kTile);
    int sbl = 0;
    while ((1 << sbl) < sb) sbl++;
    const dim3 grid((unsigned)tiles_k * tiles_n, (unsigned)splits);
    const uint16_t *dy = static_cast<const uint16_t *>(dY), *x = static_cast<const uint16_t *>(X);
#define BM(F, WD) bwd_mfma_kernel<F, WD><<<grid, kThreads, 0, st>>>(dy, x, M, N, K, chunk, W, s_fp, c, sbl, alpha, ste_clip, e8m0_floor, part_s, part_c, flag, tiles_n)
    if (fmt == kFmtMX) { if (w_dt == kBF16) BM(kFmtMX, kBF16); else BM(kFmtMX, kF32); }
    else { if (w_dt == kBF16) BM(kFmtNV, kBF16); else BM(kFmtNV, kF32); }
#undef BM
    return hipGetLastError();
}

}  // namespace focus
