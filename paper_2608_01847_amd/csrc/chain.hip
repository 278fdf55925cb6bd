// End-to-end chaining of the scale-learning step: the transposed weight operand of dX_hat = dY W_hat
// and the KL-Top objective on logits (Sec. 4.1: the paper trains end to end with the KL-Top loss,
// k = 1000, following the method it cites for that loss).
#include <cmath>

#include "focus_device.h"
#include "internal.h"

namespace focus {

namespace {

// ------------------------------------------------------------------------------------------------
// out[c][r] = in[r][c] for an R x C matrix, 64 x 64 tiles staged through LDS (rows of 64 elements
// read and written contiguously; the padded column breaks bank conflicts of the transposed reads).
template <typename T>
__global__ void __launch_bounds__(256) transpose_kernel(const T *__restrict__ in, int64_t R, int64_t C,
                                                         T *__restrict__ out) {
    __shared__ T tile[64][65];
    const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int64_t r = r0 + i, c = c0 + tx;
        if (r < R && c < C) tile[i][tx] = in[r * C + c];
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int64_t c = c0 + i, r = r0 + tx;
        if (c < C && r < R) out[c * R + r] = tile[tx][i];
    }
}

// ------------------------------------------------------------------------------------------------
// KL-Top. Keys order fp32 values as unsigned integers (negative values flipped, positive ones with
// the sign bit set); -0 is taken as +0 so that equal values have equal keys.
__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t b = __float_as_uint(f);
    b = b == 0x80000000u ? 0u : b;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

template <int IN>
__device__ __forceinline__ float load_logit(const void *p, int64_t i) {
    if (IN == kBF16) return bf16_bits_to_f32(reinterpret_cast<const uint16_t *>(p)[i]);
    return reinterpret_cast<const float *>(p)[i];
}

// the key of logit i; for bf16 logits only the high 16 bits carry information (the low half of a
// flipped negative value would be all ones), so they alone are kept
template <int IN>
__device__ __forceinline__ uint32_t logit_key(float v) {
    const uint32_t k = order_key(v);
    return IN == kBF16 ? (k & 0xFFFF0000u) : k;
}

template <int IN>
__device__ __forceinline__ void store_logit(void *p, int64_t i, float v) {
    if (IN == kBF16) reinterpret_cast<uint16_t *>(p)[i] = (uint16_t)f32_to_bf16_bits(v);
    else reinterpret_cast<float *>(p)[i] = v;
}

// the same with the non-temporal cache policy (dZ is written once and not read back here)
template <int IN>
__device__ __forceinline__ void store_logit_nt(void *p, int64_t i, float v) {
    if (IN == kBF16) __builtin_nontemporal_store((uint16_t)f32_to_bf16_bits(v), reinterpret_cast<uint16_t *>(p) + i);
    else __builtin_nontemporal_store(v, reinterpret_cast<float *>(p) + i);
}

// Logits of elements base + t + 256 u (u = 0 .. kTrips - 1) of a row: a thread's next kTrips elements
// in its usual order, loaded before any is used so that kTrips loads are in flight at once (the passes
// are bound by the latency of rows that no longer fit the caches: 16 in flight took the 8192 x 151936
// call from 9.2 to 7.3 ms, 8 or 32 less far). An index past the row is clamped to its last element
// (V >= 1), so every load is unconditional and in bounds; the callers ignore those positions. The
// element order of each thread, and so every result bit, is that of one element per trip.
constexpr int kTrips = 16;
template <int IN>
__device__ __forceinline__ void load_trips(const void *p, int64_t base, int t, int64_t V, float (&v)[kTrips]) {
#pragma unroll
    for (int u = 0; u < kTrips; u++) {
        const int64_t i = base + t + 256 * u;
        v[u] = load_logit<IN>(p, i < V ? i : V - 1);
    }
}

// inclusive scan of one value per thread over the workgroup (256 threads), in thread order
__device__ __forceinline__ uint32_t block_scan(uint32_t v, uint32_t *buf) {
    const int t = threadIdx.x;
    buf[t] = v;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const uint32_t add = t >= off ? buf[t - off] : 0u;
        __syncthreads();
        buf[t] += add;
        __syncthreads();
    }
    const uint32_t r = buf[t];
    __syncthreads();
    return r;
}

// One workgroup per token row, in one of two ways. Both give the same selected set (the teacher's k
// largest logits, ties at the k-th value in index order) and the same per-element formulas; the sums
// run in a fixed order in each, so every result is deterministic.
//  * Sample-select, when the k largest are a small part of a long row: the r-th largest of 3,072
//    teacher keys, r with a binomial margin of 3 standard deviations over the expected count, lies
//    below the k-th largest key almost always (10 rows of 8,192 miss at k = 1,000 of 151,936 on
//    independent logits). The sample is 384 evenly spaced runs of 8 adjacent keys: keys spaced
//    singly touched nearly every memory line of the row, an extra read of it (2.9 -> 2.3 ms). A
//    sample that misleads (logits correlated along the row) costs time only, never a result. One pass over both rows writes a zero dZ for every element and gathers those at or
//    above that key (about 1.8 k) into per-wave LDS lists in index order; the k-th largest key, the
//    tie cut (up to kTieMax ties at it), the softmax statistics and the KL terms then come from LDS,
//    and the gathered elements get their final dZ. Two reads of each row instead of seven, dZ stored
//    with the non-temporal policy (10% faster than the default): 8,192 x 151,936 bf16 logits 7.3 ->
//    2.0 ms.
//  * The passes below whenever the gathered set misses the k-th largest key, overflows the lists or
//    holds too many ties, or the row is short or k large: a radix select of the k-th largest teacher key (8-bit digits from
//    the top, LDS histograms); if fewer ties at that key are admitted than exist, the index of the
//    last admitted tie (256 elements per trip, ballots for the in-trip ranks); online softmax
//    statistics of both rows over the selected set (per thread, then a fixed tree); KL terms and dZ_s
//    (zero outside the set). Each dZ element is written by the same thread in both ways.
constexpr int kSample = 3072;          // sampled teacher keys (12 per thread)
constexpr int kCand = 3072;            // gathered elements (LDS lists of 768 per wave)
constexpr int kPerWave = kCand / 4;
constexpr int64_t kSampleMinV = 32768;  // shorter rows take the passes
constexpr int kTieMax = 1024;           // ties at the threshold key the gathered path resolves
template <int IN>
__global__ void __launch_bounds__(256)
kl_top_kernel(const void *__restrict__ Zs, const void *__restrict__ Zt, int64_t V, int k, double inv_T,
              void *__restrict__ dZs, double *__restrict__ row_loss, uint32_t *flag) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t scan_buf[256];
    __shared__ uint32_t sel_digit, sel_above;
    __shared__ uint32_t wave_cnt[4];
    __shared__ float red_m[2][256];
    __shared__ double red_s[2][256];
    __shared__ double red_d[256];
    __shared__ uint32_t cand_a[kCand];  // teacher logit bits (first the sampled keys)
    __shared__ uint32_t cand_idx[kCand];
    __shared__ float cand_b[kCand];
    __shared__ uint32_t wave_n[4], tie_cnt;
    __shared__ uint32_t tie_idx[kTieMax];
    __shared__ int64_t cut_sh;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t row = blockIdx.x;
    const char *zs = reinterpret_cast<const char *>(Zs) + row * V * (IN == kBF16 ? 2 : 4);
    const char *zt = reinterpret_cast<const char *>(Zt) + row * V * (IN == kBF16 ? 2 : 4);
    char *dz = reinterpret_cast<char *>(dZs) + row * V * (IN == kBF16 ? 2 : 4);
    const bool all = (int64_t)k >= V;
    bool bad = false;
    constexpr int kPasses = IN == kBF16 ? 2 : 4;  // 8-bit digits of a key (bf16 keys have zero low 16 bits)

    // online softmax statistics of one selected pair of logits (sums of exp(z - max) in double: the
    // loss needs their logs to ~1e-12)
    auto online_stats = [](float a, float b, float &mt, double &st, float &ms, double &ss) {
        if (a > mt) {
            st = st * exp((double)mt - (double)a) + 1.0;
            mt = a;
        } else {
            st += exp((double)a - (double)mt);
        }
        if (b > ms) {
            ss = ss * exp((double)ms - (double)b) + 1.0;
            ms = b;
        } else {
            ss += exp((double)b - (double)ms);
        }
    };
    // log-sum-exp of each row over the selected set from every thread's statistics (a fixed tree):
    // lt_d for the teacher and dl = lt_d - ls_d, in double
    auto row_lse = [&](float mt, double st, float ms, double ss, double &lt_d, double &dl) {
        red_m[0][t] = mt, red_s[0][t] = st, red_m[1][t] = ms, red_s[1][t] = ss;
        __syncthreads();
        for (int off = 128; off > 0; off >>= 1) {
            if (t < off) {
                for (int q = 0; q < 2; q++) {
                    const float m1 = red_m[q][t], m2 = red_m[q][t + off];
                    const double s1 = red_s[q][t], s2 = red_s[q][t + off];
                    const float m = fmaxf(m1, m2);
                    const double s = (m1 == -INFINITY ? 0.0 : s1 * exp((double)m1 - (double)m)) +
                                     (m2 == -INFINITY ? 0.0 : s2 * exp((double)m2 - (double)m));
                    red_m[q][t] = m;
                    red_s[q][t] = s;
                }
            }
            __syncthreads();
        }
        lt_d = (double)red_m[0][0] + log(red_s[0][0]);
        dl = lt_d - ((double)red_m[1][0] + log(red_s[1][0]));
        __syncthreads();
    };
    // KL term of one selected element, -p_t d, added to kl; returns dZ_s = (p_s - p_t) / T. With
    // d = log p_s - log p_t, p_s - p_t = p_t expm1(d) keeps its relative accuracy where the two
    // probabilities nearly cancel.
    auto kl_term = [&](float a, float b, double lt_d, double dl, double &kl) {
        const double pt = exp((double)a - lt_d);
        const double d = ((double)b - (double)a) + dl;
        kl -= pt * d;
        return (float)(pt * expm1(d) * inv_T);
    };
    // the row's KL from every thread's part (a fixed tree)
    auto row_total = [&](double kl) {
        red_d[t] = kl;
        __syncthreads();
        for (int off = 128; off > 0; off >>= 1) {
            if (t < off) red_d[t] += red_d[t + off];
            __syncthreads();
        }
        if (t == 0) row_loss[row] = red_d[0];
    };
    // the kth largest (1-based) of the keys for_keys hands to its argument, and how many elements with
    // that key are among the kth largest (radix select, 8-bit digits from the top)
    auto kth_key = [&](auto for_keys, uint32_t kth, uint32_t &rem) {
        uint32_t pre = 0u, msk = 0u;
        rem = kth;
        for (int p = 0; p < kPasses; p++) {
            const int shift = 24 - 8 * p;
            hist[t] = 0u;
            __syncthreads();
            for_keys([&](uint32_t key) {
                if ((key & msk) == pre) atomicAdd(&hist[(key >> shift) & 255u], 1u);
            });
            __syncthreads();
            const uint32_t h = hist[255 - t];
            const uint32_t incl = block_scan(h, scan_buf);
            if (incl - h < rem && rem <= incl) {
                sel_digit = 255u - (uint32_t)t;
                sel_above = incl - h;
            }
            __syncthreads();
            rem -= sel_above;
            pre |= sel_digit << shift;
            msk |= 0xFFu << shift;
            __syncthreads();
        }
        return pre;
    };

    bool done = false;
    const double kexp = (double)k * kSample / (double)V;  // expected sampled keys at or above the k-th
    const int r = (int)ceil(kexp) + (int)ceil(3.0 * sqrt(kexp)) + 2;
    if (!all && V >= kSampleMinV && r <= kSample / 4 && (double)r * (double)V / kSample <= 0.65 * kCand) {
        // ---- the sample: 8 adjacent keys from each of kSample / 8 evenly spaced elements (rows of at
        // least kSampleMinV keep the runs apart), its r-th largest the gather bound ----
        uint32_t sk[kSample / 256];
#pragma unroll
        for (int u = 0; u < kSample / 256; u++)
            sk[u] = logit_key<IN>(load_logit<IN>(zt, (int64_t)((t + 256 * u) >> 3) * V / (kSample / 8) + ((t + 256 * u) & 7)));
#pragma unroll
        for (int u = 0; u < kSample / 256; u++) cand_a[t + 256 * u] = sk[u];
        __syncthreads();
        uint32_t rem_s;
        const uint32_t lower = kth_key([&](auto fn) {
            for (int j = t; j < kSample; j += 256) fn(cand_a[j]);
        }, (uint32_t)r, rem_s);  // ends on a barrier: the sample is read before the gather overwrites it
        // ---- one pass over both rows: zero dZ under the bound, the rest into this wave's list ----
        uint32_t wn = 0u;  // elements this wave has met at or above the bound (wave-uniform)
        const uint32_t seg = (uint32_t)wave * kPerWave;
        auto gather = [&](int64_t i, bool valid, float a, float b) {
            bad = bad || (valid && (!(__builtin_fabsf(a) < INFINITY) || !(__builtin_fabsf(b) < INFINITY)));
            const bool cand = valid && logit_key<IN>(a) >= lower;
            const uint64_t m = __ballot(cand);
            const uint32_t slot = wn + (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
            if (cand && slot < (uint32_t)kPerWave) {
                cand_a[seg + slot] = __float_as_uint(a);
                cand_idx[seg + slot] = (uint32_t)i;
                cand_b[seg + slot] = b;
            }
            wn += (uint32_t)__popcll(m);
        };
        for (int64_t base = 0; base < V; base += 256 * kTrips) {
            float va[kTrips], vb[kTrips];
            load_trips<IN>(zt, base, t, V, va);
            load_trips<IN>(zs, base, t, V, vb);
            if (base + 256 * kTrips <= V) {
                // a whole chunk: every store unconditional, so the compiler counts the memory operations
                // in flight exactly (a conditional store makes it wait for the stores before each
                // element); the gathered elements get their final dZ later, after several barriers
#pragma unroll
                for (int u = 0; u < kTrips; u++) {
                    const int64_t i = base + t + 256 * u;
                    gather(i, true, va[u], vb[u]);
                    store_logit_nt<IN>(dz, i, 0.0f);
                }
            } else {
#pragma unroll
                for (int u = 0; u < kTrips; u++) {
                    const int64_t i = base + t + 256 * u;
                    gather(i, i < V, va[u], vb[u]);
                    if (i < V) store_logit_nt<IN>(dz, i, 0.0f);
                }
            }
        }
        if (lane == 0) wave_n[wave] = wn;
        __syncthreads();
        const uint32_t nw[4] = {wave_n[0], wave_n[1], wave_n[2], wave_n[3]};
        const bool fits = nw[0] <= (uint32_t)kPerWave && nw[1] <= (uint32_t)kPerWave &&
                          nw[2] <= (uint32_t)kPerWave && nw[3] <= (uint32_t)kPerWave;
        if (fits && (uint64_t)nw[0] + nw[1] + nw[2] + nw[3] >= (uint64_t)k) {
            // every element at or above the k-th largest key is in the lists
            auto for_cands = [&](auto fn) {
                for (int w = 0; w < 4; w++)
                    for (uint32_t j = (uint32_t)t; j < nw[w]; j += 256u) fn((uint32_t)w * kPerWave + j);
            };
            auto key_at = [&](uint32_t s) { return logit_key<IN>(__uint_as_float(cand_a[s])); };
            uint32_t rem;
            const uint32_t thr = kth_key([&](auto fn) { for_cands([&](uint32_t s) { fn(key_at(s)); }); },
                                         (uint32_t)k, rem);
            // ties at the threshold key: the first rem of them in index order are selected
            if (t == 0) tie_cnt = 0u;
            __syncthreads();
            uint32_t my_ties = 0u;
            for_cands([&](uint32_t s) { my_ties += key_at(s) == thr ? 1u : 0u; });
            atomicAdd(&tie_cnt, my_ties);  // an integer count: the order of the additions is immaterial
            __syncthreads();
            if (tie_cnt <= (uint32_t)kTieMax) {
                int64_t cut = V;
                if (rem < tie_cnt) {
                    // The rem-th smallest index among the ties. A wave's list is in index order, so
                    // each wave compacts the ties of its own list, in order, into its region of
                    // tie_idx; a tie's rank among all ties is its place in its region plus the ties
                    // of smaller index in the other three regions (binary searches).
                    const uint32_t nown = nw[wave];
                    uint32_t mine_n = 0u;
                    for (uint32_t j0 = 0; j0 < nown; j0 += 64u) {
                        const uint32_t j = j0 + (uint32_t)lane;
                        mine_n += (uint32_t)__popcll(__ballot(j < nown && key_at(seg + j) == thr));
                    }
                    if (lane == 0) wave_cnt[wave] = mine_n;
                    __syncthreads();
                    const uint32_t off[5] = {0u, wave_cnt[0], wave_cnt[0] + wave_cnt[1],
                                             wave_cnt[0] + wave_cnt[1] + wave_cnt[2],
                                             wave_cnt[0] + wave_cnt[1] + wave_cnt[2] + wave_cnt[3]};
                    uint32_t pos = off[wave];
                    for (uint32_t j0 = 0; j0 < nown; j0 += 64u) {
                        const uint32_t j = j0 + (uint32_t)lane;
                        const bool tie = j < nown && key_at(seg + j) == thr;
                        const uint64_t m = __ballot(tie);
                        if (tie) tie_idx[pos + (uint32_t)__popcll(m & ((1ull << lane) - 1ull))] = cand_idx[seg + j];
                        pos += (uint32_t)__popcll(m);
                    }
                    __syncthreads();
                    for (uint32_t e = (uint32_t)t; e < off[4]; e += 256u) {
                        const int we = (e >= off[1]) + (e >= off[2]) + (e >= off[3]);
                        const uint32_t mine = tie_idx[e];
                        uint32_t rank = e - off[we];
                        for (int w = 0; w < 4; w++) {
                            if (w == we) continue;
                            uint32_t lo = off[w], hi = off[w + 1];
                            while (lo < hi) {
                                const uint32_t mid = (lo + hi) >> 1;
                                if (tie_idx[mid] < mine) lo = mid + 1u;
                                else hi = mid;
                            }
                            rank += lo - off[w];
                        }
                        if (rank + 1u == rem) cut_sh = (int64_t)mine + 1;
                    }
                    __syncthreads();
                    cut = cut_sh;
                }
                auto chosen = [&](uint32_t s) {
                    const uint32_t key = key_at(s);
                    return key > thr || (key == thr && (int64_t)cand_idx[s] < cut);
                };
                float mt = -INFINITY, ms = -INFINITY;
                double st = 0.0, ss = 0.0;
                for_cands([&](uint32_t s) {
                    if (chosen(s)) online_stats(__uint_as_float(cand_a[s]), cand_b[s], mt, st, ms, ss);
                });
                double lt_d, dl;
                row_lse(mt, st, ms, ss, lt_d, dl);
                double kl = 0.0;
                for_cands([&](uint32_t s) {
                    const float g = chosen(s) ? kl_term(__uint_as_float(cand_a[s]), cand_b[s], lt_d, dl, kl) : 0.0f;
                    store_logit_nt<IN>(dz, cand_idx[s], g);
                });
                row_total(kl);
                done = true;
            }
        }
        // otherwise the passes below decide (and write every dZ element again, each by the thread
        // that wrote its zero here)
    }

    if (!done) {
        // ---- threshold key: the k-th largest teacher key ----
        uint32_t prefix = 0u, pmask = 0u, remaining = (uint32_t)k;
        if (!all) {
            for (int p = 0; p < kPasses; p++) {
                const int shift = 24 - 8 * p;
                hist[t] = 0u;
                __syncthreads();
                for (int64_t base = 0; base < V; base += 256 * kTrips) {
                    float v[kTrips];
                    load_trips<IN>(zt, base, t, V, v);
    #pragma unroll
                    for (int u = 0; u < kTrips; u++) {
                        const uint32_t key = logit_key<IN>(v[u]);
                        if (base + t + 256 * u < V && (key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
                    }
                }
                __syncthreads();
                // bins in descending digit order: thread j holds digit 255 - j
                const uint32_t h = hist[255 - t];
                const uint32_t incl = block_scan(h, scan_buf);
                if (incl - h < remaining && remaining <= incl) {
                    sel_digit = 255u - (uint32_t)t;
                    sel_above = incl - h;
                }
                __syncthreads();
                remaining -= sel_above;
                prefix |= sel_digit << shift;
                pmask |= 0xFFu << shift;
                __syncthreads();
            }
        }
        const uint32_t thr = prefix;  // with `all`, every element is selected
        // ---- ties at the threshold: admit the first `remaining` in index order ----
        int64_t cut = V;  // selected ties are those with index < cut
        if (!all) {
            uint32_t seen = 0u;
            bool found = false;
            for (int64_t base0 = 0; base0 < V && !found; base0 += 256 * kTrips) {
                float v[kTrips];
                load_trips<IN>(zt, base0, t, V, v);
                for (int u = 0; u < kTrips; u++) {
                    const int64_t base = base0 + 256 * u;
                    if (base >= V) break;
                    const int64_t i = base + t;
                    const bool tie = i < V && logit_key<IN>(v[u]) == thr;
                    const uint64_t m = __ballot(tie);
                    if (lane == 0) wave_cnt[wave] = (uint32_t)__popcll(m);
                    __syncthreads();
                    uint32_t before = seen;
                    for (int w = 0; w < wave; w++) before += wave_cnt[w];
                    const uint32_t total = wave_cnt[0] + wave_cnt[1] + wave_cnt[2] + wave_cnt[3];
                    const uint32_t rank = before + (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
                    __syncthreads();
                    if (seen + total >= remaining) {
                        // the remaining-th tie is in this trip: its index + 1 is the cut
                        if (tie && rank + 1u == remaining) red_d[0] = (double)(i + 1);
                        __syncthreads();
                        cut = (int64_t)red_d[0];
                        found = true;
                        break;
                    }
                    seen += total;
                }
            }
        }
        auto selected = [&](int64_t i, uint32_t key) { return all || key > thr || (key == thr && i < cut); };

        // ---- softmax statistics over the selected set (online per thread) ----
        float mt = -INFINITY, ms = -INFINITY;
        double st = 0.0, ss = 0.0;  // sums of exp(z - max) in double: the loss needs their logs to ~1e-12
        for (int64_t base = 0; base < V; base += 256 * kTrips) {
            float va[kTrips], vb[kTrips];
            load_trips<IN>(zt, base, t, V, va);
            load_trips<IN>(zs, base, t, V, vb);
            for (int u = 0; u < kTrips; u++) {
                const int64_t i = base + t + 256 * u;
                if (i >= V) break;
                const float a = va[u], b = vb[u];
                bad = bad || !(__builtin_fabsf(a) < INFINITY) || !(__builtin_fabsf(b) < INFINITY);
                if (!selected(i, logit_key<IN>(a))) continue;
                online_stats(a, b, mt, st, ms, ss);
            }
        }
        double lt_d, dl;
        row_lse(mt, st, ms, ss, lt_d, dl);

        // ---- KL(p_t || p_s) over the set and dZ_s = (p_s - p_t) / T ----
        double kl = 0.0;
        for (int64_t base = 0; base < V; base += 256 * kTrips) {
            float va[kTrips], vb[kTrips];
            load_trips<IN>(zt, base, t, V, va);
            load_trips<IN>(zs, base, t, V, vb);
            const bool whole = base + 256 * kTrips <= V;  // stores unconditional (see the gather pass)
            for (int u = 0; u < kTrips; u++) {
                const int64_t i = base + t + 256 * u;
                if (!whole && i >= V) break;
                const float a = va[u], b = vb[u];
                float g = 0.0f;
                if (selected(i, logit_key<IN>(a))) g = kl_term(a, b, lt_d, dl, kl);
                store_logit<IN>(dz, i, g);
            }
        }
        row_total(kl);
    }
    if (bad && t == 0) raise_domain_flag(flag);
}

// loss = (sum of row losses) / T, in a fixed order
__global__ void __launch_bounds__(256) row_mean_kernel(const double *__restrict__ row_loss, int64_t T,
                                                        double *__restrict__ loss) {
    __shared__ double red[256];
    double acc = 0.0;
    for (int64_t i = threadIdx.x; i < T; i += 256) acc += row_loss[i];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = red[0] / (double)T;
}

// zero fill of a 16-byte-aligned buffer (whole 16-byte words, then the tail bytes)
__global__ void __launch_bounds__(256) zero_fill_kernel(char *__restrict__ p, size_t bytes) {
    const size_t words = bytes / 16;
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < words; i += (size_t)gridDim.x * 256)
        reinterpret_cast<uint4 *>(p)[i] = make_uint4(0u, 0u, 0u, 0u);
    if (blockIdx.x == 0 && threadIdx.x < bytes % 16) p[words * 16 + threadIdx.x] = 0;
}

}  // namespace

hipError_t launch_zero_fill(void *p, size_t bytes, hipStream_t st) {
    const size_t words = bytes / 16;
    const unsigned grid = (unsigned)std::max<size_t>(1, std::min<size_t>((words + 255) / 256, kStreamGridCap));
    zero_fill_kernel<<<grid, 256, 0, st>>>(static_cast<char *>(p), bytes);
    return hipGetLastError();
}

hipError_t launch_transpose(int dt, const void *in, int64_t R, int64_t C, void *out, hipStream_t st) {
    const dim3 grid((unsigned)((C + 63) / 64), (unsigned)((R + 63) / 64));
    if (dt == kBF16)
        transpose_kernel<uint16_t><<<grid, 256, 0, st>>>(static_cast<const uint16_t *>(in), R, C,
                                                         static_cast<uint16_t *>(out));
    else
        transpose_kernel<float><<<grid, 256, 0, st>>>(static_cast<const float *>(in), R, C, static_cast<float *>(out));
    return hipGetLastError();
}

hipError_t launch_kl_top(int dt, const void *Zs, const void *Zt, int64_t T, int64_t V, int k, void *dZs,
                         double *row_loss, double *loss, uint32_t *flag, hipStream_t st) {
    const double inv_T = 1.0 / (double)T;
    if (dt == kBF16) kl_top_kernel<kBF16><<<(unsigned)T, 256, 0, st>>>(Zs, Zt, V, k, inv_T, dZs, row_loss, flag);
    else kl_top_kernel<kF32><<<(unsigned)T, 256, 0, st>>>(Zs, Zt, V, k, inv_T, dZs, row_loss, flag);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    row_mean_kernel<<<1, 256, 0, st>>>(row_loss, T, loss);
    return hipGetLastError();
}

}  // namespace focus
