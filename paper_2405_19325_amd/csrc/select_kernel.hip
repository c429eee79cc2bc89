// Top-r stage, optionally fused with the mixture stage, and the standalone
// mixture stage on caller-given neighbours.
//
// Top-r: for every query, the r keys of its own set with the smallest squared
// distance (largest similarity s = -d, paper Section 2.2; the paper retrieves
// r = 1024, Appendix A), returned ascending by (distance, key index).  The
// paper does not order equal distances; the lower key index wins here.
//
// One 1024-thread workgroup per query.  Key i is ordered by (bits(d_i), i):
// distances are >= +0, so their fp32 bit patterns order like the values, and
// the index makes every key distinct.  Selection is a radix refinement: a
// range known to hold the r-th smallest key is narrowed with 2048-bin LDS
// histograms -- first on the distance bits, then, if a single distance value
// remains, on the key index -- starting from the per-tile min/max the distance
// stage leaves.
//
// Fast path (rows of at most 64 Ki keys, r <= 1024): the whole distance row is
// read once into registers (sixteen 16-byte loads per thread, all in flight
// together).  A histogram of 1024 keys sampled across the row picks a
// threshold that keeps, with overwhelming probability, between r and 4096 keys;
// one pass compacts them into LDS, and a bucket sort on their distance bits
// orders them; the first r are pi.  If the sample misjudges the count, the
// general path below takes over for that query, so the answer never depends on
// the sample.
//
// General path: every pass streams the distance row in 16 Ki-key batches with
// the next batch prefetched; the keys before the end of the final range (at
// most CAP) are compacted and bitonic-sorted in LDS.
//
// Mixture (eq. non-parametric and eq. kNN-LM), when p_m is given: the softmax
// of mu * s over the r neighbours (the largest mu * s, i.e. the smallest
// distance, is subtracted first), scattered onto the neighbours' value tokens
// in LDS vocabulary tiles with LDS float atomics (tokens no neighbour carries
// get 0; duplicates accumulate), then p_M = fmaf(lambda, p_LM, acc * ((1 -
// lambda) / Z)), so lambda = 1 returns p_LM bit for bit.  The order of the LDS
// atomics is not fixed, so p_kNN may differ between runs in the last bits,
// except in the split select's sliced finish, which adds the weights as 64-bit
// fixed-point integers (weight * 2^31, exact) and rounds each sum to fp32 once.
// With relative retrieval confidence (Section 3.2, eq. rrc) lambda is each
// query's own lambda_t = sigmoid((d_(1) / d_(r) - alpha) / tau), from the
// nearest and the r-th nearest distance (|s| is the distance); the split path
// then writes the whole p_M row in the finish kernel, since the parts kernel
// cannot know lambda_t.
#include <math.h>

#include "knnlm_device.h"
#include "select_internal.h"

namespace knnlm {

namespace {

constexpr int kT = kSelectThreads;                          // 1024 threads
constexpr int kNumWaves = kT / kWave;
constexpr int kPer = (KNNLM_MAX_R + kT - 1) / kT;            // neighbours per thread, general path
constexpr int kU = 4;                                       // 16-byte loads per thread per streamed batch
constexpr int64_t kBatch = static_cast<int64_t>(kT) * 4 * kU;  // keys per streamed batch (16384)
constexpr int kFastU = 16;                                  // fast path: the whole row in registers
constexpr int64_t kFastMaxN = static_cast<int64_t>(kT) * 4 * kFastU;  // 65536
constexpr int kFastCap = 4096;                              // candidates the fast path keeps in LDS
constexpr int kVocabTile = 8192;                            // mixture tile, general path
constexpr int kVocabTileFast = 32768;                       // mixture tile, fast path (128 KiB)
constexpr int kVocabSlice = 4 * kT;                         // p_M entries per workgroup, sliced split finish
constexpr int64_t kSliceMaxBlocks = 256;                    // workgroups a sliced split finish may take

// Target of the mixture's 16-byte stores from lanes past the end of a row.
__device__ float4 g_mix_sink;

// What a select launch does after pi: nothing, the mixture with one lambda,
// the mixture with lambda_t from relative retrieval confidence, or that and
// the decoding outputs of a NEST step (greedy token, span start, draft
// probability).
enum MixMode { kNoMix = 0, kMixFixed = 1, kMixRrc = 2, kMixNest = 3 };
constexpr bool rrc_mode(int mode) { return mode == kMixRrc || mode == kMixNest; }

struct Shared {
    uint32_t red_u[2][kNumWaves];
    alignas(16) uint32_t wave_tot[kNumWaves];
    float red_f[kNumWaves];
    uint32_t lo, hi, below, cnt, found, total;
    uint32_t ccount, cmin;  // split path: a part's candidates so far, and their smallest distance bits
    float dmin, dlast;
};

// The weight of p_LM for one query from its nearest (d_first) and r-th nearest
// (d_last) distance: m.lambda, or with RRC (eq. rrc, |s| = the distance)
// sigmoid((d_first / d_last - alpha) / tau), a row of zero distances having
// ratio 1.  Thread 0 records it in m.lambda_out (when `record`).
template <int MODE>
__device__ __forceinline__ float query_lambda(const MixArgs &m, int64_t b, float d_first, float d_last,
                                              bool record = true) {
    if constexpr (!rrc_mode(MODE)) {
        return m.lambda;
    } else {
        const float ratio = d_last > 0.0f ? d_first / d_last : 1.0f;
        const float lam = 1.0f / (1.0f + expf(-(ratio - m.alpha) / m.tau));
        if (record && threadIdx.x == 0 && m.lambda_out != nullptr) m.lambda_out[b] = lam;
        return lam;
    }
}

__device__ __forceinline__ uint64_t sort_key(uint32_t dbits, uint32_t i) {
    return (static_cast<uint64_t>(dbits) << 32) | i;
}

// Exclusive prefix sum of one value per thread over the block: a scan within
// each wave, then every wave adds the totals of the waves before it (one
// barrier between).  Without TAIL_BARRIER the caller must pass a barrier
// before wave_tot is written again.
template <bool TAIL_BARRIER = true>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t *wave_tot) {
    static_assert(kNumWaves % 4 == 0, "whole 16-byte words of wave totals");
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const uint32_t incl = wave_incl_scan_u32(v, lane);
    if (lane == kWave - 1) wave_tot[wave] = incl;
    __syncthreads();
    uint32_t before = 0u;
#pragma unroll
    for (int i = 0; i < kNumWaves / 4; ++i) {
        const uint4 t = reinterpret_cast<const uint4 *>(wave_tot)[i];
        before += (4 * i < wave ? t.x : 0u) + (4 * i + 1 < wave ? t.y : 0u) + (4 * i + 2 < wave ? t.z : 0u) +
                  (4 * i + 3 < wave ? t.w : 0u);
    }
    if constexpr (TAIL_BARRIER) __syncthreads();
    return before + incl - v;
}

__device__ __forceinline__ float block_sum(float v, float *red) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    v = wave_allsum(v);
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float t = 0.0f;
#pragma unroll
    for (int w = 0; w < kNumWaves; ++w) t += red[w];
    __syncthreads();
    return t;
}

__device__ __forceinline__ float block_min(float v, float *red) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    v = wave_allmin(v);
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float t = red[0];
#pragma unroll
    for (int w = 1; w < kNumWaves; ++w) t = fminf(t, red[w]);
    __syncthreads();
    return t;
}

// min and max of the per-thread values over the block (every thread gets both).
// Without TAIL_BARRIER the caller must pass a barrier before sh.red_u is
// written again.
template <bool TAIL_BARRIER = true>
__device__ __forceinline__ void block_minmax_u32(uint32_t &mn, uint32_t &mx, Shared &sh) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    mn = wave_allmin_u32(mn);
    mx = wave_allmax_u32(mx);
    if (lane == 0) {
        sh.red_u[0][wave] = mn;
        sh.red_u[1][wave] = mx;
    }
    __syncthreads();
    mn = sh.red_u[0][0];
    mx = sh.red_u[1][0];
#pragma unroll
    for (int w = 1; w < kNumWaves; ++w) {
        mn = min(mn, sh.red_u[0][w]);
        mx = max(mx, sh.red_u[1][w]);
    }
    if constexpr (TAIL_BARRIER) __syncthreads();
}

// Range of a query's distance bits from the distance stage's per-tile extrema.
__device__ __forceinline__ void row_range(const SelectArgs &a, int64_t b, int64_t N, uint32_t &bmin, uint32_t &bmax,
                                          Shared &sh) {
    bmin = 0xffffffffu;
    bmax = 0u;
    const int64_t ntiles = (N + a.rows_per_tile - 1) / a.rows_per_tile;
    for (int64_t t = threadIdx.x; t < ntiles; t += kT) {
        bmin = min(bmin, __float_as_uint(a.tile_min[b * a.tiles_per_set + t]));
        bmax = max(bmax, __float_as_uint(a.tile_max[b * a.tiles_per_set + t]));
    }
    block_minmax_u32(bmin, bmax, sh);
    if (N == 0 || bmin > bmax) {  // no key, or every key masked
        bmin = 0u;
        bmax = 0u;
    }
}

__device__ __forceinline__ uint32_t lane_word(const uint4 &v, int e) {
    return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w;
}

// Element (u, e) of a thread's registers sits at key index base + u * 4096 + e.
__device__ __forceinline__ int32_t elem_off(int u, int e) { return u * kT * 4 + e; }

// Given the histogram of the keys inside the current range, move the range to
// the bin holding the need-th of them.  Thread t owns bins 2t and 2t+1.
__device__ __forceinline__ void pick_bin(const uint32_t *hist, uint32_t need, int shift, Shared &sh) {
    const int tid = threadIdx.x;
    const uint32_t c0 = hist[2 * tid], c1 = hist[2 * tid + 1];
    const uint32_t lo = sh.lo, hi = sh.hi;
    const uint32_t excl = block_excl_scan(c0 + c1, sh.wave_tot);
    int j = -1;
    uint32_t before = 0, cj = 0;
    if (excl < need && excl + c0 >= need) {
        j = 2 * tid; before = excl; cj = c0;
    } else if (excl + c0 < need && excl + c0 + c1 >= need) {
        j = 2 * tid + 1; before = excl + c0; cj = c1;
    }
    if (j >= 0) {
        const uint32_t nlo = lo + (static_cast<uint32_t>(j) << shift);
        const uint64_t nhi = static_cast<uint64_t>(nlo) + (1ull << shift);
        sh.hi = nhi < hi ? static_cast<uint32_t>(nhi) : hi;
        sh.lo = nlo;
        sh.below += before;
        sh.cnt = cj;
        sh.found = 1u;
    }
    __syncthreads();
}

template <int BLOG = kSelectBinsLog2>
__device__ __forceinline__ int range_shift(uint32_t w) {
    const int nbits = 32 - __clz(static_cast<int>(w - 1u));
    return nbits > BLOG ? nbits - BLOG : 0;
}

// One wave (lane = its lane index): the bin of hist[0, 2048) holding the
// need-th (1-based) of the counted keys, or ~0u if there are fewer.  Each lane
// sums 32 consecutive bins, a wave scan finds the lane where the running count
// reaches need, and that lane walks its 32 bins.
__device__ __forceinline__ uint32_t wave_pick_bin(const uint32_t *hist, uint32_t need, int lane) {
    static_assert(kSelectBins == 32 * kWave, "32 bins per lane");
    uint32_t c[32];
    uint32_t sum = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const uint4 q = reinterpret_cast<const uint4 *>(hist + 32 * lane)[i];
        c[4 * i] = q.x; c[4 * i + 1] = q.y; c[4 * i + 2] = q.z; c[4 * i + 3] = q.w;
        sum += q.x + q.y + q.z + q.w;
    }
    const uint32_t incl = wave_incl_scan_u32(sum, lane);
    const uint32_t excl = incl - sum;
    const bool mine = excl < need && incl >= need;
    const uint64_t who = __ballot(mine);
    if (who == 0) return ~0u;
    uint32_t j = 0, run = excl;
    bool done = false;
#pragma unroll
    for (int i = 0; i < 32; ++i) {
        run += c[i];
        if (!done && run >= need) { j = static_cast<uint32_t>(32 * lane + i); done = true; }
    }
    return readlane_u32(j, __ffsll(static_cast<unsigned long long>(who)) - 1);
}

// Is key (bits, i) before the end of the range?  In the distance regime the
// range ends at bits == hi; in the index regime (fix) it ends at (fv, hi).
__device__ __forceinline__ bool before_end(uint32_t bits, uint32_t i, bool fix, uint32_t fv, uint32_t hi) {
    return fix ? (bits < fv || (bits == fv && i < hi)) : bits < hi;
}

// Ascending bitonic sort of cand[0, P) in LDS (P a power of two).
__device__ __forceinline__ void lds_bitonic(uint64_t *cand, uint32_t P) {
    const uint32_t tid = threadIdx.x;
    for (uint32_t k = 2; k <= P; k <<= 1) {
        for (uint32_t jj = k >> 1; jj > 0; jj >>= 1) {
            for (uint32_t t = tid; t < P / 2; t += kT) {
                const uint32_t i = ((t & ~(jj - 1)) << 1) | (t & (jj - 1));
                const uint32_t p = i | jj;
                const uint64_t x = cand[i], y = cand[p];
                const bool up = (i & k) == 0;
                if ((x > y) == up) {
                    cand[i] = y;
                    cand[p] = x;
                }
            }
            __syncthreads();
        }
    }
}

struct NoHook {
    __device__ void operator()() const {}
};

// Ascending sort of the n <= PER * 1024 keys in cand[0, n), in place, by
// 2^BLOG buckets of their distance bits over [lo, lo + w): each key takes a
// slot in its bucket with an LDS atomic, a block scan turns bucket sizes into
// bucket starts, the keys are scattered to tmp, and each key's final place is
// its bucket start plus its rank among the (few) keys of its bucket (a key
// alone in its bucket compares nothing; otherwise the first eight are compared
// at once, reads past the bucket discarded).  A bucket
// holding many equal distances only costs time, never order.  With ZEROED the
// caller has cleared count[] and ordered that with a barrier.  `mid` runs
// between the scan and the scatter (callers issue loads there that the rest
// of the sort hides).  Only cand[0, keep) is guaranteed on return: keys whose
// bucket starts at or after `keep` are not placed.
template <int PER, int BLOG = kSelectBinsLog2, bool ZEROED = false, typename Hook = NoHook>
__device__ __forceinline__ void bucket_sort(uint64_t *cand, uint32_t n, uint32_t lo, uint32_t w, uint32_t *count,
                                            uint32_t *start, uint64_t *tmp, Shared &sh, Hook mid = Hook(),
                                            uint32_t keep = ~0u) {
    constexpr int BINS = 1 << BLOG;
    constexpr int BPT = BINS / kT;  // bins per thread in the scan
    static_assert(BPT >= 1 && BINS % kT == 0, "whole bins per thread");
    const int tid = threadIdx.x;
    const int shift = range_shift<BLOG>(w > 1u ? w : 2u);
    if (!ZEROED) {
        for (int i = tid; i < BINS; i += kT) count[i] = 0u;
        __syncthreads();
    }
    uint64_t key[PER];
    uint32_t bin[PER], slot[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        const uint32_t j = static_cast<uint32_t>(q * kT + tid);
        key[q] = j < n ? cand[j] : ~0ull;
        bin[q] = j < n ? ((static_cast<uint32_t>(key[q] >> 32) - lo) >> shift) : 0u;
        if (bin[q] >= static_cast<uint32_t>(BINS)) bin[q] = BINS - 1;  // never for consistent input
        slot[q] = j < n ? atomicAdd(&count[bin[q]], 1u) : 0u;
    }
    __syncthreads();
    uint32_t cb[BPT], tsum = 0;
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
        cb[i] = count[BPT * tid + i];
        tsum += cb[i];
    }
    uint32_t run = block_excl_scan<false>(tsum, sh.wave_tot);  // the barrier below ends its reads
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
        start[BPT * tid + i] = run;
        run += cb[i];
    }
    mid();
    __syncthreads();
#pragma unroll
    for (int q = 0; q < PER; ++q)
        if (q * kT + tid < static_cast<int>(n)) tmp[start[bin[q]] + slot[q]] = key[q];
    __syncthreads();
    uint32_t b0[PER], nb[PER], rank[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        b0[q] = start[bin[q]];
        nb[q] = b0[q] < keep ? count[bin[q]] : 0u;  // a bucket past `keep` holds no key of the first `keep`
        rank[q] = 0u;
    }
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        if (nb[q] > 1u) {
#pragma unroll
            for (uint32_t i = 0; i < 8; ++i) {
                const uint32_t at = b0[q] + i < static_cast<uint32_t>(PER * kT) ? b0[q] + i : PER * kT - 1;
                rank[q] += (i < nb[q] && tmp[at] < key[q]) ? 1u : 0u;
            }
        }
    }
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        for (uint32_t i = 8; i < nb[q]; ++i) rank[q] += tmp[b0[q] + i] < key[q] ? 1u : 0u;
        if (q * kT + tid < static_cast<int>(n) && b0[q] < keep) cand[b0[q] + rank[q]] = key[q];
    }
    __syncthreads();
}

// ------------------------------------------------------------ general path

__device__ __forceinline__ void load_batch(const float *drow, int64_t N, int64_t bb, uint4 (&v)[kU]) {
    const int64_t base = bb * kBatch;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const int64_t i = base + (static_cast<int64_t>(u) * kT + threadIdx.x) * 4;
        v[u] = (i < N) ? *reinterpret_cast<const uint4 *>(drow + i) : make_uint4(0u, 0u, 0u, 0u);
    }
}

__device__ __forceinline__ void next_batch(const float *drow, int64_t N, int64_t bb, int64_t nbatch, uint4 (&nx)[kU]) {
    if (bb + 1 < nbatch) {
        load_batch(drow, N, bb + 1, nx);
    } else {
#pragma unroll
        for (int u = 0; u < kU; ++u) nx[u] = make_uint4(0u, 0u, 0u, 0u);
    }
}

__device__ __forceinline__ void advance(uint4 (&v)[kU], const uint4 (&nx)[kU]) {
#pragma unroll
    for (int u = 0; u < kU; ++u) v[u] = nx[u];
}

// Select over a streamed row: on return cand[0, n) holds, sorted ascending,
// every key before the end of the final range (n >= r_eff, n <= CAP); returns n.
template <int CAP>
__device__ uint32_t select_stream(const float *drow, int64_t N, uint32_t r_eff, uint32_t bmin, uint32_t bmax,
                                  uint64_t *cand, uint32_t *hist, Shared &sh) {
    const int tid = threadIdx.x;
    const int64_t nbatch = (N + kBatch - 1) / kBatch;
    uint4 v[kU], nx[kU];
    if (tid == 0) {
        sh.lo = bmin;
        sh.hi = bmax + 1u;  // distances are >= +0, so bmax < 0x80000000
        sh.below = 0u;
        sh.cnt = static_cast<uint32_t>(N);
    }
    __syncthreads();
    uint32_t lo = sh.lo, hi = sh.hi, below = sh.below, cnt = sh.cnt, fv = 0u;
    bool fix = false;
    for (int pass = 0; pass < 12 && below + cnt > static_cast<uint32_t>(CAP); ++pass) {
        if (!fix && hi - lo == 1u) {  // one distance value left: order by index
            fix = true;
            fv = lo;
            lo = 0u;
            hi = static_cast<uint32_t>(N);
        }
        const uint32_t w = hi - lo;
        const int shift = range_shift(w);
        for (int i = tid; i < kSelectBins; i += kT) hist[i] = 0u;
        if (tid == 0) { sh.found = 0u; sh.lo = lo; sh.hi = hi; }
        __syncthreads();
        load_batch(drow, N, 0, v);
        for (int32_t bb = 0; bb < nbatch; ++bb) {
            next_batch(drow, N, bb, nbatch, nx);
            const int32_t base = bb * static_cast<int32_t>(kBatch) + 4 * tid;
            const int32_t limit = static_cast<int32_t>(N) - base;
#pragma unroll
            for (int u = 0; u < kU; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t bits = lane_word(v[u], e);
                    const uint32_t off = (fix ? static_cast<uint32_t>(base + elem_off(u, e)) : bits) - lo;
                    if (elem_off(u, e) < limit && off < w && (!fix || bits == fv)) atomicAdd(&hist[off >> shift], 1u);
                }
            advance(v, nx);
        }
        __syncthreads();
        pick_bin(hist, r_eff - below, shift, sh);
        const bool found = sh.found != 0u;
        lo = sh.lo; hi = sh.hi; below = sh.below; cnt = sh.cnt;
        __syncthreads();
        if (!found) break;
    }

    // Compaction of every key before the end of the range.
    uint32_t written = 0;
    load_batch(drow, N, 0, v);
    for (int32_t bb = 0; bb < nbatch; ++bb) {
        next_batch(drow, N, bb, nbatch, nx);
        const int32_t base = bb * static_cast<int32_t>(kBatch) + 4 * tid;
        const int32_t limit = static_cast<int32_t>(N) - base;
        uint32_t c = 0;
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t i = static_cast<uint32_t>(base + elem_off(u, e));
                c += (elem_off(u, e) < limit && before_end(lane_word(v[u], e), i, fix, fv, hi)) ? 1u : 0u;
            }
        uint32_t pos = written + block_excl_scan(c, sh.wave_tot);
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t bits = lane_word(v[u], e);
                const uint32_t i = static_cast<uint32_t>(base + elem_off(u, e));
                if (elem_off(u, e) < limit && before_end(bits, i, fix, fv, hi)) {
                    if (pos < static_cast<uint32_t>(CAP)) cand[pos] = sort_key(bits, i);
                    ++pos;
                }
            }
        if (tid == kT - 1) sh.total = pos;  // the last thread's end offset
        __syncthreads();
        written = sh.total;
        __syncthreads();
        advance(v, nx);
    }
    const uint32_t n = written < static_cast<uint32_t>(CAP) ? written : static_cast<uint32_t>(CAP);
    uint32_t P = 1;
    while (P < n) P <<= 1;
    for (uint32_t i = n + tid; i < P; i += kT) cand[i] = ~0ull;
    __syncthreads();
    lds_bitonic(cand, P);
    return n;
}

// ------------------------------------------------------------------ mixture

__device__ __forceinline__ bool mix_vec4(const MixArgs &m, int64_t b) {
    return (m.V % 4 == 0) &&
           ((reinterpret_cast<uintptr_t>(m.p_lm + b * m.V) | reinterpret_cast<uintptr_t>(m.p_m + b * m.V)) & 15u) == 0;
}

// The draft token row b checks (NEST; -1 for none), read at a kernel's start
// through the scalar cache so that only its use waits for it.
template <int MODE>
__device__ __forceinline__ int32_t draft_token(const MixArgs &m, int64_t b) {
    return (MODE == kMixNest && m.draft != nullptr) ? load_scalar_i32(m.draft + b) : -1;
}

// This thread's float4s of the p_LM tile starting at v0 (16-byte path only):
// unconditional loads, lanes past the row reading its last float4 (or, off the
// 16-byte path, the sink), so that no branch sits around them; those lanes'
// values are never used.
template <int NV4>
__device__ __forceinline__ void mix_prefetch(const MixArgs &m, int64_t b, int64_t v0, float4 (&pre)[NV4]) {
    const int64_t nv = (m.V - v0 < static_cast<int64_t>(NV4) * 4 * kT) ? m.V - v0 : static_cast<int64_t>(NV4) * 4 * kT;
    const bool row = mix_vec4(m, b) && nv >= 4;
    const float4 *src = row ? reinterpret_cast<const float4 *>(m.p_lm + b * m.V + v0) : &g_mix_sink;
    const int64_t last = row ? nv / 4 - 1 : 0;  // the sink has one element
#pragma unroll
    for (int q = 0; q < NV4; ++q) {
        const int64_t i = static_cast<int64_t>(q) * kT + threadIdx.x;
        pre[q] = src[i < last ? i : last];
    }
}

// Waits for the loads of a prefetch that a path does not use, so that no code
// after that path and another one meet waits for the other path's stores.
template <int NV4>
__device__ __forceinline__ void consume_loads(const float4 (&pre)[NV4]) {
    float t = 0.0f;
#pragma unroll
    for (int q = 0; q < NV4; ++q) t += (pre[q].x + pre[q].y) + (pre[q].z + pre[q].w);
    asm volatile("" ::"v"(t));
}

// p_M row b with weight lam of p_LM: weights wj (unnormalised softmax terms, sum z) are scatter-added
// onto their tokens tok (-1: none) one vocabulary tile of TILE entries at a
// time in LDS; each tile's p_LM slice sits in registers (prefetched by the
// caller for the first tile when `first` is given) and is mixed with 16-byte
// accesses.
// The largest value over the block and the lowest index holding it (every
// thread gets both): v >= 0 or -1 for "none"; red holds 2 * kNumWaves words
// and is free again on return.
__device__ __forceinline__ void block_argmax(float &v, uint32_t &i, uint32_t *red) {
    const float m = wave_allmax(v);
    const uint32_t j = wave_allmin_u32(v == m ? i : ~0u);
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    if (lane == 0) {
        red[wave] = __float_as_uint(m);
        red[kNumWaves + wave] = j;
    }
    __syncthreads();
    // the waves' results, one a lane, reduced the same way again
    const float x = lane < kNumWaves ? __uint_as_float(red[lane]) : -__builtin_huge_valf();
    const uint32_t y = lane < kNumWaves ? red[kNumWaves + lane] : ~0u;
    const float bm = wave_allmax(x);
    const uint32_t bj = wave_allmin_u32(x == bm ? y : ~0u);
    __syncthreads();
    v = bm;
    i = bj;
}

// Entry (v, w) of a p_M row seen by this thread: entries come in increasing w,
// so a strictly larger value keeps the lowest token among equal values.
template <bool NEST>
__device__ __forceinline__ void note_entry(float v, int32_t w, int32_t dtok, float &bv, int32_t &bw, float &pd) {
    if constexpr (NEST) {
        bw = v > bv ? w : bw;
        bv = v > bv ? v : bv;
        pd = w == dtok ? v : pd;
    }
}

// p_M row b with weight lam of p_LM: weights wj (unnormalised softmax terms, sum z) are scatter-added
// onto their tokens tok (-1: none) one vocabulary tile of TILE entries at a
// time in LDS; each tile's p_LM slice sits in registers (prefetched by the
// caller for the first tile when `first` is given) and is mixed with 16-byte
// accesses.
// 64-bit max / min over the block (every thread gets the result); red holds
// kNumWaves entries and is free again on return.
__device__ __forceinline__ uint64_t block_max_u64(uint64_t v, uint64_t *red) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const uint64_t o = __shfl_xor(v, off);
        v = o > v ? o : v;
    }
    if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = v;
    __syncthreads();
    uint64_t t = red[0];
#pragma unroll
    for (int w = 1; w < kNumWaves; ++w) t = red[w] > t ? red[w] : t;
    __syncthreads();
    return t;
}

__device__ __forceinline__ uint64_t block_min_u64(uint64_t v, uint64_t *red) {
    return ~block_max_u64(~v, red);
}

// p_M entry (value, token) as a key whose largest is the largest value, the
// lowest token among equal values (p_M >= 0, so the bits order like values).
__device__ __forceinline__ uint64_t best_key(float v, int64_t w) {
    return (static_cast<uint64_t>(__float_as_uint(v)) << 32) | (0xffffffffu - static_cast<uint32_t>(w));
}

template <bool NEST>
__device__ __forceinline__ void note_entry(float v, int64_t w, int32_t dtok, uint64_t &best, float &pd) {
    if constexpr (NEST) {
        const uint64_t k = best_key(v, w);
        best = k > best ? k : best;
        pd = w == dtok ? v : pd;
    }
}

// p_M row b with weight lam of p_LM: weights wj (unnormalised softmax terms, sum z) are scatter-added
// onto their tokens tok (-1: none) one vocabulary tile of TILE entries at a
// time in LDS; each tile's p_LM slice sits in registers in pre (the first
// tile's loaded by the caller when PREFETCHED) and is mixed with 16-byte
// accesses.  With no neighbour (z = 0) p_kNN is 0.
//
// NEST: the decoding outputs of the row from the values just written (Algorithm
// 1; Section 3.3): the greedy token w_t = the lowest argmax of p_M and its
// value, p_M at the row's draft token, and the span start -- the nearest
// neighbour carrying w_t, from nkey = (distance bits << 32 | key id) of each
// neighbour (~0 for none) -- with the span flag lambda <= delta.
//
// dtok is the draft token of the row (NEST; -1 for none), read by the caller
// at its start.  A workgroup writes entries [c0, c1) of the row (c1 < 0: to
// the end), c0 a multiple of 4 kT.  ONE_TILE: they fit one tile, and pre
// holds it.  SCATTERED (with ONE_TILE): the caller has already added the
// weights into acc and ordered that with a barrier.  When `slices` workgroups
// share the row, the one with first_slice set writes what belongs to the row
// as a whole but not to an entry, and the NEST outputs come from the last of
// them to finish, through m.best[b] and m.ticket[b] (both zero before the
// first one starts).
template <int PER, int TILE, bool NEST, bool PREFETCHED, bool ONE_TILE = false, bool SCATTERED = false>
__device__ __forceinline__ void mix_row(const float (&wj)[PER], const int32_t (&tok)[PER], const uint64_t (&nkey)[PER],
                                        float z, float lam, const MixArgs &m, int64_t b, float *acc,
                                        float4 (&pre)[TILE / 4 / kT], int32_t dtok, int64_t c0 = 0,
                                        int64_t c1 = -1, int slices = 1, bool first_slice = true) {
    const int64_t end = c1 < 0 ? m.V : c1;  // this workgroup writes entries [c0, end)
    constexpr int kV4 = TILE / 4 / kT;  // float4 per thread per tile
    const int tid = threadIdx.x;
    const float scale = z > 0.0f ? (1.0f - lam) / z : 0.0f;
    const float *plm = m.p_lm + b * m.V;
    float *pm = m.p_m + b * m.V;
    const bool vec4 = mix_vec4(m, b);
    float bv = -1.0f;  // this thread's largest entry and its token
    int32_t bw = 0;
    float pd = 0.0f;   // p_M(dtok), held by the thread that writes it
    if constexpr (!PREFETCHED) mix_prefetch(m, b, c0, pre);
    int64_t v0 = c0;
    do {  // at least once, so that pre is used on every path
        const int64_t nv = (end - v0 < TILE) ? end - v0 : TILE;
        const bool more = v0 + TILE < end;
        if (!ONE_TILE && v0 != c0) mix_prefetch(m, b, v0, pre);
        if constexpr (!SCATTERED) {
#pragma unroll
            for (int q = 0; q < kV4; ++q) reinterpret_cast<float4 *>(acc)[q * kT + tid] = make_float4(0.f, 0.f, 0.f, 0.f);
            __syncthreads();
#pragma unroll
            for (int q = 0; q < PER; ++q)
                if (tok[q] >= v0 && tok[q] < v0 + nv) atomicAdd(&acc[tok[q] - v0], wj[q]);
            __syncthreads();
        }
        if (vec4) {
            // Stores with no branch around them (lanes past the row store to a
            // sink), so that no store waits for the one before it.
            float4 *dst = reinterpret_cast<float4 *>(pm + v0);
#pragma unroll
            for (int q = 0; q < kV4; ++q) {
                const int64_t i = static_cast<int64_t>(q) * kT + tid;
                const bool in = i < nv / 4;
                const float4 a4 = reinterpret_cast<const float4 *>(acc)[i];
                float4 o;
                o.x = fmaf(lam, pre[q].x, a4.x * scale);
                o.y = fmaf(lam, pre[q].y, a4.y * scale);
                o.z = fmaf(lam, pre[q].z, a4.z * scale);
                o.w = fmaf(lam, pre[q].w, a4.w * scale);
                *(in ? dst + i : &g_mix_sink) = o;
                if constexpr (NEST) {
                    const int32_t w = static_cast<int32_t>(v0 + 4 * i);
                    note_entry<NEST>(in ? o.x : -1.0f, w, dtok, bv, bw, pd);
                    note_entry<NEST>(in ? o.y : -1.0f, w + 1, dtok, bv, bw, pd);
                    note_entry<NEST>(in ? o.z : -1.0f, w + 2, dtok, bv, bw, pd);
                    note_entry<NEST>(in ? o.w : -1.0f, w + 3, dtok, bv, bw, pd);
                }
            }
        } else {
            consume_loads(pre);  // unused on this path
            for (int64_t i = tid; i < nv; i += kT) {
                const float o = fmaf(lam, plm[v0 + i], acc[i] * scale);
                pm[v0 + i] = o;
                note_entry<NEST>(o, static_cast<int32_t>(v0 + i), dtok, bv, bw, pd);
            }
        }
        if (!ONE_TILE && more) __syncthreads();  // acc is cleared again next
        v0 += TILE;
    } while (!ONE_TILE && v0 < end);
    if constexpr (NEST) {
        __shared__ uint32_t red[2 * kNumWaves];
        __shared__ uint64_t row_best;  // sliced rows: the row's largest entry key, seen by the last workgroup
        __shared__ uint32_t is_last;
        float top = bv;
        uint32_t wtu = static_cast<uint32_t>(bw);
        block_argmax(top, wtu, red);
        if (m.p_draft != nullptr) {
            // entry w was written by thread (w / 4) % kT on the 16-byte path, w % kT otherwise
            const bool valid = dtok >= 0 && dtok < m.V;
            const bool mine = valid && dtok >= c0 && dtok < end &&
                              (vec4 ? ((dtok / 4) % kT == tid) : (dtok % kT == tid));
            if (mine) m.p_draft[b] = pd;
            if (tid == 0 && first_slice && !valid) m.p_draft[b] = 0.0f;
        }
        if (slices > 1) {
            // The row's workgroups each add their largest entry to the row's
            // 64-bit maximum (largest value, then lowest token; 0 for none) and
            // count themselves; the last one to count goes on with the row's.
            if (tid == 0) {
                atomicMax(reinterpret_cast<unsigned long long *>(m.best + b),
                          static_cast<unsigned long long>(top >= 0.0f ? best_key(top, wtu) : 0ull));
                const uint32_t t = __hip_atomic_fetch_add(m.ticket + b, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
                is_last = t == static_cast<uint32_t>(slices - 1) ? 1u : 0u;
                row_best = is_last ? __hip_atomic_load(m.best + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0ull;
            }
            __syncthreads();
            if (is_last == 0u) return;
            const uint64_t k = row_best;
            top = k == 0ull ? -1.0f : __uint_as_float(static_cast<uint32_t>(k >> 32));
            wtu = k == 0ull ? 0u : 0xffffffffu - static_cast<uint32_t>(k);
        }
        const int32_t wt = static_cast<int32_t>(wtu);
        // the nearest neighbour carrying wt: smallest (distance bits, id)
        uint32_t nd = ~0u, ni = ~0u;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const uint32_t kd = static_cast<uint32_t>(nkey[q] >> 32), ki = static_cast<uint32_t>(nkey[q]);
            const bool better = tok[q] == wt && (kd < nd || (kd == nd && ki < ni));
            nd = better ? kd : nd;
            ni = better ? ki : ni;
        }
        // over the block: the argmax of 0x7f800000 - bits (a nonnegative float
        // that grows as the distance shrinks), lowest id among equals
        float nearness = nd == ~0u ? -1.0f : __uint_as_float(kMaskedBits - nd);
        block_argmax(nearness, ni, red);
        const uint64_t near = nearness < 0.0f ? ~0ull : static_cast<uint64_t>(ni);
        if (tid == 0) {
            const int32_t span = near == ~0ull ? -1 : static_cast<int32_t>(static_cast<uint32_t>(near));
            m.next_token[b] = wt;
            m.p_max[b] = top;
            m.span_key[b] = span;
            m.use_span[b] = (lam <= m.delta && span >= 0) ? 1 : 0;
        }
    }
}

// ------------------------------------------------------------------ kernels

// General path: any row length, r <= KNNLM_MAX_R.
template <int CAP, int MODE>
__global__ __launch_bounds__(kT) void k_select(SelectArgs a, MixArgs m) {
    constexpr bool MIX = MODE != kNoMix;
    __shared__ uint32_t hist[kSelectBins];
    __shared__ uint64_t cand[CAP];
    __shared__ __align__(16) float acc[MIX ? kVocabTile : 4];
    __shared__ Shared sh;

    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int32_t dtok = draft_token<MODE>(m, b);
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
    uint32_t bmin, bmax;
    row_range(a, b, N, bmin, bmax, sh);
    const uint32_t n = select_stream<CAP>(a.dist + b * a.ld, N, r_eff, bmin, bmax, cand, hist, sh);

    int32_t *out_ids = a.ids + b * a.r;
    float *out_d = a.dists + b * a.r;
    for (int j = tid; j < a.r; j += kT) {
        if (static_cast<uint32_t>(j) < r_eff && static_cast<uint32_t>(j) < n) {
            const uint64_t key = cand[j];
            out_ids[j] = static_cast<int32_t>(key & 0xffffffffu);
            out_d[j] = __uint_as_float(static_cast<uint32_t>(key >> 32));
        } else {  // fewer than r unmasked keys, or a key set smaller than r (a false hint)
            out_ids[j] = -1;
            out_d[j] = __builtin_huge_valf();
        }
    }
    if constexpr (MIX) {
        const uint32_t rn = r_eff < n ? r_eff : n;
        const float dmin = rn > 0 ? __uint_as_float(static_cast<uint32_t>(cand[0] >> 32)) : 0.0f;
        const float dlast = rn > 0 ? __uint_as_float(static_cast<uint32_t>(cand[rn - 1] >> 32)) : 0.0f;
        const float lam = query_lambda<MODE>(m, b, dmin, dlast);
        float wj[kPer];
        int32_t tok[kPer];
        uint64_t nkey[kPer];
        float zpart = 0.0f;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const uint32_t j = static_cast<uint32_t>(q * kT + tid);
            tok[q] = -1;
            wj[q] = 0.0f;
            nkey[q] = ~0ull;
            if (j < rn) {
                const uint64_t key = cand[j];
                wj[q] = expf(-m.mu * (__uint_as_float(static_cast<uint32_t>(key >> 32)) - dmin));
                zpart += wj[q];
                tok[q] = m.values[k0 + static_cast<int32_t>(key & 0xffffffffu)];
                nkey[q] = key;
            }
        }
        const float z = block_sum(zpart, sh.red_f);
        float4 pre[kVocabTile / 4 / kT];
        mix_row<kPer, kVocabTile, MODE == kMixNest, false>(wj, tok, nkey, z, lam, m, b, acc, pre, dtok);
    }
}

// Fast path: rows of at most kFastMaxN keys (ld <= kFastMaxN), r <= 1024.
template <int MODE>
__global__ __launch_bounds__(kT) void k_select_fast(SelectArgs a, MixArgs m) {
    constexpr bool MIX = MODE != kNoMix;
    constexpr int kSelBytes = 2 * kFastCap * 8 + 2 * kSelectBins * 4;
    constexpr int kSmem = (MIX && kVocabTileFast * 4 > kSelBytes) ? kVocabTileFast * 4 : kSelBytes;
    constexpr int kPre = MIX ? kVocabTileFast / 4 / kT : 1;
    __shared__ __align__(16) unsigned char smem[kSmem];
    __shared__ Shared sh;
    uint64_t *cand = reinterpret_cast<uint64_t *>(smem);                                   // [kFastCap]
    uint64_t *tmp = reinterpret_cast<uint64_t *>(smem + kFastCap * 8);                     // [kFastCap]
    uint32_t *hist = reinterpret_cast<uint32_t *>(smem + 2 * kFastCap * 8);                // [2 * kSelectBins]
    float *acc = reinterpret_cast<float *>(smem);  // mixture phase, after the keys are in registers

    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int32_t dtok = draft_token<MODE>(m, b);
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    if (N > kFastMaxN) N = kFastMaxN;  // the host launches this kernel only when ld <= kFastMaxN
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
    const float *drow = a.dist + b * a.ld;

    // The whole row into registers: element (u, e) is key 4 * tid + u * 4096 + e.
    uint4 v[kFastU];
#pragma unroll
    for (int u = 0; u < kFastU; ++u) {
        const int64_t i = (static_cast<int64_t>(u) * kT + tid) * 4;
        v[u] = (i < N) ? *reinterpret_cast<const uint4 *>(drow + i) : make_uint4(0u, 0u, 0u, 0u);
    }
    const int32_t limit = static_cast<int32_t>(N) - 4 * tid;
    uint32_t bmin, bmax;
    row_range(a, b, N, bmin, bmax, sh);

    // Threshold on the distance bits: every key if they fit, else from a
    // histogram of one key per thread, sampled across the whole row.
    uint32_t thr = bmax + 1u;
    if (N > kFastCap) {
        const int us = tid & (kFastU - 1), es = (tid >> 4) & 3;
        uint32_t sbits = 0u;
#pragma unroll
        for (int u = 0; u < kFastU; ++u)
            if (u == us) sbits = lane_word(v[u], es);
        const bool sval = elem_off(us, es) < limit;
        for (int i = tid; i < kSelectBins; i += kT) hist[i] = 0u;
        __syncthreads();
        const uint32_t w = bmax + 1u - bmin;
        const int shift = range_shift(w);
        if (sval && sbits - bmin < w) atomicAdd(&hist[(sbits - bmin) >> shift], 1u);
        const uint64_t votes = __ballot(sval);  // every lane votes
        if ((tid & (kWave - 1)) == 0) sh.red_u[0][tid / kWave] = static_cast<uint32_t>(__popcll(votes));
        __syncthreads();
        uint32_t ns = 0;
#pragma unroll
        for (int wv = 0; wv < kNumWaves; ++wv) ns += sh.red_u[0][wv];
        // Sample rank aiming at about r + 4 sd + 4 samples' worth of keys: the
        // count of keys below the threshold then lies in [r, kFastCap] with
        // overwhelming probability; otherwise the general path runs.
        const float k0f = ceilf(static_cast<float>(r_eff) * static_cast<float>(ns) / static_cast<float>(N));
        const uint32_t ks = static_cast<uint32_t>(k0f + ceilf(4.0f * sqrtf(k0f)) + 4.0f);
        if (ks < ns) {
            if (tid == 0) { sh.lo = bmin; sh.hi = bmax + 1u; sh.below = 0u; sh.cnt = ns; }
            __syncthreads();
            pick_bin(hist, ks, shift, sh);
            thr = sh.hi;  // bin end: at least ks samples lie below it
            __syncthreads();
        }
    }

    // One compaction pass of the keys below the threshold.
    uint32_t c = 0;
#pragma unroll
    for (int u = 0; u < kFastU; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) c += (elem_off(u, e) < limit && lane_word(v[u], e) < thr) ? 1u : 0u;
    uint32_t pos = block_excl_scan(c, sh.wave_tot);
    if (tid == kT - 1) sh.total = pos + c;
    __syncthreads();
    const uint32_t C = sh.total;
    const bool fast = C >= r_eff && C <= static_cast<uint32_t>(kFastCap);
    if (c > 0 && pos + c <= static_cast<uint32_t>(kFastCap)) {
#pragma unroll
        for (int u = 0; u < kFastU; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (elem_off(u, e) < limit && lane_word(v[u], e) < thr)
                    cand[pos++] = sort_key(lane_word(v[u], e), static_cast<uint32_t>(4 * tid + elem_off(u, e)));
    }
    __syncthreads();
    uint64_t x = ~0ull;
    uint32_t nvalid = r_eff;  // neighbours found: fewer than r_eff only when masked keys leave too few
    if (fast) {
        // Sort every candidate (all keys below the threshold); the first r are pi.
        bucket_sort<kFastCap / kT>(cand, C, bmin, thr - bmin, hist, hist + kSelectBins, tmp, sh);
        x = static_cast<uint32_t>(tid) < r_eff ? cand[tid] : ~0ull;
    } else {
        // The sample misjudged the count: select over the streamed row.
        const uint32_t n = select_stream<kFastCap>(drow, N, r_eff, bmin, bmax, cand, hist, sh);
        nvalid = n < r_eff ? n : r_eff;
        x = static_cast<uint32_t>(tid) < nvalid ? cand[tid] : ~0ull;
    }
    __syncthreads();

    // Start fetching this query's p_LM row while the neighbours are written out.
    float4 pre[kPre];
    if constexpr (MIX) mix_prefetch(m, b, 0, pre);

    // Thread t holds the t-th nearest key (t < nvalid).
    const bool ok = static_cast<uint32_t>(tid) < nvalid;
    if (tid < a.r) {
        a.ids[b * a.r + tid] = ok ? static_cast<int32_t>(x & 0xffffffffu) : -1;
        a.dists[b * a.r + tid] = ok ? __uint_as_float(static_cast<uint32_t>(x >> 32)) : __builtin_huge_valf();
    }
    if constexpr (MIX) {
        int32_t tok[1] = {ok ? m.values[k0 + static_cast<int32_t>(x & 0xffffffffu)] : -1};
        const uint64_t nkey[1] = {ok ? x : ~0ull};
        const float dj = __uint_as_float(static_cast<uint32_t>(x >> 32));
        if (tid == 0) sh.dmin = ok ? dj : 0.0f;
        if (static_cast<uint32_t>(tid) == (nvalid > 0 ? nvalid - 1 : 0u)) sh.dlast = ok ? dj : 0.0f;
        __syncthreads();
        const float lam = query_lambda<MODE>(m, b, sh.dmin, sh.dlast);
        float wj[1] = {ok ? expf(-m.mu * (dj - sh.dmin)) : 0.0f};
        const float z = block_sum(wj[0], sh.red_f);
        mix_row<1, kVocabTileFast, MODE == kMixNest, true>(wj, tok, nkey, z, lam, m, b, acc, pre, dtok);
    }
}

// Split path: rows of at most kSplitMaxN keys, r <= kSplitMaxR, few queries.
// Where the streaming distance kernels left group minima (16- or 32-row tiles,
// at least 2 r groups a row) and the finish runs without a mixture or in
// vocabulary slices, the finish alone selects from them (GROUPS below).
// Otherwise query b's row is cut into `parts` parts of kSplitKeys keys so that
// one query keeps many CUs busy; two kernels, and no atomics or fences between
// workgroups (the kernel boundary orders them).
//
// Parts kernel (blockIdx.x = b * parts + part): every part of query b reads
// the same kSplitSamples keys sampled across the row (1024 runs of 4
// consecutive keys, one run every N / 1024) and takes as threshold the end of the histogram bin, over the
// samples' own range, that holds the ks-th smallest of them, ks aiming at
// about r + 4 sd + 4 samples' worth of keys; it writes its keys below the
// threshold to its own list (distance bits << 32 | key index << 12) and their
// count, and part 0 records the threshold.  With a fixed lambda and a finish
// that writes only the neighbours' entries, each part also writes its slice of
// the dense term of p_M: lambda * p_LM is what fmaf(lambda, p_LM, acc * scale)
// gives wherever no neighbour carries the token.  The part's keys and samples are requested before the row length is
// known (as if the row filled the stride) and corrected after.
constexpr int kSplitSamples = 4 * kT;

template <int MODE, bool DENSE_TERM>
__global__ __launch_bounds__(kT) void k_select_parts(SelectArgs a, MixArgs m, int parts) {
    // the dense term lambda * p_LM is known here; written here unless the
    // finish writes whole slices of the row
    constexpr bool DENSE = MODE == kMixFixed && DENSE_TERM;
    __shared__ __align__(16) uint32_t hist[kSelectBins];
    __shared__ Shared sh;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int64_t b = blockIdx.x / parts;
    const int part = static_cast<int>(blockIdx.x - b * parts);
    const float *drow = a.dist + b * a.ld;
    const int64_t ld = a.ld < kSplitMaxN ? a.ld : kSplitMaxN;  // the host launches this kernel only when ld <= kSplitMaxN
    if (tid == 0) {
        sh.ccount = 0u;
        sh.cmin = ~0u;
    }

    // Requests first: the part's keys (4 per thread), 4 samples per thread for
    // a full row, and the first float4 of the part's p_LM slice.
    const int64_t i0 = static_cast<int64_t>(part) * kSplitKeys + 4 * tid;
    uint4 v = make_uint4(~0u, ~0u, ~0u, ~0u);
    if (i0 < ld) v = *reinterpret_cast<const uint4 *>(drow + i0);
    // samples: 4 consecutive keys per thread, 1024 runs spread across the row
    // (a run starts at a multiple of 4 at most N - 4, so it stays in the row)
    uint4 sv = *reinterpret_cast<const uint4 *>(drow + (((static_cast<uint64_t>(tid) * static_cast<uint64_t>(ld)) >> 10) & ~3ull));
    int64_t v0 = 0, nv = 0;
    bool vec4 = false;
    float4 pl4 = make_float4(0.f, 0.f, 0.f, 0.f);
    if constexpr (DENSE) {
        const int64_t slice = ((m.V + parts - 1) / parts + 3) / 4 * 4;
        v0 = static_cast<int64_t>(part) * slice;
        nv = m.V - v0 < slice ? m.V - v0 : slice;
        if (nv < 0) nv = 0;
        vec4 = mix_vec4(m, b);
        if (vec4 && tid < nv / 4) pl4 = reinterpret_cast<const float4 *>(m.p_lm + b * m.V + v0)[tid];
    }
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > ld) N = ld;
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
    const bool sampled = N > kSplitCap;
    // words past the row end read as all-ones, above any threshold
    if (i0 >= N) v = make_uint4(~0u, ~0u, ~0u, ~0u);
    if (i0 + 1 >= N) v.y = ~0u;
    if (i0 + 2 >= N) v.z = ~0u;
    if (i0 + 3 >= N) v.w = ~0u;
    if (sampled && N != ld)  // a shorter row: sample it again
        sv = *reinterpret_cast<const uint4 *>(drow + (((static_cast<uint64_t>(tid) * static_cast<uint64_t>(N)) >> 10) & ~3ull));
    const uint32_t sb[4] = {sv.x, sv.y, sv.z, sv.w};

    uint32_t thr = kMaskedBits;  // a row that fits: every key (but masked ones)
    if (sampled) {
        // distances are >= +0 and never NaN: bits <= 0x7f800000, which only
        // masked keys reach; those samples are left out
        uint32_t smin = ~0u, smax = 0u;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            smin = sb[u] < kMaskedBits ? min(smin, sb[u]) : smin;
            smax = sb[u] < kMaskedBits ? max(smax, sb[u]) : smax;
        }
        block_minmax_u32(smin, smax, sh);
        if (smin > smax) smin = smax = 0u;  // every sample masked
        for (int i = tid; i < kSelectBins; i += kT) hist[i] = 0u;
        __syncthreads();
        const uint32_t w = smax + 1u - smin;
        const int shift = range_shift(w);
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (sb[u] - smin < w) atomicAdd(&hist[(sb[u] - smin) >> shift], 1u);
        const float k0f = ceilf(static_cast<float>(r_eff) * static_cast<float>(kSplitSamples) / static_cast<float>(N));
        const uint32_t ks = static_cast<uint32_t>(k0f + ceilf(4.0f * sqrtf(k0f)) + 4.0f);
        __syncthreads();
        if (tid < kWave) {
            // the end of the bin holding the ks-th sample: at least ks samples lie below it
            const uint32_t j = ks < static_cast<uint32_t>(kSplitSamples) ? wave_pick_bin(hist, ks, lane) : ~0u;
            const uint64_t end = static_cast<uint64_t>(smin) + ((static_cast<uint64_t>(j) + 1u) << shift);
            if (lane == 0) sh.hi = j == ~0u ? kMaskedBits : static_cast<uint32_t>(end < smax + 1ull ? end : smax + 1ull);
        }
    }
    __syncthreads();
    if (sampled) thr = sh.hi;

    // Keys below the threshold go to the part's list: each wave reserves its
    // range with one LDS atomic (the list's order is free: the finish sorts).
    uint32_t c = 0, cmin = ~0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t bits = lane_word(v, e);
        c += bits < thr ? 1u : 0u;
        cmin = bits < thr ? min(cmin, bits) : cmin;
    }
    const uint32_t incl = wave_incl_scan_u32(c, lane);
    const uint32_t wtot = readlane_u32(incl, kWave - 1);
    const uint32_t wmin = wave_allmin_u32(cmin);
    uint32_t base = 0;
    if (lane == 0 && wtot > 0) {
        base = atomicAdd(&sh.ccount, wtot);
        atomicMin(&sh.cmin, wmin);
    }
    uint32_t pos = readlane_u32(base, 0) + incl - c;
    const int64_t bp = b * parts + part;
    uint64_t *list = a.cand + bp * kSplitKeys;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t bits = lane_word(v, e);
        if (bits < thr)
            list[pos++] = (static_cast<uint64_t>(bits) << 32) | (static_cast<uint64_t>(static_cast<uint32_t>(i0) + e) << 12);
    }
    if constexpr (DENSE) {
        const float lam = m.lambda;
        float *pm = m.p_m + b * m.V + v0;
        const float *plm = m.p_lm + b * m.V + v0;
        if (vec4) {
            for (int64_t i = tid; i < nv / 4; i += kT) {
                const float4 x = i == tid ? pl4 : reinterpret_cast<const float4 *>(plm)[i];
                reinterpret_cast<float4 *>(pm)[i] =
                    make_float4(fmaf(lam, x.x, 0.0f), fmaf(lam, x.y, 0.0f), fmaf(lam, x.z, 0.0f), fmaf(lam, x.w, 0.0f));
            }
        } else {
            for (int64_t i = tid; i < nv; i += kT) pm[i] = fmaf(lam, plm[i], 0.0f);
        }
    }
    __syncthreads();
    if (tid == 0) {
        a.part_count[bp] = sh.ccount;
        a.part_min[bp] = sh.cmin;
        if (part == 0) a.part_thr[b] = thr;
        if (MODE == kMixNest && part == 0 && m.best != nullptr) {  // the sliced finish's row maximum and count
            m.best[b] = 0ull;
            m.ticket[b] = 0u;
        }
    }
}

// Finish kernel (one workgroup per query).  It loads the part counts together
// with the first kSplitCap / parts entries of every list, gathers the
// candidates into LDS (the rest of a longer list afterwards), and bucket-sorts
// them on their distance bits while their tokens load.  Then it writes pi;
// with mixing, each neighbour adds its unnormalised weight at its token in an
// LDS vocabulary tile that takes over the sort buffers, and the tokens' p_M
// entries are written.  If the sample misjudged the count (fewer than r
// candidates, or more than kSplitCap) it selects over the whole row instead.
// In LDS a candidate carries its slot (< 4096) in the low 12 bits, below the
// key index, which it cannot reorder since indices are distinct; the slot
// names where its token was staged.
constexpr int kFinishBinsLog2 = 12;  // 4096 buckets: about one candidate each where they crowd

template <int PER>
__device__ __forceinline__ void finish_sort(uint64_t *cand, uint32_t total, uint32_t lo, uint32_t thr, uint32_t *hist,
                                            uint64_t *tmp, Shared &sh, uint32_t keep) {
    bucket_sort<PER, kFinishBinsLog2, true>(cand, total, lo, thr - lo, hist, hist + (1 << kFinishBinsLog2), tmp, sh,
                                             NoHook(), keep);
}

// Zeroes the sliced finish's fixed-point vocabulary tile (32 bytes per thread).
__device__ __forceinline__ void clear_slice_tile(uint64_t *acc_s) {
    static_assert(kVocabSlice == 4 * kT, "four entries per thread");
    const uint4 z = make_uint4(0u, 0u, 0u, 0u);
    reinterpret_cast<uint4 *>(acc_s)[2 * threadIdx.x] = z;
    reinterpret_cast<uint4 *>(acc_s)[2 * threadIdx.x + 1] = z;
}

// The nonnegative 64-bit integer (hi << 32 | lo), below 2^42, in fp32: hi is
// exact in fp32 and hi * 2^32 + fp32(lo) is rounded once more (within an ulp
// of the integer; the same bits for the same integer).
__device__ __forceinline__ float fixed_to_float(uint32_t lo, uint32_t hi) {
    return fmaf(static_cast<float>(hi), 4294967296.0f, static_cast<float>(lo));
}

// GROUPS: no parts kernel.  The finish reads the row's group minima (from the
// distance stage: group 4 t + w holds the rows of distance tile t that wave w
// of the streaming kernel took, rows 4 gr t + w + 4 e for e < gr), takes as
// threshold the end of the histogram bin holding the r-th smallest of them, so
// that at least r groups, hence at least r keys, lie below it, lists in LDS
// the groups whose minimum is below it (a group whose minimum is not below it
// holds no key below it), loads those groups' distances, and keeps the keys
// below the threshold.  Then the same sort, fallback and mixture.
constexpr int kGroupItems = 12;                          // distances of listed groups loaded per thread
constexpr int kGroupList = kGroupItems * kT / 4;         // listed groups kept (of at least 4 keys each)

template <int MODE, bool SLICED, bool GROUPS, int GL = 0>
__global__ __launch_bounds__(kT) void k_select_finish(SelectArgs a, MixArgs m, int parts, int slices) {
    static_assert(!GROUPS || GL == 2 || GL == 4, "GL 16-byte loads of group minima per thread");
    constexpr bool MIX = MODE != kNoMix;
    static_assert(!SLICED || MIX, "slices are of the p_M row");
    constexpr int PER = kSplitCap / kT;
    constexpr int kSortBytes = 2 * kSplitCap * 8 + (8 << kFinishBinsLog2);
    constexpr int kSmem = MIX ? kSortBytes + kSplitCap * 4 + 16384 : kSortBytes;  // + tokens, + room for the tile
    static_assert(!MIX || kVocabTileFast * 4 <= kSmem, "the vocabulary tile fits over the sort buffers");
    __shared__ __align__(16) unsigned char smem[kSmem];
    uint64_t *cand = reinterpret_cast<uint64_t *>(smem);                          // [kSplitCap]
    uint64_t *tmp = cand + kSplitCap;                                              // [kSplitCap]
    uint32_t *hist = reinterpret_cast<uint32_t *>(tmp + kSplitCap);                // [2 << kFinishBinsLog2]: counts, starts
    int32_t *tok_of = reinterpret_cast<int32_t *>(smem + kSortBytes);              // [kSplitCap]
    float *acc = reinterpret_cast<float *>(smem);  // mixture: a vocabulary tile, over everything above
    // sliced: the slice's tile in fixed point (weight * 2^31, 64-bit integer
    // LDS atomics: exact, so independent of their order, and faster than fp32
    // LDS atomics where many neighbours share a token) over the sort's scratch,
    // then in fp32 over the bucket counts (both dead once the sort returns)
    uint64_t *acc_s = tmp;
    float *acc_f = reinterpret_cast<float *>(hist);
    static_assert(kVocabSlice * 8 <= kSplitCap * 8 && kVocabSlice * 4 <= (8 << kFinishBinsLog2),
                  "the slice's tiles fit over the sort scratch and the bucket counts");
    // GROUPS: the minima's histogram and the list of groups below the
    // threshold, over the sort's scratch too (both dead before the sort)
    uint32_t *ghist = reinterpret_cast<uint32_t *>(tmp);                           // [kSelectBins]
    uint32_t *glist = ghist + kSelectBins;                                         // [kGroupList]
    static_assert((kSelectBins + kGroupList) * 4 <= kSplitCap * 8, "histogram and list fit the sort scratch");
    __shared__ Shared sh;
    __shared__ uint32_t part_off[kWave + 1];

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int64_t b = SLICED ? blockIdx.x / slices : blockIdx.x;
    const int g = SLICED ? static_cast<int>(blockIdx.x - b * slices) : 0;  // the row's slice
    const int32_t dtok = draft_token<MODE>(m, b);
    const uint64_t *lists = a.cand + b * parts * kSplitKeys;
    const float *drow = a.dist + b * a.ld;

    // Lists: counts, threshold and the first `win` entries of every list, all
    // in flight together.  Groups: the row's group minima.
    const uint32_t win = GROUPS ? 0u : static_cast<uint32_t>(kSplitCap / parts);
    uint32_t cnt = 0u, pmin = ~0u, thr = 0u;
    uint64_t key[PER];
    uint4 gv[GROUPS ? GL : 1];
    if constexpr (GROUPS) {
        const int64_t nq4 = a.groups_per_set / 4;  // 16-byte words of a row's minima (groups_per_set % 4 == 0)
        const uint4 *gm = reinterpret_cast<const uint4 *>(a.group_min + b * a.groups_per_set);
#pragma unroll
        for (int u = 0; u < GL; ++u) {
            const int64_t i = static_cast<int64_t>(u) * kT + tid;
            gv[u] = gm[i < nq4 ? i : 0];  // unconditional: words past the row reread its first
        }
        if (tid == 0) {
            sh.total = 0u;
            sh.ccount = 0u;
        }
    } else {
        cnt = (tid < kWave && lane < parts) ? a.part_count[b * parts + lane] : 0u;
        pmin = (tid < kWave && lane < parts) ? a.part_min[b * parts + lane] : ~0u;
        thr = a.part_thr[b];
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const uint32_t e = static_cast<uint32_t>(q * kT + tid);
            const uint32_t p = e / win;
            key[q] = p < static_cast<uint32_t>(parts) ? lists[p * kSplitKeys + (e - p * win)] : ~0ull;
        }
    }
    // The p_LM entries this workgroup mixes: its slice, or the row's first tile
    // (loaded during the write-out below).
    float4 pre[SLICED ? kVocabSlice / 4 / kT : kVocabTileFast / 4 / kT];
    if constexpr (SLICED) mix_prefetch(m, b, static_cast<int64_t>(g) * kVocabSlice, pre);
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    if (N > kSplitMaxN) N = kSplitMaxN;
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
    // Bucket counts to clear while the loads are in flight.
    for (int i = tid; i < (1 << kFinishBinsLog2); i += kT) hist[i] = 0u;
    uint32_t total, lo;
    bool fast;
    if constexpr (GROUPS) {
        for (int i = tid; i < kSelectBins; i += kT) ghist[i] = 0u;
        const int gr = a.group_rows;  // 4 or 8
        // every group of the tiles that hold the row's keys (a group of the
        // last tile may hold no key: its minimum is then +infinity)
        const uint32_t ng = static_cast<uint32_t>((N + 4 * gr - 1) / (4 * gr) * 4);
        // groups past the row read as all-ones, above +infinity (masked keys) and any threshold
        uint32_t gmn = ~0u, gmx = 0u;
#pragma unroll
        for (int u = 0; u < GL; ++u) {
            const uint32_t g0 = static_cast<uint32_t>(u * kT + tid) * 4u;
            gv[u].x = g0 < ng ? gv[u].x : ~0u;
            gv[u].y = g0 + 1u < ng ? gv[u].y : ~0u;
            gv[u].z = g0 + 2u < ng ? gv[u].z : ~0u;
            gv[u].w = g0 + 3u < ng ? gv[u].w : ~0u;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t v = lane_word(gv[u], e);
                gmn = v < kMaskedBits ? min(gmn, v) : gmn;
                gmx = v < kMaskedBits ? max(gmx, v) : gmx;
            }
        }
        block_minmax_u32<false>(gmn, gmx, sh);  // its barrier also orders the clears above
        lo = gmn;
        if (gmn <= gmx) {
            const uint32_t w = gmx + 1u - gmn;
            const int shift = range_shift(w);
#pragma unroll
            for (int u = 0; u < GL; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t v = lane_word(gv[u], e);
                    if (v < kMaskedBits) atomicAdd(&ghist[(v - gmn) >> shift], 1u);
                }
            __syncthreads();
            if (tid < kWave) {
                // fewer than r groups: every unmasked key (then more than the sort holds, or all of them)
                const uint32_t j = wave_pick_bin(ghist, r_eff > 0 ? r_eff : 1u, lane);
                const uint64_t end = static_cast<uint64_t>(gmn) + ((static_cast<uint64_t>(j) + 1u) << shift);
                if (lane == 0) sh.hi = j == ~0u ? kMaskedBits : static_cast<uint32_t>(end < gmx + 1ull ? end : gmx + 1ull);
            }
            __syncthreads();
            thr = sh.hi;
        }
        // The groups below the threshold, listed in LDS (each wave reserves its slots with one LDS atomic).
        {
            uint32_t c = 0u;
#pragma unroll
            for (int u = 0; u < GL; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) c += lane_word(gv[u], e) < thr ? 1u : 0u;
            const uint32_t incl = wave_incl_scan_u32(c, lane);
            const uint32_t wtot = readlane_u32(incl, kWave - 1);
            uint32_t base = 0u;
            if (lane == 0 && wtot > 0u) base = atomicAdd(&sh.total, wtot);
            uint32_t pos = readlane_u32(base, 0) + incl - c;
#pragma unroll
            for (int u = 0; u < GL; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (lane_word(gv[u], e) < thr) {
                        if (pos < static_cast<uint32_t>(kGroupList)) glist[pos] = static_cast<uint32_t>(u * kT + tid) * 4u + e;
                        ++pos;
                    }
        }
        __syncthreads();
        // The listed groups' distances, one word per key, all in flight
        // together: group 4 t + w holds rows 4 gr t + w + 4 e, e < gr, of the row.
        const uint32_t items = sh.total * static_cast<uint32_t>(gr);
        const bool fits = items <= static_cast<uint32_t>(kGroupItems * kT);
        const int lg = gr == 8 ? 3 : 2;
        uint32_t dv[kGroupItems];
        uint32_t key_of[kGroupItems];  // each word's key index (N: none)
#pragma unroll
        for (int u = 0; u < kGroupItems; ++u) {
            const uint32_t i = static_cast<uint32_t>(u * kT + tid);
            const bool in = i < items && fits;
            const uint32_t gi = in ? glist[i >> lg] : 0u;
            const uint32_t row = ((gi >> 2) << (lg + 2)) + (gi & 3u) + 4u * (i & static_cast<uint32_t>(gr - 1));
            key_of[u] = in ? row : static_cast<uint32_t>(N);
            dv[u] = __float_as_uint(drow[in ? row : 0u]);  // unconditional: the row's first word otherwise
        }
        // The keys below the threshold, into the sort's buffer (each with its slot).
        uint32_t c = 0u;
#pragma unroll
        for (int u = 0; u < kGroupItems; ++u) c += (key_of[u] < N && dv[u] < thr) ? 1u : 0u;
        const uint32_t incl = wave_incl_scan_u32(c, lane);
        const uint32_t wtot = readlane_u32(incl, kWave - 1);
        uint32_t base = 0u;
        if (lane == 0 && wtot > 0u) base = atomicAdd(&sh.ccount, wtot);
        uint32_t pos = readlane_u32(base, 0) + incl - c;
#pragma unroll
        for (int u = 0; u < kGroupItems; ++u)
            if (key_of[u] < N && dv[u] < thr) {
                if (pos < static_cast<uint32_t>(kSplitCap))
                    cand[pos] = (static_cast<uint64_t>(dv[u]) << 32) | (static_cast<uint64_t>(key_of[u]) << 12) | pos;
                ++pos;
            }
        __syncthreads();  // the candidates are in LDS
        total = sh.ccount;
        fast = fits && total >= r_eff && total <= static_cast<uint32_t>(kSplitCap);
    } else {
        if (tid < kWave) {  // list starts, and whether any list is longer than its window
            const uint32_t incl = wave_incl_scan_u32(cnt, lane);
            if (lane < parts) part_off[lane] = incl - cnt;
            if (lane == parts - 1) part_off[parts] = incl;
            const uint32_t longest = wave_allmax_u32(cnt);
            const uint32_t cmin = wave_allmin_u32(pmin);
            if (lane == 0) {
                sh.found = longest > win ? 1u : 0u;
                sh.cmin = cmin;  // the smallest candidate distance bits
            }
        }
        __syncthreads();
        total = part_off[parts];
        lo = sh.cmin;
        fast = total >= r_eff && total <= static_cast<uint32_t>(kSplitCap);
    }

    uint64_t x = ~0ull;
    uint32_t id = 0;
    int32_t tok = -1;
    float plm_t = 0.0f;
    uint32_t nvalid = r_eff;  // neighbours found: fewer only when masked keys leave too few
    bool ok = static_cast<uint32_t>(tid) < r_eff;
    const float *plm_row = m.p_lm + b * m.V;
    if (fast) {
        uint32_t slot[PER];
        bool valid[PER];
        int32_t tv[PER];
        if constexpr (GROUPS) {
            // Tokens of the listed keys: unconditional loads (past the list, key 0's).
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                const uint32_t e = static_cast<uint32_t>(q * kT + tid);
                valid[q] = e < total;
                slot[q] = e;
                const uint32_t i = valid[q] ? static_cast<uint32_t>(cand[e]) >> 12 : 0u;
                tv[q] = MIX ? m.values[k0 + i] : -1;
            }
        } else {
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                const uint32_t e = static_cast<uint32_t>(q * kT + tid);
                const uint32_t p = e / win;
                const uint32_t pc = p < static_cast<uint32_t>(parts) ? p : static_cast<uint32_t>(parts - 1);
                const uint32_t i = e - p * win;
                const uint32_t start = part_off[pc], end = part_off[pc + 1];
                valid[q] = p < static_cast<uint32_t>(parts) && i < end - start;
                slot[q] = start + i;
                if (valid[q]) cand[slot[q]] = key[q] | slot[q];
            }
            // Tokens: unconditional loads (an invalid entry reads key 0's), so
            // that nothing waits for them before the sort needs them.
#pragma unroll
            for (int q = 0; q < PER; ++q)
                tv[q] = MIX ? m.values[k0 + (valid[q] ? (static_cast<uint32_t>(key[q]) >> 12) : 0u)] : -1;
            if (sh.found != 0u) {  // longer lists: the rest, one part after another (rare)
                for (int p = 0; p < parts; ++p) {
                    const uint32_t n_p = part_off[p + 1] - part_off[p];
                    for (uint32_t i = win + tid; i < n_p; i += kT) {
                        const uint64_t k = lists[p * kSplitKeys + i];
                        const uint32_t sl = part_off[p] + i;
                        cand[sl] = k | sl;
                        if constexpr (MIX) tok_of[sl] = m.values[k0 + (static_cast<uint32_t>(k) >> 12)];
                    }
                }
            }
            __syncthreads();  // the candidates are in LDS
        }
        if (total <= static_cast<uint32_t>(kSplitCap / 2))
            finish_sort<PER / 2>(cand, total, lo, thr, hist, tmp, sh, r_eff);
        else
            finish_sort<PER>(cand, total, lo, thr, hist, tmp, sh, r_eff);
        if constexpr (MIX) {
#pragma unroll
            for (int q = 0; q < PER; ++q)
                if (valid[q]) tok_of[slot[q]] = tv[q];
            if constexpr (SLICED) clear_slice_tile(acc_s);
            __syncthreads();
        }
        x = ok ? cand[tid] : ~0ull;
        id = static_cast<uint32_t>(x) >> 12;
        if (MIX && ok) tok = tok_of[static_cast<uint32_t>(x) & (kSplitCap - 1)];
    } else {
        // The sample misjudged the count: select over the whole row.
        uint32_t bmin, bmax;
        row_range(a, b, N, bmin, bmax, sh);
        const uint32_t n = select_stream<kSplitCap>(a.dist + b * a.ld, N, r_eff, bmin, bmax, cand, hist, sh);
        nvalid = n < r_eff ? n : r_eff;
        ok = static_cast<uint32_t>(tid) < nvalid;
        x = ok ? cand[tid] : ~0ull;
        id = static_cast<uint32_t>(x);
        if (MIX && ok) tok = m.values[k0 + id];
        if constexpr (SLICED) {
            clear_slice_tile(acc_s);
            __syncthreads();
        }
    }
    if (tok < 0 || tok >= m.V) tok = -1;  // tokens outside [0, V) carry no mass
    if (MODE == kMixFixed && !SLICED && tok >= 0) plm_t = plm_row[tok];  // needed only at the end
    // the nearest and (RRC) the r-th nearest distance: the ends of pi, in LDS in both branches above
    const float d0 = nvalid > 0 ? __uint_as_float(static_cast<uint32_t>(cand[0] >> 32)) : 0.0f;
    const float dlast = nvalid > 0 ? __uint_as_float(static_cast<uint32_t>(cand[nvalid - 1] >> 32)) : 0.0f;
    if constexpr (rrc_mode(MODE) && !SLICED) mix_prefetch(m, b, 0, pre);  // during the write-out
    if (g == 0 && tid < a.r) {
        a.ids[b * a.r + tid] = ok ? static_cast<int32_t>(id) : -1;
        a.dists[b * a.r + tid] = ok ? __uint_as_float(static_cast<uint32_t>(x >> 32)) : __builtin_huge_valf();
    }
    if constexpr (MIX) {
        const float dj = __uint_as_float(static_cast<uint32_t>(x >> 32));
        const float wj = ok ? expf(-m.mu * (dj - d0)) : 0.0f;
        const int64_t c0 = static_cast<int64_t>(g) * kVocabSlice;  // sliced: this workgroup's entries
        if constexpr (SLICED) {
            // wj <= 1, so wj * 2^31 fits 32 bits; it is an integer for wj >= 2^-8 (conversion exact) and
            // loses less than 2^-31 below; r such terms stay below 2^42
            if (tok >= c0 && tok < c0 + kVocabSlice)
                atomicAdd(reinterpret_cast<unsigned long long *>(acc_s + (tok - c0)),
                          static_cast<unsigned long long>(static_cast<uint32_t>(wj * 2147483648.0f)));
        }
        // Z; the barrier also ends every use of the sort buffers, which an
        // unsliced vocabulary tile then takes over, and orders a slice's
        // additions before its reads.
        const float wsum = wave_allsum(wj);
        if (lane == 0) sh.red_f[tid / kWave] = wsum;
        __syncthreads();
        float z = 0.0f;
#pragma unroll
        for (int w = 0; w < kNumWaves; ++w) z += sh.red_f[w];
        const float lam = query_lambda<MODE>(m, b, d0, dlast, g == 0);
        const float w1[1] = {wj};
        const int32_t t1[1] = {tok};
        const uint64_t k1[1] = {ok ? ((x >> 32) << 32) | id : ~0ull};
        if constexpr (SLICED) {
            // this workgroup's slice of the row, with any lambda
            const int64_t c1 = m.V - c0 < kVocabSlice ? m.V : c0 + kVocabSlice;
            // each thread's four entries back to fp32 (the row writer's 16-byte path reads its own
            // 16 bytes; its 4-byte path, entries tid + 1024 k, needs a barrier)
            const uint4 e01 = reinterpret_cast<const uint4 *>(acc_s)[2 * tid];
            const uint4 e23 = reinterpret_cast<const uint4 *>(acc_s)[2 * tid + 1];
            constexpr float kInv = 1.0f / 2147483648.0f;
            reinterpret_cast<float4 *>(acc_f)[tid] =
                make_float4(fixed_to_float(e01.x, e01.y) * kInv, fixed_to_float(e01.z, e01.w) * kInv,
                            fixed_to_float(e23.x, e23.y) * kInv, fixed_to_float(e23.z, e23.w) * kInv);
            if (!mix_vec4(m, b)) __syncthreads();
            mix_row<1, kVocabSlice, MODE == kMixNest, true, true, true>(w1, t1, k1, z, lam, m, b, acc_f, pre, dtok,
                                                                        c0, c1, slices, g == 0);
            return;
        } else if constexpr (rrc_mode(MODE)) {
            // lambda_t is known only now: the whole row, tile by tile
            mix_row<1, kVocabTileFast, MODE == kMixNest, true>(w1, t1, k1, z, lam, m, b, acc, pre, dtok);
            return;
        }
        const float scale = z > 0.0f ? (1.0f - lam) / z : 0.0f;
        // Each neighbour adds its weight at its token in a vocabulary tile
        // (only the touched entries are cleared); the tokens' p_M entries are
        // then written, duplicates writing the same value; the parts kernel
        // wrote lambda * p_LM everywhere else.
        for (int64_t t0 = 0; t0 < m.V; t0 += kVocabTileFast) {
            const bool in = tok >= t0 && tok < t0 + kVocabTileFast;
            if (t0 > 0) __syncthreads();  // the previous tile's reads are done
            if (in) acc[tok - t0] = 0.0f;
            __syncthreads();
            if (in) atomicAdd(&acc[tok - t0], wj);
            __syncthreads();
            if (in) m.p_m[b * m.V + tok] = fmaf(lam, plm_t, acc[tok - t0] * scale);
        }
    }
}

// Standalone mixture on caller-given neighbours (any order): one workgroup per query.
template <int MODE>
__global__ __launch_bounds__(kT) void k_mix(MixArgs m) {
    __shared__ __align__(16) float acc[kVocabTile];
    __shared__ float red_f[kNumWaves];
    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int32_t dtok = draft_token<MODE>(m, b);
    const int64_t s = set_of_query(m.query_offsets, m.S, b);
    const int64_t k0 = m.key_offsets[s];
    const int64_t N = m.key_offsets[s + 1] - k0;
    float dj[kPer];
    int32_t id[kPer];
    // a neighbour whose id lies outside [0, N) is absent: no weight, no part in
    // the softmax's maximum or (RRC) in the ratio
    bool present[kPer];
    float dmin = __builtin_huge_valf(), neg_dmax = __builtin_huge_valf();
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int j = q * kT + tid;
        dj[q] = j < m.r ? m.dists[b * m.r + j] : __builtin_huge_valf();
        id[q] = j < m.r ? m.ids[b * m.r + j] : -1;
        present[q] = j < m.r && id[q] >= 0 && id[q] < N;
        if (present[q]) {
            dmin = fminf(dmin, dj[q]);
            neg_dmax = fminf(neg_dmax, -dj[q]);
        }
    }
    dmin = block_min(dmin, red_f);
    float dmax = 0.0f;
    if constexpr (rrc_mode(MODE)) dmax = -block_min(neg_dmax, red_f);
    const bool any = dmin != __builtin_huge_valf();
    const float lam = query_lambda<MODE>(m, b, any ? dmin : 0.0f, any ? dmax : 0.0f);
    float wj[kPer];
    int32_t tok[kPer];
    uint64_t nkey[kPer];
    float zpart = 0.0f;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        wj[q] = present[q] ? expf(-m.mu * (dj[q] - dmin)) : 0.0f;
        zpart += wj[q];
        tok[q] = present[q] ? m.values[k0 + id[q]] : -1;
        nkey[q] = present[q] ? (static_cast<uint64_t>(__float_as_uint(dj[q])) << 32) | static_cast<uint32_t>(id[q])
                             : ~0ull;
    }
    const float z = block_sum(zpart, red_f);
    float4 pre[kVocabTile / 4 / kT];
    mix_row<kPer, kVocabTile, MODE == kMixNest, false>(wj, tok, nkey, z, lam, m, b, acc, pre, dtok);
}

// Wide path: rows longer than the split path's (ld > kSplitMaxN), r <= kWideMaxR,
// when the distance stage's tiles are fine enough (at least 2 r tiles per row).
// Query b's row is cut into `parts` slices, one workgroup each, so that few
// queries with long rows still fill the chip; two kernels, no atomics or
// fences between workgroups.
//
// Parts kernel (blockIdx.x = b * parts + part): the threshold is the end of
// the histogram bin (2048 bins over their range) that holds the r-th smallest
// of the row's tile minima: at least r tiles have their minimum below it, so
// at least r keys do.  With at least 2 r tiles it keeps about r to 1.5 r keys
// of random data.  Every part computes it (from tiles_per_set floats); each
// streams its slice once, 16 keys per thread per step with the next step's
// loads in flight, and appends the keys below the threshold (distance bits
// << 32 | key index) to its list, each wave reserving its slots with one LDS
// atomic; the list keeps its first kWideCap keys and the count is the true one.
//
// Finish kernel (one workgroup per query): if the lists hold between r and
// kWideCap keys in all, it gathers them into LDS and bucket-sorts them (4096
// buckets over [smallest, threshold)), else it selects over the streamed row
// (the general path's select); then pi and the mixture as on the general path.
constexpr int kWideMaxR = 2048;
constexpr int kWideCap = kSplitKeys;       // candidates per list and in all (the lists share the split layout)
constexpr int kWideU = 4;                  // 16-byte loads per thread per step
constexpr int64_t kWideStep = static_cast<int64_t>(kT) * 4 * kWideU;  // keys per step (16384)

__global__ __launch_bounds__(kT) void k_select_wide_parts(SelectArgs a, int parts) {
    __shared__ __align__(16) uint32_t hist[kSelectBins];
    __shared__ uint32_t qtile[kT];  // tiles of the current chunk with keys below the threshold
    __shared__ Shared sh;
    if (a.gate != nullptr && *a.gate != a.gate_run) return;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int64_t b = blockIdx.x / parts;
    const int part = static_cast<int>(blockIdx.x - b * parts);
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
    const float *drow = a.dist + b * a.ld;
    if (tid == 0) sh.ccount = 0u;

    // The threshold from the tile minima (masked keys, at +infinity, stay out).
    const int64_t ntiles = (N + a.rows_per_tile - 1) / a.rows_per_tile;
    const float *tmin = a.tile_min + b * a.tiles_per_set;
    uint32_t lo = ~0u, hi = 0u;
    for (int64_t t = tid; t < ntiles; t += kT) {
        const uint32_t v = __float_as_uint(tmin[t]);
        lo = v < kMaskedBits ? min(lo, v) : lo;
        hi = v < kMaskedBits ? max(hi, v) : hi;
    }
    block_minmax_u32(lo, hi, sh);
    uint32_t thr = 0u;  // no unmasked key: nothing below
    if (lo <= hi) {
        for (int i = tid; i < kSelectBins; i += kT) hist[i] = 0u;
        __syncthreads();
        const uint32_t w = hi + 1u - lo;
        const int shift = range_shift(w);
        for (int64_t t = tid; t < ntiles; t += kT) {
            const uint32_t v = __float_as_uint(tmin[t]);
            if (v < kMaskedBits) atomicAdd(&hist[(v - lo) >> shift], 1u);
        }
        __syncthreads();
        if (tid < kWave) {
            // fewer than r tiles: every unmasked key (the finish then selects over the row)
            const uint32_t j = wave_pick_bin(hist, r_eff > 0 ? r_eff : 1u, lane);
            const uint64_t end = static_cast<uint64_t>(lo) + ((static_cast<uint64_t>(j) + 1u) << shift);
            if (lane == 0) sh.hi = j == ~0u ? kMaskedBits : static_cast<uint32_t>(end < hi + 1ull ? end : hi + 1ull);
        }
        __syncthreads();
        thr = sh.hi;
    }

    // This part's tiles, kT at a time: those whose minimum is below the
    // threshold are listed in LDS (a tile whose minimum is not below it holds
    // no key below it), and only their rows are streamed, as one run of
    // nq * R rows, 16 keys per thread per step with the next step's loads in
    // flight.  R is a multiple of 8, so a 16-byte load stays in one tile.
    const int64_t R = a.rows_per_tile;
    const int64_t tpp = (ntiles + parts - 1) / parts;
    const int64_t tb = static_cast<int64_t>(part) * tpp;
    const int64_t te = tb + tpp < ntiles ? tb + tpp : ntiles;
    const uint32_t R32 = static_cast<uint32_t>(R);
    uint64_t *list = a.cand + (b * parts + part) * static_cast<int64_t>(kWideCap);
    for (int64_t c0 = tb; c0 < te; c0 += kT) {
        __syncthreads();  // the previous chunk's reads of sh.total and qtile are done
        if (tid == 0) sh.total = 0u;
        __syncthreads();
        const int64_t tt = c0 + tid;
        const uint32_t qual = (tt < te && __float_as_uint(tmin[tt]) < thr) ? 1u : 0u;
        const uint32_t qincl = wave_incl_scan_u32(qual, lane);
        const uint32_t qtot = readlane_u32(qincl, kWave - 1);
        uint32_t qbase = 0u;
        if (lane == 0 && qtot > 0) qbase = atomicAdd(&sh.total, qtot);
        if (qual) qtile[readlane_u32(qbase, 0) + qincl - 1u] = static_cast<uint32_t>(tt);
        __syncthreads();
        const uint32_t nrows = sh.total * R32;  // <= kT * 4096
        // virtual row v of the run: row (v % R) of listed tile v / R; past the run, or past the row's
        // end in its last tile, a lane reads the row's first keys and counts nothing
        auto row_of = [&](uint32_t v) __attribute__((always_inline)) -> int64_t {
            const uint32_t slot = v / R32;
            return v < nrows ? static_cast<int64_t>(qtile[slot < static_cast<uint32_t>(kT) ? slot : 0u]) * R + (v - slot * R32)
                             : N;
        };
        auto load = [&](uint32_t base, int64_t (&ri)[kWideU], uint4 (&v)[kWideU]) __attribute__((always_inline)) {
#pragma unroll
            for (int u = 0; u < kWideU; ++u) {
                ri[u] = row_of(base + (static_cast<uint32_t>(u) * kT + tid) * 4u);
                v[u] = *reinterpret_cast<const uint4 *>(drow + (ri[u] < N ? ri[u] : 0));
            }
        };
        if (nrows == 0u) continue;
        int64_t ri[kWideU], rn[kWideU];
        uint4 v[kWideU], nx[kWideU];
        load(0u, ri, v);
        for (uint32_t base = 0u; base < nrows; base += static_cast<uint32_t>(kWideStep)) {
            load(base + static_cast<uint32_t>(kWideStep), rn, nx);
            uint32_t c = 0;
#pragma unroll
            for (int u = 0; u < kWideU; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) c += (ri[u] + e < N && lane_word(v[u], e) < thr) ? 1u : 0u;
            const uint32_t incl = wave_incl_scan_u32(c, lane);
            const uint32_t wtot = readlane_u32(incl, kWave - 1);
            uint32_t wbase = 0u;
            if (lane == 0 && wtot > 0) wbase = atomicAdd(&sh.ccount, wtot);
            uint32_t pos = readlane_u32(wbase, 0) + incl - c;
#pragma unroll
            for (int u = 0; u < kWideU; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t bits = lane_word(v[u], e);
                    if (ri[u] + e < N && bits < thr) {
                        if (pos < static_cast<uint32_t>(kWideCap))
                            list[pos] = sort_key(bits, static_cast<uint32_t>(ri[u] + e));
                        ++pos;
                    }
                }
#pragma unroll
            for (int u = 0; u < kWideU; ++u) {
                v[u] = nx[u];
                ri[u] = rn[u];
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        a.part_count[b * parts + part] = sh.ccount;
        if (part == 0) a.part_thr[b] = thr;
    }
}

template <int MODE>
__global__ __launch_bounds__(kT) void k_select_wide_finish(SelectArgs a, MixArgs m, int parts) {
    constexpr bool MIX = MODE != kNoMix;
    constexpr int kBinsLog2 = 12;
    __shared__ __align__(16) uint64_t cand[kWideCap];
    __shared__ __align__(16) uint64_t tmp[kWideCap];  // sort scratch, then the mixture's vocabulary tile
    __shared__ __align__(16) uint32_t bins[2 << kBinsLog2];
    __shared__ Shared sh;
    __shared__ uint32_t part_off[kWave + 1];
    static_assert(kVocabTile * 4 <= kWideCap * 8, "the vocabulary tile fits over the sort scratch");
    float *acc = reinterpret_cast<float *>(tmp);
    if (a.gate != nullptr && *a.gate != a.gate_run) return;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int64_t b = blockIdx.x;
    const int32_t dtok = draft_token<MODE>(m, b);
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
    const uint64_t *lists = a.cand + b * parts * static_cast<int64_t>(kWideCap);
    if (tid < kWave) {
        const uint32_t cnt = lane < parts ? a.part_count[b * parts + lane] : 0u;
        const uint32_t incl = wave_incl_scan_u32(cnt, lane);
        if (lane < parts) part_off[lane] = incl - cnt;
        if (lane == parts - 1) part_off[parts] = incl;
    }
    __syncthreads();
    const uint32_t total = part_off[parts];
    uint32_t n;
    if (total >= r_eff && total <= static_cast<uint32_t>(kWideCap)) {
        uint32_t mn = ~0u;
        for (uint32_t e = tid; e < total; e += kT) {
            int p = 0;
            while (p + 1 < parts && part_off[p + 1] <= e) ++p;
            const uint64_t key = lists[p * static_cast<int64_t>(kWideCap) + (e - part_off[p])];
            cand[e] = key;
            mn = min(mn, static_cast<uint32_t>(key >> 32));
        }
        uint32_t mx = 0u;
        block_minmax_u32(mn, mx, sh);  // also orders the gather before the sort
        const uint32_t thr = a.part_thr[b];
        bucket_sort<kWideCap / kT, kBinsLog2>(cand, total, mn, thr > mn ? thr - mn : 1u, bins, bins + (1 << kBinsLog2),
                                             tmp, sh, NoHook(), r_eff);
        n = total;
    } else {
        // The threshold kept too few or too many keys: select over the streamed row.
        uint32_t bmin, bmax;
        row_range(a, b, N, bmin, bmax, sh);
        n = select_stream<kWideCap>(a.dist + b * a.ld, N, r_eff, bmin, bmax, cand, bins, sh);
    }

    int32_t *out_ids = a.ids + b * a.r;
    float *out_d = a.dists + b * a.r;
    const uint32_t rn = r_eff < n ? r_eff : n;
    for (int j = tid; j < a.r; j += kT) {
        if (static_cast<uint32_t>(j) < rn) {
            const uint64_t key = cand[j];
            out_ids[j] = static_cast<int32_t>(key & 0xffffffffu);
            out_d[j] = __uint_as_float(static_cast<uint32_t>(key >> 32));
        } else {  // fewer than r unmasked keys, or a key set smaller than r (a false hint)
            out_ids[j] = -1;
            out_d[j] = __builtin_huge_valf();
        }
    }
    if constexpr (MIX) {
        const float dmin = rn > 0 ? __uint_as_float(static_cast<uint32_t>(cand[0] >> 32)) : 0.0f;
        const float dlast = rn > 0 ? __uint_as_float(static_cast<uint32_t>(cand[rn - 1] >> 32)) : 0.0f;
        const float lam = query_lambda<MODE>(m, b, dmin, dlast);
        float wj[kPer];
        int32_t tok[kPer];
        uint64_t nkey[kPer];
        float zpart = 0.0f;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const uint32_t j = static_cast<uint32_t>(q * kT + tid);
            tok[q] = -1;
            wj[q] = 0.0f;
            nkey[q] = ~0ull;
            if (j < rn) {
                const uint64_t key = cand[j];
                wj[q] = expf(-m.mu * (__uint_as_float(static_cast<uint32_t>(key >> 32)) - dmin));
                zpart += wj[q];
                tok[q] = m.values[k0 + static_cast<int32_t>(key & 0xffffffffu)];
                nkey[q] = key;
            }
        }
        const float z = block_sum(zpart, sh.red_f);  // its barrier also ends the sort scratch's use
        float4 pre[kVocabTile / 4 / kT];
        mix_row<kPer, kVocabTile, MODE == kMixNest, false>(wj, tok, nkey, z, lam, m, b, acc, pre, dtok);
    }
}

// Fused select (query batches on long rows), threshold kernel: one workgroup
// per query.  The sample is the first sample_rows rows of every
// sample_every-th distance tile of the query's row, whose distances (and the
// tiles' extrema over them) the distance stage has written.  The threshold is
// the end of the histogram bin (2048 bins) holding the ks-th smallest sampled
// distance, ks = k0 + ceil(4 sqrt(k0)) + 4 with k0 = ceil(r M / N) for M
// sampled keys of N: about r + 4 standard deviations of keys of random data
// lie below it.  The histogram's range ends at the ks-th smallest of the
// pieces' minima when there are enough pieces (ks pieces, so at least ks
// sampled keys, lie at or below it), so only the sample's low end is counted.
// The sample's own keys below the threshold start the query's list; thread 0
// of query 0 clears the fallback word.  Masked keys (+infinity) stay out.
constexpr int kFusedU = 4;  // 16-byte loads per thread per step over the sample

__global__ __launch_bounds__(kT) void k_fused_threshold(SelectArgs a, FusedArgs f) {
    __shared__ __align__(16) uint32_t hist[kSelectBins];
    __shared__ uint32_t pmin[kT];  // the pieces' minima (up to kT pieces)
    __shared__ Shared sh;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int64_t b = blockIdx.x;
    if (b == 0 && tid == 0) *f.fallback = 0u;
    if (tid == 0) sh.ccount = 0u;
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
    const int64_t R = a.rows_per_tile, sp = f.sample_rows, se = f.sample_every;
    const int64_t ntiles = (N + R - 1) / R;
    const int64_t npieces = (ntiles + se - 1) / se;
    const float *drow = a.dist + b * a.ld;
    const float *tmin = a.tile_min + b * a.tiles_per_set;
    // piece p: rows [p se R, p se R + rows_p), rows_p = sp but for the last piece
    const int64_t last0 = (npieces - 1) * se * R;
    const int64_t last_rows = N - last0 < sp ? N - last0 : sp;
    const int64_t M = npieces > 0 ? (npieces - 1) * sp + last_rows : 0;  // sampled keys
    const int64_t slots_pp = sp / 4;                                     // 16-byte slots per piece
    const int64_t nslots = npieces * slots_pp;

    // The sample's range: its pieces' minima (the tile extrema the distance stage wrote over them).
    uint32_t lo = ~0u, hi = 0u;
    for (int64_t p = tid; p < npieces; p += kT) {
        const uint32_t v = __float_as_uint(tmin[p * se]);
        lo = v < kMaskedBits ? min(lo, v) : lo;
        if (p < kT) pmin[p] = v;  // an all-masked piece reads as 0xffffffff
    }
    const float k0f = ceilf(static_cast<float>(r_eff) * static_cast<float>(M) / static_cast<float>(N > 0 ? N : 1));
    const uint32_t ks = static_cast<uint32_t>(k0f + ceilf(4.0f * sqrtf(k0f)) + 4.0f);
    __syncthreads();
    // the end of the range: the ks-th smallest piece minimum (rank by comparison), else +infinity
    uint32_t hb = kMaskedBits;
    if (npieces <= kT && static_cast<int64_t>(ks) <= npieces) {
        if (tid < npieces) {
            const uint32_t v = pmin[tid];
            uint32_t rank = 0;
            for (int64_t j = 0; j < npieces; ++j) {
                const uint32_t u = pmin[j];
                rank += (u < v || (u == v && j < tid)) ? 1u : 0u;
            }
            if (rank == ks - 1u && v < kMaskedBits) sh.hi = v;
            if (rank == ks - 1u && v >= kMaskedBits) sh.hi = kMaskedBits - 1u;
        }
        __syncthreads();
        hb = sh.hi;
    } else {
        hi = 0u;
        for (int64_t p = tid; p < npieces; p += kT) {
            const uint32_t v = __float_as_uint(a.tile_max[b * a.tiles_per_set + p * se]);
            hi = v < kMaskedBits ? max(hi, v) : hi;
        }
    }
    block_minmax_u32(lo, hi, sh);
    if (hb != kMaskedBits) hi = hb;
    // Step over the sample: kFusedU slots per thread; slot e is piece e / slots_pp, its 16 bytes
    // at 4 (e % slots_pp) rows in (inside the tile, so inside the row's stride); past the
    // sample a lane rereads the last slot and counts nothing.
    auto step = [&](int64_t e0, uint4 (&v)[kFusedU], int64_t (&row)[kFusedU], int64_t (&lim)[kFusedU])
        __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kFusedU; ++u) {
            const int64_t e = e0 + static_cast<int64_t>(u) * kT + tid;
            const int64_t ec = e < nslots ? e : nslots - 1;
            const int64_t p = ec / slots_pp;
            row[u] = p * se * R + 4 * (ec - p * slots_pp);
            const int64_t pend = p * se * R + (p == npieces - 1 ? last_rows : sp);
            lim[u] = e < nslots ? pend : 0;  // elements at row + k < lim[u] are sampled
            v[u] = *reinterpret_cast<const uint4 *>(drow + row[u]);
        }
    };
    uint32_t thr = kMaskedBits;  // every unmasked key: too small a sample to judge
    if (lo <= hi && static_cast<int64_t>(ks) < M) {
        for (int i = tid; i < kSelectBins; i += kT) hist[i] = 0u;
        __syncthreads();
        const uint32_t w = hi + 1u - lo;
        const int shift = range_shift(w);
        for (int64_t e0 = 0; e0 < nslots; e0 += static_cast<int64_t>(kT) * kFusedU) {
            uint4 v[kFusedU];
            int64_t row[kFusedU], lim[kFusedU];
            step(e0, v, row, lim);
#pragma unroll
            for (int u = 0; u < kFusedU; ++u)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t bits = lane_word(v[u], k);
                    if (row[u] + k < lim[u] && bits - lo < w) atomicAdd(&hist[(bits - lo) >> shift], 1u);
                }
        }
        __syncthreads();
        if (tid < kWave) {
            const uint32_t j = wave_pick_bin(hist, ks, lane);
            const uint64_t end = static_cast<uint64_t>(lo) + ((static_cast<uint64_t>(j) + 1u) << shift);
            if (lane == 0) sh.hi = j == ~0u ? kMaskedBits : static_cast<uint32_t>(end < hi + 1ull ? end : hi + 1ull);
        }
        __syncthreads();
        thr = sh.hi;
    }
    // The sample's keys below the threshold: the start of the query's list.
    uint64_t *list = f.list + b * static_cast<int64_t>(kFusedCap);
    for (int64_t e0 = 0; e0 < nslots; e0 += static_cast<int64_t>(kT) * kFusedU) {
        uint4 v[kFusedU];
        int64_t row[kFusedU], lim[kFusedU];
        step(e0, v, row, lim);
        uint32_t c = 0;
#pragma unroll
        for (int u = 0; u < kFusedU; ++u)
#pragma unroll
            for (int k = 0; k < 4; ++k) c += (row[u] + k < lim[u] && lane_word(v[u], k) < thr) ? 1u : 0u;
        const uint32_t incl = wave_incl_scan_u32(c, lane);
        const uint32_t wtot = readlane_u32(incl, kWave - 1);
        uint32_t wbase = 0u;
        if (lane == 0 && wtot > 0) wbase = atomicAdd(&sh.ccount, wtot);
        uint32_t pos = readlane_u32(wbase, 0) + incl - c;
#pragma unroll
        for (int u = 0; u < kFusedU; ++u)
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t bits = lane_word(v[u], k);
                if (row[u] + k < lim[u] && bits < thr) {
                    if (pos < static_cast<uint32_t>(kFusedCap))
                        list[pos] = sort_key(bits, static_cast<uint32_t>(row[u] + k));
                    ++pos;
                }
            }
    }
    __syncthreads();
    if (tid == 0) {
        f.count[b] = sh.ccount;
        f.thr[b] = thr;
    }
}

// Fused select, check kernel (one workgroup): the fallback word is set when a
// query's list holds fewer than min(r, N) or more than kFusedCap candidates.
__global__ __launch_bounds__(kT) void k_fused_check(SelectArgs a, FusedArgs f, int64_t B) {
    int bad = 0;
    for (int64_t b = threadIdx.x; b < B; b += kT) {
        const int64_t s = set_of_query(a.query_offsets, a.S, b);
        int64_t N = a.key_offsets[s + 1] - a.key_offsets[s];
        if (N > a.ld) N = a.ld;
        const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
        const uint32_t c = f.count[b];
        bad |= (c < r_eff || c > static_cast<uint32_t>(kFusedCap)) ? 1 : 0;
    }
    if (__syncthreads_or(bad) && threadIdx.x == 0) *f.fallback = 1u;
}

__global__ void k_set_word(uint32_t *word, uint32_t v) {
    if (threadIdx.x == 0) *word = v;
}

template <int MODE>
hipError_t launch_sel_fused(const SelectArgs &a, const MixArgs &m, const FusedArgs &f, int64_t B, hipStream_t st) {
    if (B < 1 || B > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const int wparts = select_wide_parts(B, a.ld, a.r, a.tiles_per_set);
    if (wparts < 1 || a.tile_min == nullptr || a.tile_max == nullptr) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(B)), block(kT);
    // from the lists, unless the fallback word is set
    SelectArgs lf = a;
    lf.cand = f.list;
    lf.part_count = f.count;
    lf.part_thr = f.thr;
    lf.gate = f.fallback;
    lf.gate_run = 0u;
    hipLaunchKernelGGL((k_select_wide_finish<MODE>), grid, block, 0, st, lf, m, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // otherwise the wide select over the distance matrix
    SelectArgs lw = a;
    lw.gate = f.fallback;
    lw.gate_run = 1u;
    hipLaunchKernelGGL(k_select_wide_parts, dim3(static_cast<unsigned>(B * wparts)), block, 0, st, lw, wparts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((k_select_wide_finish<MODE>), grid, block, 0, st, lw, m, wparts);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_sel(const SelectArgs &a, const MixArgs &m, int64_t B, hipStream_t st) {
    if (B == 0) return hipSuccess;
    if (B > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    if (a.tile_min == nullptr || a.tile_max == nullptr) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(B)), block(kT);
    const int parts = select_split_parts(B, a.ld, a.r);
    if (parts > 0) {
        if (a.cand == nullptr || a.part_count == nullptr || a.part_thr == nullptr) return hipErrorInvalidValue;
        // With mixing and few rows, the finish runs once per vocabulary slice
        // of each row, every one of those workgroups selecting pi again, so
        // that the row is written by many CUs.
        constexpr bool MIX = MODE != kNoMix;
        const int64_t slices = MIX ? (m.V + kVocabSlice - 1) / kVocabSlice : 1;
        const bool sliced = MIX && B * slices <= kSliceMaxBlocks &&
                            (MODE != kMixNest || (m.best != nullptr && m.ticket != nullptr));
        if (a.group_min != nullptr && (!MIX || sliced)) {  // no parts kernel: the finish reads the group minima
            if (a.group_rows != 4 && a.group_rows != 8) return hipErrorInvalidValue;
            if (a.groups_per_set % 4 != 0 || a.groups_per_set > kGroupMaxPerRow) return hipErrorInvalidValue;
            const bool wide = a.groups_per_set > 2 * 4 * kT;  // more than two 16-byte words of minima per thread
            if constexpr (MIX) {
                const dim3 sgrid(static_cast<unsigned>(B * slices));
                if (wide)
                    hipLaunchKernelGGL((k_select_finish<MODE, true, true, 4>), sgrid, block, 0, st, a, m, 0,
                                       static_cast<int>(slices));
                else
                    hipLaunchKernelGGL((k_select_finish<MODE, true, true, 2>), sgrid, block, 0, st, a, m, 0,
                                       static_cast<int>(slices));
            } else {
                if (wide)
                    hipLaunchKernelGGL((k_select_finish<MODE, false, true, 4>), grid, block, 0, st, a, m, 0, 1);
                else
                    hipLaunchKernelGGL((k_select_finish<MODE, false, true, 2>), grid, block, 0, st, a, m, 0, 1);
            }
            return hipGetLastError();
        }
        const dim3 pgrid(static_cast<unsigned>(B * parts));
        if constexpr (MODE == kMixFixed) {  // the dense term: in the parts kernel unless the finish is sliced
            if (sliced)
                hipLaunchKernelGGL((k_select_parts<MODE, false>), pgrid, block, 0, st, a, m, parts);
            else
                hipLaunchKernelGGL((k_select_parts<MODE, true>), pgrid, block, 0, st, a, m, parts);
        } else {
            hipLaunchKernelGGL((k_select_parts<MODE, false>), pgrid, block, 0, st, a, m, parts);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if constexpr (MIX) {
            if (sliced) {
                hipLaunchKernelGGL((k_select_finish<MODE, true, false>), dim3(static_cast<unsigned>(B * slices)), block, 0,
                                   st, a, m, parts, static_cast<int>(slices));
                return hipGetLastError();
            }
        }
        hipLaunchKernelGGL((k_select_finish<MODE, false, false>), grid, block, 0, st, a, m, parts, 1);
        return hipGetLastError();
    }
    const int wparts = select_wide_parts(B, a.ld, a.r, a.tiles_per_set);
    if (wparts > 0) {
        if (a.cand == nullptr || a.part_count == nullptr || a.part_thr == nullptr) return hipErrorInvalidValue;
        hipLaunchKernelGGL(k_select_wide_parts, dim3(static_cast<unsigned>(B * wparts)), block, 0, st, a, wparts);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((k_select_wide_finish<MODE>), grid, block, 0, st, a, m, wparts);
        return hipGetLastError();
    }
    if (a.ld <= kFastMaxN && a.r <= kT) {
        hipLaunchKernelGGL((k_select_fast<MODE>), grid, block, 0, st, a, m);
        return hipGetLastError();
    }
    switch (select_capacity(a.r)) {
    case 2048: hipLaunchKernelGGL((k_select<2048, MODE>), grid, block, 0, st, a, m); break;
    case 4096: hipLaunchKernelGGL((k_select<4096, MODE>), grid, block, 0, st, a, m); break;
    case 8192: hipLaunchKernelGGL((k_select<8192, MODE>), grid, block, 0, st, a, m); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

int select_split_parts(int64_t B, int64_t ld, int r) {
    if (B < 1 || ld < 1 || ld > kSplitMaxN || r > kSplitMaxR) return 0;
    const int64_t parts = (ld + kSplitKeys - 1) / kSplitKeys;
    return B * parts <= kSplitMaxBlocks ? static_cast<int>(parts) : 0;
}

int select_group_rows(int64_t B, int64_t ld, int r, int rows_per_tile, bool streaming) {
    if (!streaming || select_split_parts(B, ld, r) == 0) return 0;
    if (rows_per_tile != 16 && rows_per_tile != 32) return 0;
    const int gr = rows_per_tile / 4;  // the streaming kernels' four waves each take a quarter of a tile
    const int64_t groups = ld / gr;
    if (groups > kGroupMaxPerRow || groups < 2 * static_cast<int64_t>(r)) return 0;
    return gr;
}

int select_wide_parts(int64_t B, int64_t ld, int r, int64_t tiles_per_set) {
    if (B < 1 || ld <= kSplitMaxN || r > kWideMaxR || tiles_per_set < 2 * static_cast<int64_t>(r)) return 0;
    int64_t parts = (kWideBlocks + B - 1) / B;  // about kWideBlocks workgroups
    const int64_t by_len = ld / kWideStep;      // at least one step of keys per part
    if (parts > by_len) parts = by_len;
    if (parts > kWave) parts = kWave;           // the finish scans the counts with one wave
    return parts < 1 ? 1 : static_cast<int>(parts);
}

int select_capacity(int r) {
    int p = 1;
    while (p < r) p <<= 1;
    int cap = 2 * p;
    if (cap < 2048) cap = 2048;
    return cap;  // <= 8192 for r <= KNNLM_MAX_R
}

hipError_t launch_fused_threshold(const SelectArgs &args, const FusedArgs &f, int64_t B, hipStream_t stream) {
    if (B < 1 || B > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    if (args.tile_min == nullptr || f.sample_rows < 4 || f.sample_rows % 4 != 0 || f.sample_rows > args.rows_per_tile ||
        f.sample_every < 1)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_fused_threshold, dim3(static_cast<unsigned>(B)), dim3(kT), 0, stream, args, f);
    return hipGetLastError();
}

hipError_t launch_fused_check(const SelectArgs &args, const FusedArgs &f, int64_t B, hipStream_t stream) {
    hipLaunchKernelGGL(k_fused_check, dim3(1), dim3(kT), 0, stream, args, f, B);
    return hipGetLastError();
}

hipError_t launch_select_fused(const SelectArgs &args, const MixArgs *mix, const FusedArgs &f, int64_t B,
                               hipStream_t stream) {
    if (mix == nullptr) {
        MixArgs none{};
        return launch_sel_fused<kNoMix>(args, none, f, B, stream);
    }
    if (mix->next_token != nullptr) {
        if (!mix->rrc || mix->p_max == nullptr || mix->span_key == nullptr || mix->use_span == nullptr)
            return hipErrorInvalidValue;
        return launch_sel_fused<kMixNest>(args, *mix, f, B, stream);
    }
    return mix->rrc ? launch_sel_fused<kMixRrc>(args, *mix, f, B, stream)
                    : launch_sel_fused<kMixFixed>(args, *mix, f, B, stream);
}

hipError_t launch_set_word(uint32_t *word, uint32_t v, hipStream_t stream) {
    hipLaunchKernelGGL(k_set_word, dim3(1), dim3(kWave), 0, stream, word, v);
    return hipGetLastError();
}

hipError_t launch_select(const SelectArgs &args, int64_t B, hipStream_t stream) {
    MixArgs none{};
    return launch_sel<kNoMix>(args, none, B, stream);
}

hipError_t launch_select_mix(const SelectArgs &args, const MixArgs &mix, int64_t B, hipStream_t stream) {
    if (mix.next_token != nullptr) {
        if (!mix.rrc || mix.p_max == nullptr || mix.span_key == nullptr || mix.use_span == nullptr)
            return hipErrorInvalidValue;
        return launch_sel<kMixNest>(args, mix, B, stream);
    }
    return mix.rrc ? launch_sel<kMixRrc>(args, mix, B, stream) : launch_sel<kMixFixed>(args, mix, B, stream);
}

hipError_t launch_mix(const MixArgs &args, int64_t B, hipStream_t stream) {
    if (B == 0) return hipSuccess;
    if (B > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    if (args.rrc)
        hipLaunchKernelGGL(k_mix<kMixRrc>, dim3(static_cast<unsigned>(B)), dim3(kT), 0, stream, args);
    else
        hipLaunchKernelGGL(k_mix<kMixFixed>, dim3(static_cast<unsigned>(B)), dim3(kT), 0, stream, args);
    return hipGetLastError();
}

}  // namespace knnlm
