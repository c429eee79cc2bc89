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
// the index makes every key distinct.  A radix refinement narrows a range
// known to hold the r-th smallest key -- first on the distance bits, then, if
// a single distance value remains, on the key index -- with 2048-bin LDS
// histograms until every key before the range's end fits in LDS; those keys
// are compacted as 64-bit (bits << 32 | i) words, bitonic-sorted, and the
// first r are the answer.
// The range starts from the per-tile extrema the distance stage leaves, so one
// histogram pass usually suffices.  Every pass streams the distance row in
// 16 Ki-key batches (four 16-byte loads per thread), the next batch loading
// while the current one is processed.
//
// Mixture (eq. non-parametric and eq. kNN-LM), when p_m is given: the softmax
// of mu * s over the r neighbours (the largest mu * s, i.e. the smallest
// distance, is subtracted first), scattered onto the neighbours' value tokens
// in 8 Ki-entry LDS tiles of the vocabulary with LDS float atomics (tokens no
// neighbour carries get 0; duplicates accumulate), then
// p_M = fmaf(lambda, p_LM, acc * ((1 - lambda) / Z)), so lambda = 1 returns p_LM
// bit for bit.  The order of the LDS atomics is not fixed, so p_kNN may differ
// between runs in the last bits.
#include "knnlm_device.h"
#include "knnlm_internal.h"

namespace knnlm {

namespace {

constexpr int kNumWaves = kSelectThreads / kWave;
constexpr int kU = 4;                                             // 16-byte loads per thread per batch
constexpr int64_t kBatch = static_cast<int64_t>(kSelectThreads) * 4 * kU;  // keys per batch (16384)
constexpr int kVocabTile = 8192;                                  // vocabulary entries per LDS tile

__device__ __forceinline__ uint64_t sort_key(uint32_t dbits, int64_t i) {
    return (static_cast<uint64_t>(dbits) << 32) | static_cast<uint32_t>(i);
}

// Exclusive prefix sum of one value per thread over the 1024-thread block.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t *wave_tot) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const uint32_t incl = wave_incl_scan_u32(v, lane);
    if (lane == kWave - 1) wave_tot[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        uint32_t t = lane < kNumWaves ? wave_tot[lane] : 0u;
        t = wave_incl_scan_u32(t, lane);
        if (lane < kNumWaves) wave_tot[lane] = t;  // inclusive totals
    }
    __syncthreads();
    const uint32_t before = wave == 0 ? 0u : wave_tot[wave - 1];
    __syncthreads();  // wave_tot may be reused right after
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

// Batch `b` of a distance row: thread t holds keys (u * 1024 + t) * 4 + e of
// the batch, e < 4, for u < kU.  Keys past N are never used.
__device__ __forceinline__ void load_batch(const float *drow, int64_t N, int64_t b, uint4 (&v)[kU]) {
    const int64_t base = b * kBatch;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const int64_t i = base + (static_cast<int64_t>(u) * kSelectThreads + threadIdx.x) * 4;
        v[u] = (i < N) ? *reinterpret_cast<const uint4 *>(drow + i) : make_uint4(0u, 0u, 0u, 0u);
    }
}

// Position of element (u, e) of this thread inside its batch, relative to the
// thread's first element: keys of a batch are at base + u * 4096 + e with
// base = batch start + 4 * threadIdx.x, and the key is valid iff this offset
// is below limit = N - base.
// Prefetch batch bb + 1 (zeros past the last batch).
__device__ __forceinline__ void next_batch(const float *drow, int64_t N, int32_t bb, int64_t nbatch, uint4 (&nx)[kU]) {
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

__device__ __forceinline__ int32_t elem_off(int u, int e) { return u * kSelectThreads * 4 + e; }

__device__ __forceinline__ uint32_t lane_word(const uint4 &v, int e) {
    return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w;
}

constexpr int kPer = (KNNLM_MAX_R + kSelectThreads - 1) / kSelectThreads;  // neighbours per thread

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

// p_M row b: the weights wj (unnormalised softmax terms, sum z) are
// scatter-added onto their tokens tok (-1: none) one vocabulary tile at a time
// in LDS, and each tile of p_LM is mixed and written with 16-byte accesses.
__device__ __forceinline__ void mix_row(const float (&wj)[kPer], const int32_t (&tok)[kPer], float z,
                                        const MixArgs &m, int64_t b, float *acc) {
    const int tid = threadIdx.x;
    const float lam = m.lambda;
    const float scale = (1.0f - lam) / z;
    const float *plm = m.p_lm + b * m.V;
    float *pm = m.p_m + b * m.V;
    const bool vec4 = (m.V % 4 == 0) && ((reinterpret_cast<uintptr_t>(plm) | reinterpret_cast<uintptr_t>(pm)) & 15u) == 0;
    for (int64_t v0 = 0; v0 < m.V; v0 += kVocabTile) {
        const int64_t nv = (m.V - v0 < kVocabTile) ? m.V - v0 : kVocabTile;
        for (int i = tid; i < kVocabTile; i += kSelectThreads) acc[i] = 0.0f;
        __syncthreads();
#pragma unroll
        for (int q = 0; q < kPer; ++q)
            if (tok[q] >= v0 && tok[q] < v0 + nv) atomicAdd(&acc[tok[q] - v0], wj[q]);
        __syncthreads();
        if (vec4) {
            const float4 *src = reinterpret_cast<const float4 *>(plm + v0);
            float4 *dst = reinterpret_cast<float4 *>(pm + v0);
            for (int64_t i = tid; i < nv / 4; i += kSelectThreads) {
                const float4 p = src[i];
                float4 o;
                o.x = fmaf(lam, p.x, acc[4 * i + 0] * scale);
                o.y = fmaf(lam, p.y, acc[4 * i + 1] * scale);
                o.z = fmaf(lam, p.z, acc[4 * i + 2] * scale);
                o.w = fmaf(lam, p.w, acc[4 * i + 3] * scale);
                dst[i] = o;
            }
        } else {
            for (int64_t i = tid; i < nv; i += kSelectThreads) pm[v0 + i] = fmaf(lam, plm[v0 + i], acc[i] * scale);
        }
        __syncthreads();
    }
}

template <int CAP, bool MIX>
__global__ __launch_bounds__(kSelectThreads) void k_select(SelectArgs a, MixArgs m) {
    __shared__ uint32_t hist[kSelectBins];
    __shared__ uint64_t cand[CAP];
    __shared__ float acc[MIX ? kVocabTile : 1];
    __shared__ uint32_t red_u[2][kNumWaves];
    __shared__ uint32_t wave_tot[kNumWaves];
    __shared__ float red_f[kNumWaves];
    __shared__ uint32_t sh_lo, sh_hi, sh_below, sh_cnt, sh_found, sh_fix;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int64_t b = blockIdx.x;
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    const float *drow = a.dist + b * a.ld;
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);
    const int64_t nbatch = (N + kBatch - 1) / kBatch;

    // Range of the keys from the per-tile extrema (or one pass over the row).
    uint32_t bmin = 0xffffffffu, bmax = 0u;
    uint4 v[kU], nx[kU];
    if (a.tile_min != nullptr) {
        const int64_t ntiles = (N + a.rows_per_tile - 1) / a.rows_per_tile;
        for (int64_t t = tid; t < ntiles; t += kSelectThreads) {
            bmin = min(bmin, __float_as_uint(a.tile_min[b * a.tiles_per_set + t]));
            bmax = max(bmax, __float_as_uint(a.tile_max[b * a.tiles_per_set + t]));
        }
    } else {
        load_batch(drow, N, 0, v);
        for (int32_t bb = 0; bb < nbatch; ++bb) {
            next_batch(drow, N, bb, nbatch, nx);
            const int32_t limit = static_cast<int32_t>(N) - (bb * static_cast<int32_t>(kBatch) + 4 * tid);
#pragma unroll
            for (int u = 0; u < kU; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (elem_off(u, e) < limit) {
                        bmin = min(bmin, lane_word(v[u], e));
                        bmax = max(bmax, lane_word(v[u], e));
                    }
            advance(v, nx);
        }
    }
    bmin = wave_allmin_u32(bmin);
    bmax = wave_allmax_u32(bmax);
    if (lane == 0) {
        red_u[0][wave] = bmin;
        red_u[1][wave] = bmax;
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t mn = red_u[0][0], mx = red_u[1][0];
        for (int w = 1; w < kNumWaves; ++w) {
            mn = min(mn, red_u[0][w]);
            mx = max(mx, red_u[1][w]);
        }
        if (N == 0) { mn = 0u; mx = 0u; }
        sh_lo = mn;
        sh_hi = mx + 1u;  // distances are >= +0, so mx < 0x80000000
        sh_below = 0u;
        sh_cnt = static_cast<uint32_t>(N);
        sh_fix = 0u;
    }
    __syncthreads();
    // The candidate range is [lo, hi) on distance bits while fix == 0; once it
    // holds a single distance value fv, it becomes [lo, hi) on key indices
    // among the keys at exactly fv (fix == 1).  `below` counts the keys known
    // to precede the range, `cnt` the keys inside it.
    uint32_t lo = sh_lo, hi = sh_hi, fv = 0u, fix = 0u;
    uint32_t below = sh_below, cnt = sh_cnt;

    // Refinement: keep the range holding the r-th smallest key.  Each pass
    // shrinks it by 2^10 at least (or switches to the index regime), so a few
    // passes always suffice; the cap and the found flag only guard against
    // inconsistent inputs.
    for (int pass = 0; pass < 12 && below + cnt > static_cast<uint32_t>(CAP); ++pass) {
        if (fix == 0u && hi - lo == 1u) {  // one distance value left: order by index
            fix = 1u;
            fv = lo;
            lo = 0u;
            hi = static_cast<uint32_t>(N);
        }
        const uint32_t w = hi - lo;  // >= 2 here
        const int nbits = 32 - __clz(static_cast<int>(w - 1u));
        const int shift = nbits > kSelectBinsLog2 ? nbits - kSelectBinsLog2 : 0;
        for (int i = tid; i < kSelectBins; i += kSelectThreads) hist[i] = 0u;
        if (tid == 0) sh_found = 0u;
        __syncthreads();
        load_batch(drow, N, 0, v);
        for (int32_t bb = 0; bb < nbatch; ++bb) {
            next_batch(drow, N, bb, nbatch, nx);
            const int32_t base = bb * static_cast<int32_t>(kBatch) + 4 * tid;
            const int32_t limit = static_cast<int32_t>(N) - base;
            if (!fix) {
#pragma unroll
                for (int u = 0; u < kU; ++u)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t off = lane_word(v[u], e) - lo;
                        if (elem_off(u, e) < limit && off < w) atomicAdd(&hist[off >> shift], 1u);
                    }
            } else {
#pragma unroll
                for (int u = 0; u < kU; ++u)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t off = static_cast<uint32_t>(base + elem_off(u, e)) - lo;
                        if (elem_off(u, e) < limit && off < w && lane_word(v[u], e) == fv)
                            atomicAdd(&hist[off >> shift], 1u);
                    }
            }
            advance(v, nx);
        }
        __syncthreads();
        // thread t owns bins 2t and 2t+1
        const uint32_t c0 = hist[2 * tid], c1 = hist[2 * tid + 1];
        const uint32_t excl = block_excl_scan(c0 + c1, wave_tot);
        const uint32_t need = r_eff - below;  // >= 1
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
            sh_lo = nlo;
            sh_hi = nhi < hi ? static_cast<uint32_t>(nhi) : hi;
            sh_below = below + before;
            sh_cnt = cj;
            sh_found = 1u;
        }
        __syncthreads();
        const bool found = sh_found != 0u;
        lo = sh_lo; hi = sh_hi; below = sh_below; cnt = sh_cnt;
        __syncthreads();
        if (!found) break;
    }

    // Compaction of every key before the end of the range (below + cnt <= CAP
    // of them), at offsets from a block scan of the per-thread counts.
    uint32_t written = 0;
    load_batch(drow, N, 0, v);
    for (int32_t bb = 0; bb < nbatch; ++bb) {
        next_batch(drow, N, bb, nbatch, nx);
        const int32_t base = bb * static_cast<int32_t>(kBatch) + 4 * tid;
        const int32_t limit = static_cast<int32_t>(N) - base;
        // a key is taken iff it precedes the end of the range
        const uint32_t end_bits = fix ? fv : hi;
        const uint32_t end_idx = fix ? hi : 0u;  // at bits == fv: indices below hi (none outside fix)
        uint32_t c = 0;
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t bits = lane_word(v[u], e);
                const uint32_t i = static_cast<uint32_t>(base + elem_off(u, e));
                const bool take = bits < end_bits || (bits == end_bits && i < end_idx);
                c += (elem_off(u, e) < limit && take) ? 1u : 0u;
            }
        uint32_t pos = written + block_excl_scan(c, wave_tot);
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t bits = lane_word(v[u], e);
                const uint32_t i = static_cast<uint32_t>(base + elem_off(u, e));
                const bool take = bits < end_bits || (bits == end_bits && i < end_idx);
                if (elem_off(u, e) < limit && take) {
                    if (pos < static_cast<uint32_t>(CAP)) cand[pos] = sort_key(bits, i);
                    ++pos;
                }
            }
        // total written so far: the last thread's end offset
        if (tid == kSelectThreads - 1) red_u[0][0] = pos;
        __syncthreads();
        written = red_u[0][0];
        __syncthreads();
        advance(v, nx);
    }
    const uint32_t n = written < static_cast<uint32_t>(CAP) ? written : static_cast<uint32_t>(CAP);
    uint32_t P = 1;
    while (P < n) P <<= 1;
    for (uint32_t i = n + tid; i < P; i += kSelectThreads) cand[i] = ~0ull;
    __syncthreads();

    // Bitonic sort of cand[0, P), ascending.
    for (uint32_t k = 2; k <= P; k <<= 1) {
        for (uint32_t jj = k >> 1; jj > 0; jj >>= 1) {
            for (uint32_t t = tid; t < P / 2; t += kSelectThreads) {
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

    int32_t *out_ids = a.ids + b * a.r;
    float *out_d = a.dists + b * a.r;
    for (int j = tid; j < a.r; j += kSelectThreads) {
        if (static_cast<uint32_t>(j) < r_eff && static_cast<uint32_t>(j) < n) {
            const uint64_t key = cand[j];
            out_ids[j] = static_cast<int32_t>(key & 0xffffffffu);
            out_d[j] = __uint_as_float(static_cast<uint32_t>(key >> 32));
        } else {  // only reachable when a key set is smaller than r (a false hint)
            out_ids[j] = -1;
            out_d[j] = __builtin_huge_valf();
        }
    }
    if (!MIX) return;

    // ---- mixture over the r neighbours now sorted in cand[0, r_eff)
    const uint32_t rn = r_eff < n ? r_eff : n;
    const float dmin = rn > 0 ? __uint_as_float(static_cast<uint32_t>(cand[0] >> 32)) : 0.0f;
    float wj[kPer];
    int32_t tok[kPer];
    float zpart = 0.0f;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const uint32_t j = static_cast<uint32_t>(q * kSelectThreads + tid);
        tok[q] = -1;
        wj[q] = 0.0f;
        if (j < rn) {
            const uint64_t key = cand[j];
            const int32_t id = static_cast<int32_t>(key & 0xffffffffu);
            const float dj = __uint_as_float(static_cast<uint32_t>(key >> 32));
            wj[q] = expf(-m.mu * (dj - dmin));
            zpart += wj[q];
            tok[q] = m.values[k0 + id];
        }
    }
    const float z = block_sum(zpart, red_f);
    mix_row(wj, tok, z, m, b, acc);
}

// Standalone mixture on caller-given neighbours (any order): one workgroup per query.
__global__ __launch_bounds__(kSelectThreads) void k_mix(MixArgs m) {
    __shared__ float acc[kVocabTile];
    __shared__ float red_f[kNumWaves];
    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int64_t s = set_of_query(m.query_offsets, m.S, b);
    const int64_t k0 = m.key_offsets[s];
    const int64_t N = m.key_offsets[s + 1] - k0;
    float dj[kPer];
    int32_t id[kPer];
    float dmin = __builtin_huge_valf();
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int j = q * kSelectThreads + tid;
        dj[q] = j < m.r ? m.dists[b * m.r + j] : __builtin_huge_valf();
        id[q] = j < m.r ? m.ids[b * m.r + j] : -1;
        dmin = fminf(dmin, dj[q]);
    }
    dmin = block_min(dmin, red_f);
    float wj[kPer];
    int32_t tok[kPer];
    float zpart = 0.0f;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int j = q * kSelectThreads + tid;
        wj[q] = j < m.r ? expf(-m.mu * (dj[q] - dmin)) : 0.0f;
        zpart += wj[q];
        tok[q] = (j < m.r && id[q] >= 0 && id[q] < N) ? m.values[k0 + id[q]] : -1;
    }
    const float z = block_sum(zpart, red_f);
    mix_row(wj, tok, z, m, b, acc);
}

template <int CAP, bool MIX>
hipError_t launch_cap(const SelectArgs &a, const MixArgs &m, dim3 grid, hipStream_t st) {
    hipLaunchKernelGGL((k_select<CAP, MIX>), grid, dim3(kSelectThreads), 0, st, a, m);
    return hipGetLastError();
}

template <bool MIX>
hipError_t launch_sel(const SelectArgs &a, const MixArgs &m, int64_t B, hipStream_t st) {
    if (B == 0) return hipSuccess;
    if (B > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(B));
    switch (select_capacity(a.r)) {
    case 2048: return launch_cap<2048, MIX>(a, m, grid, st);
    case 4096: return launch_cap<4096, MIX>(a, m, grid, st);
    case 8192: return launch_cap<8192, MIX>(a, m, grid, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

int select_capacity(int r) {
    int p = 1;
    while (p < r) p <<= 1;
    int cap = 2 * p;
    if (cap < 2048) cap = 2048;
    return cap;  // <= 8192 for r <= KNNLM_MAX_R
}

hipError_t launch_select(const SelectArgs &args, int64_t B, hipStream_t stream) {
    MixArgs none{};
    return launch_sel<false>(args, none, B, stream);
}

hipError_t launch_select_mix(const SelectArgs &args, const MixArgs &mix, int64_t B, hipStream_t stream) {
    return launch_sel<true>(args, mix, B, stream);
}

hipError_t launch_mix(const MixArgs &args, int64_t B, hipStream_t stream) {
    if (B == 0) return hipSuccess;
    if (B > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_mix, dim3(static_cast<unsigned>(B)), dim3(kSelectThreads), 0, stream, args);
    return hipGetLastError();
}

}  // namespace knnlm
