// Top-r stage: for every query, the r keys of its own set with the smallest
// squared distance (largest similarity s = -d, paper Section 2.2; the paper
// retrieves r = 1024, Appendix A), returned ascending by (distance, key index).
// The paper does not order equal distances; the lower key index wins here.
//
// One 1024-thread workgroup per query.  Every key i is given the 64-bit key
// (bits(d_i) << 32) | i: distances are >= +0, so their fp32 bit patterns order
// like the values, and the index makes all keys distinct.  A radix refinement
// narrows [lo, hi) -- the key range known to hold the r-th smallest key --
// with 2048-bin LDS histograms until every key below hi fits in LDS; those
// keys are then compacted, bitonic-sorted and the first r written out.  With
// the range initialised from the per-tile min/max the distance stage leaves,
// one histogram pass usually suffices.
#include "knnlm_device.h"
#include "knnlm_internal.h"

namespace knnlm {

namespace {

constexpr int kNumWaves = kSelectThreads / kWave;

__device__ __forceinline__ uint64_t sort_key(float d, int64_t i) {
    return (static_cast<uint64_t>(__float_as_uint(d)) << 32) | static_cast<uint32_t>(i);
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
    return before + incl - v;
}

template <int CAP>
__global__ __launch_bounds__(kSelectThreads) void k_select(SelectArgs a) {
    __shared__ uint32_t hist[kSelectBins];
    __shared__ uint64_t cand[CAP];
    __shared__ uint32_t red_u[2][kNumWaves];
    __shared__ uint32_t wave_tot[kNumWaves];
    __shared__ uint64_t sh_lo, sh_hi;
    __shared__ uint32_t sh_below, sh_cnt, sh_n, sh_found;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int64_t b = blockIdx.x;
    const int64_t s = set_of_query(a.query_offsets, a.S, b);
    int64_t N = a.key_offsets[s + 1] - a.key_offsets[s];
    if (N > a.ld) N = a.ld;
    const float *drow = a.dist + b * a.ld;
    int32_t *out_ids = a.ids + b * a.r;
    float *out_d = a.dists + b * a.r;
    const uint32_t r_eff = static_cast<uint32_t>(N < a.r ? N : a.r);

    // ---- range of the keys: from the per-tile extrema, or one pass.
    uint32_t bmin = 0xffffffffu, bmax = 0u;
    if (a.tile_min != nullptr) {
        const int64_t ntiles = (N + a.rows_per_tile - 1) / a.rows_per_tile;
        for (int64_t t = tid; t < ntiles; t += kSelectThreads) {
            bmin = min(bmin, __float_as_uint(a.tile_min[b * a.tiles_per_set + t]));
            bmax = max(bmax, __float_as_uint(a.tile_max[b * a.tiles_per_set + t]));
        }
    } else {
        for (int64_t i = tid; i < N; i += kSelectThreads) {
            const uint32_t u = __float_as_uint(drow[i]);
            bmin = min(bmin, u);
            bmax = max(bmax, u);
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
        uint32_t m = red_u[0][0], M = red_u[1][0];
        for (int w = 1; w < kNumWaves; ++w) {
            m = min(m, red_u[0][w]);
            M = max(M, red_u[1][w]);
        }
        if (N == 0) { m = 0u; M = 0u; }
        sh_lo = static_cast<uint64_t>(m) << 32;
        sh_hi = (static_cast<uint64_t>(M) << 32) + static_cast<uint64_t>(N);
        sh_below = 0u;
        sh_cnt = static_cast<uint32_t>(N);
    }
    __syncthreads();
    uint64_t lo = sh_lo, hi = sh_hi;
    uint32_t below = sh_below, cnt = sh_cnt;

    // ---- refinement: keep [lo, hi) holding the r-th smallest key.  Each pass
    // shrinks the 64-bit range by 2^10 at least, so 7 passes always suffice;
    // the cap and the found flag only guard against inconsistent inputs.
    for (int pass = 0; pass < 8 && below + cnt > static_cast<uint32_t>(CAP); ++pass) {
        const uint64_t w = hi - lo;  // >= 2 here
        const int nbits = 64 - __clzll(static_cast<long long>(w - 1));
        const int shift = nbits > kSelectBinsLog2 ? nbits - kSelectBinsLog2 : 0;
        for (int i = tid; i < kSelectBins; i += kSelectThreads) hist[i] = 0u;
        if (tid == 0) sh_found = 0u;
        __syncthreads();
        for (int64_t i = tid; i < N; i += kSelectThreads) {
            const uint64_t off = sort_key(drow[i], i) - lo;
            if (off < w) atomicAdd(&hist[off >> shift], 1u);
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
            const uint64_t nlo = lo + (static_cast<uint64_t>(j) << shift);
            const uint64_t nhi = nlo + (1ull << shift);
            sh_lo = nlo;
            sh_hi = nhi < hi ? nhi : hi;
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

    // ---- compaction of every key below hi (exactly below + cnt <= CAP of them).
    if (tid == 0) sh_n = 0u;
    __syncthreads();
    for (int64_t i = tid; i < N; i += kSelectThreads) {
        const uint64_t key = sort_key(drow[i], i);
        if (key < hi) {
            const uint32_t pos = atomicAdd(&sh_n, 1u);
            if (pos < static_cast<uint32_t>(CAP)) cand[pos] = key;
        }
    }
    __syncthreads();
    const uint32_t n = sh_n < static_cast<uint32_t>(CAP) ? sh_n : static_cast<uint32_t>(CAP);
    uint32_t P = 1;
    while (P < n) P <<= 1;
    for (uint32_t i = n + tid; i < P; i += kSelectThreads) cand[i] = ~0ull;
    __syncthreads();

    // ---- bitonic sort of cand[0, P), ascending.
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
    if (B == 0) return hipSuccess;
    if (B > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(B));
    switch (select_capacity(args.r)) {
    case 2048: hipLaunchKernelGGL((k_select<2048>), grid, dim3(kSelectThreads), 0, stream, args); break;
    case 4096: hipLaunchKernelGGL((k_select<4096>), grid, dim3(kSelectThreads), 0, stream, args); break;
    case 8192: hipLaunchKernelGGL((k_select<8192>), grid, dim3(kSelectThreads), 0, stream, args); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace knnlm
