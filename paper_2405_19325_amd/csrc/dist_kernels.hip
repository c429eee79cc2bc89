// Distance stage: d(q, k) = ||q||^2 - 2 q.k + ||k||^2 (fp32 accumulation), the
// squared L2 distance whose negative is the similarity s(q, k) of the paper
// (Section 2.2, sentence after eq. non-parametric; Appendix A).
//
// The work is HBM-bound for every batch size this kernel serves (one to eight
// queries per key set): each key row is read from HBM exactly once and dotted
// with every query of its set while it sits in registers.
//
// Numerics (shared by the on-the-fly norms here and knn_key_sqnorms): a row is
// cut into 32-bit words (two bf16/f16 elements or one fp32 element) and
// 16-byte chunks of four words; lane l of a wave accumulates chunks l, l+64,
// l+128, ... word by word into one fp32 accumulator (v_dot2_f32_bf16 /
// v_dot2_f32_f16 for 16-bit elements, FMA for fp32); the 64 lane partials are
// then summed by a fixed reduction tree that leaves the same bits in every lane.
// ||q||^2, ||k||^2 and q.k all use this order, so q == k gives exactly 0.
//
// Key masking (Section 3.4: the keys of an accepted span are not used again in
// that generation): a masked row's distance is written as +infinity and left
// out of the tile extrema, so no select path takes it while unmasked keys
// remain.  The streaming kernel loads a row's mask bit with the row's key
// loads, one pipeline stage ahead of its use.
#include "knnlm_device.h"
#include "knnlm_internal.h"

namespace knnlm {

namespace {

constexpr int kWavesPerDistBlock = kDistThreads / kWave;

// Where the streaming kernel stores the (discarded) distances of the sets it
// loads past its tile's end: one word per device, written, never read.
__device__ float g_dist_sink;
constexpr int kQueryRegChunks = 16;  // 16-byte query chunks a lane may hold in registers

// ---------------------------------------------------------------- vector path

// Per-set tile bounds shared by both distance kernels.  Returns false when the
// workgroup has no work (uniform over the block).
struct TileWork {
    int64_t k0, r0, r1, qb;
    int nq;
};

template <int NQ>
__device__ __forceinline__ bool tile_work(const DistArgs &a, TileWork &t) {
    const int64_t tiles = a.tiles_per_set;
    const int64_t s = blockIdx.x / tiles;
    const int64_t tile = blockIdx.x - s * tiles;
    t.k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - t.k0;
    if (N > a.ld) N = a.ld;
    t.qb = a.query_offsets[s] + static_cast<int64_t>(blockIdx.y) * NQ;
    const int64_t qe = a.query_offsets[s + 1];
    t.r0 = tile * a.rows_per_tile;
    if (t.qb >= qe || t.r0 >= N) return false;
    t.nq = static_cast<int>(qe - t.qb < NQ ? qe - t.qb : NQ);
    t.r1 = (t.r0 + a.rows_per_tile < N) ? t.r0 + a.rows_per_tile : N;
    return true;
}

// Block-wide min/max of each query's distances over this tile, for the select
// stage, and (group_min) each wave's minimum: the select's group minima, group
// 4 * tile + wave holding the rows r0 + wave, r0 + wave + 4, ... of the tile
// (+infinity where the wave has no row or only masked ones).
template <int NQ>
__device__ __forceinline__ void write_tile_extrema(const DistArgs &a, const TileWork &t, const float (&mn)[NQ],
                                                   const float (&mx)[NQ]) {
    static_assert(kWavesPerDistBlock == 4, "one 16-byte word of group minima per tile");
    constexpr int NW = kWavesPerDistBlock;
    __shared__ float smin[NW][NQ];
    __shared__ float smax[NW][NQ];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    if (lane == 0) {
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
            smin[wave][j] = mn[j];
            smax[wave][j] = mx[j];
        }
    }
    __syncthreads();
    if (static_cast<int>(threadIdx.x) < t.nq) {
        const int j = threadIdx.x;
        float m = smin[0][j], M = smax[0][j];
        for (int w = 1; w < NW; ++w) {
            m = fminf(m, smin[w][j]);
            M = fmaxf(M, smax[w][j]);
        }
        const int64_t tile = t.r0 / a.rows_per_tile;
        if (a.tile_min != nullptr) {
            a.tile_min[(t.qb + j) * a.tiles_per_set + tile] = m;
            a.tile_max[(t.qb + j) * a.tiles_per_set + tile] = M;
        }
        if (a.group_min != nullptr)
            *reinterpret_cast<float4 *>(a.group_min + (t.qb + j) * a.groups_per_set + 4 * tile) =
                make_float4(smin[0][j], smin[1][j], smin[2][j], smin[3][j]);
    }
}

// The select stage's counters, cleared by the launch's first workgroup (so
// that no memset is needed between the stages, and a captured graph holds none).
__device__ __forceinline__ void clear_select_words(const DistArgs &a) {
    if (a.zero_words == nullptr || blockIdx.x != 0 || blockIdx.y != 0) return;
    for (int64_t i = threadIdx.x; i < a.n_zero_words; i += blockDim.x) a.zero_words[i] = 0u;
}

// 16-byte loads: d % VEC == 0, 16-byte aligned rows, at most CPL chunks per lane.
// Queries stay packed in registers (NQ x CPL chunks per lane).  A wave takes
// the tile's rows wave, wave + 4, ... in sets of at most 8 chunks per lane
// (8 KiB per wave: a whole row, or half of a 16-chunk row) and keeps two rows
// in flight in register sets used in turn (the loop is unrolled over the sets,
// so no set is ever copied); a set is reloaded as soon as it is consumed.  A
// row's halves add into the same partial sums in chunk order, so the sums are
// those of a whole-row pass.  (Measured against deeper pipelines and
// whole-row sets: this keeps HBM busiest at 8 and 16 KiB rows.)
//
// The loop body has no branch: a branch around a load makes the compiler wait
// for every load in flight at the join, which would drain the pipeline once
// per set.  So every load is issued unconditionally --
//   * a set past the tile's end reads the group's first query row (in cache,
//     so the pipeline's tail costs no HBM traffic) and its distance goes to a
//     sink word, outside the tile's extrema;
//   * query slots past the group's last query repeat that query, so their
//     distances and stores repeat its own;
//   * ||k||^2 reads the given norms, or a valid dummy word that is ignored;
//   * every lane stores the (wave-uniform) distance to the same address.
// MASK: a.key_mask is given.
template <knn_dtype DT, int CPL, int NQ, bool MASK>
__global__ __launch_bounds__(kDistThreads) void k_dist_vec(DistArgs a) {
    constexpr int NW = kWavesPerDistBlock;
    constexpr int CPS = CPL > 8 ? 8 : CPL;  // chunks per set
    constexpr int SPR = CPL / CPS;          // sets per row
    constexpr int D = 2 * SPR;              // sets in flight: two rows
    constexpr int RPI = D / SPR;            // rows per loop iteration
    static_assert(CPL % CPS == 0 && D % SPR == 0, "whole sets per row, whole rows per iteration");
    constexpr int EB = Elem<DT>::BYTES;
    clear_select_words(a);
    TileWork t;
    if (!tile_work<NQ>(a, t)) return;

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int nchunks = static_cast<int>(a.d * EB / 16);
    const int64_t row_bytes = a.d * EB;
    const u32x4_t zero = {0u, 0u, 0u, 0u};

    u32x4_t qv[NQ][CPL];
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
        const int jj = j < t.nq ? j : t.nq - 1;
        const char *qrow = static_cast<const char *>(a.queries) + (t.qb + jj) * row_bytes;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const int ch = lane + kWave * c;
            const u32x4_t v = *reinterpret_cast<const u32x4_t *>(qrow + 16 * (ch < nchunks ? ch : 0));
            qv[j][c] = ch < nchunks ? v : zero;
        }
    }
    float mn[NQ], mx[NQ];
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
        mn[j] = __builtin_huge_valf();
        mx[j] = 0.0f;
    }
    const bool have_norms = a.key_sqnorms != nullptr;
    const float *knorm = have_norms ? a.key_sqnorms + t.k0 : a.dist;  // a.dist: a valid word, never used
    const char *kset = static_cast<const char *>(a.keys) + t.k0 * row_bytes;
    // the group's first query row: what the sets past the tile's end read (it is in cache)
    const char *qrow0 = static_cast<const char *>(a.queries) + t.qb * row_bytes;
    float *dq[NQ];  // this group's distance rows (repeated past the last query)
#pragma unroll
    for (int j = 0; j < NQ; ++j) dq[j] = a.dist + (t.qb + (j < t.nq ? j : t.nq - 1)) * a.ld;

    float qq[NQ];  // ||q||^2, computed once the first key loads are in flight
    u32x4_t kv[D][CPS];
    float kn[D];    // ||k||^2 of the set's row (sets that end a row)
    uint32_t mw[D], mb[D];  // its mask word and bit (MASK; sets that end a row)
    int64_t rc[D];  // the row each set holds (clamped into the tile)
    bool in[D];     // the set's row is in the tile
    float acc_k, acc_q[NQ];  // the current row's partial sums
    // set s holds part s % SPR of row rw
    auto load = [&](int s, int64_t rw) __attribute__((always_inline)) {
        const int part = s % SPR;
        const bool inside = rw < t.r1;
        const int64_t r = inside ? rw : t.r0;
        rc[s] = r;
        in[s] = inside;
        const char *krow = inside ? kset + r * row_bytes : qrow0;
#pragma unroll
        for (int c = 0; c < CPS; ++c) {
            const int ch = lane + kWave * (part * CPS + c);
            kv[s][c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(krow + 16 * (ch < nchunks ? ch : 0)));
        }
        if (part == SPR - 1) {  // with the row's last set: it is reloaded only after the row is done
            kn[s] = knorm[have_norms ? r : 0];
            if constexpr (MASK) {  // the word now, its bit where it is used (a test here would wait for the load)
                mw[s] = a.key_mask[(t.k0 + r) >> 5];
                mb[s] = static_cast<uint32_t>((t.k0 + r) & 31);
            }
        }
    };
    auto consume = [&](int s) __attribute__((always_inline)) {
        const int part = s % SPR;
        if (part == 0) {
            acc_k = 0.0f;
#pragma unroll
            for (int j = 0; j < NQ; ++j) acc_q[j] = 0.0f;
        }
#pragma unroll
        for (int c = 0; c < CPS; ++c) {
            const int cc = part * CPS + c;
            // chunks past the row read its first chunk: zeroed here, where the data is used
            // (a select at the load would wait for the load)
            const u32x4_t kc = lane + kWave * cc < nchunks ? kv[s][c] : zero;
            const uint4 k4 = make_uint4(kc.x, kc.y, kc.z, kc.w);
            acc_k = dot_chunk<DT>(k4, k4, acc_k);
#pragma unroll
            for (int j = 0; j < NQ; ++j)
                acc_q[j] = dot_chunk<DT>(make_uint4(qv[j][cc].x, qv[j][cc].y, qv[j][cc].z, qv[j][cc].w), k4, acc_q[j]);
        }
        if (part != SPR - 1) return;
        const float kk_sum = wave_allsum(acc_k);
        const float kk = have_norms ? kn[s] : kk_sum;
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
            const float dot = wave_allsum(acc_q[j]);
            float dist = clamp_nonneg(fmaf(-2.0f, dot, qq[j] + kk));
            bool counted = in[s];
            if constexpr (MASK) {
                const bool masked = ((mw[s] >> mb[s]) & 1u) != 0u;
                dist = masked ? __uint_as_float(kMaskedBits) : dist;
                counted = counted && !masked;
            }
            *(in[s] ? dq[j] + rc[s] : &g_dist_sink) = dist;
            mn[j] = counted ? fminf(mn[j], dist) : mn[j];
            mx[j] = counted ? fmaxf(mx[j], dist) : mx[j];
        }
    };

    int64_t row = t.r0 + wave;
#pragma unroll
    for (int s = 0; s < D; ++s) load(s, row + static_cast<int64_t>(s / SPR) * NW);
    // ||q||^2 after the first key loads are issued, so they overlap the query's latency.
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
        float acc = 0.0f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const uint4 q4 = make_uint4(qv[j][c].x, qv[j][c].y, qv[j][c].z, qv[j][c].w);
            acc = dot_chunk<DT>(q4, q4, acc);
        }
        qq[j] = wave_allsum(acc);
    }
    for (; row < t.r1; row += static_cast<int64_t>(RPI) * NW) {
#pragma unroll
        for (int s = 0; s < D; ++s) {
            // the scheduler may not mix the sets' work: mixing them needs every set's
            // data at once, that is a wait for every load in flight
            __builtin_amdgcn_sched_barrier(0);
            consume(s);
            load(s, row + static_cast<int64_t>(s / SPR + RPI) * NW);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (a.tile_min != nullptr || a.group_min != nullptr) write_tile_extrema<NQ>(a, t, mn, mx);
}

// --------------------------------------------------- element path (any d)

// Same word/chunk layout and accumulation order as the vector path, with
// element loads (elements past d read as 0): serves d that is not a multiple
// of VEC, rows that are not 16-byte aligned and d above the vector path's
// register budget.
template <knn_dtype DT, int NQ>
__global__ __launch_bounds__(kDistThreads) void k_dist_elem(DistArgs a) {
    constexpr int EB = Elem<DT>::BYTES;
    constexpr int PW = Elem<DT>::PER_WORD;
    constexpr int NW = kWavesPerDistBlock;
    clear_select_words(a);
    TileWork t;
    if (!tile_work<NQ>(a, t)) return;

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t d = a.d;
    const int64_t nwords = (d + PW - 1) / PW;
    const int64_t nchunks = (nwords + 3) / 4;
    const int64_t cpl = (nchunks + kWave - 1) / kWave;
    const char *qbase = static_cast<const char *>(a.queries) + t.qb * d * EB;

    float qq[NQ];
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
        float acc = 0.0f;
        if (j < t.nq) {
            const void *qrow = qbase + j * d * EB;
            for (int64_t c = 0; c < cpl; ++c) {
                const int64_t w0 = (lane + kWave * c) * 4;
                for (int u = 0; u < 4; ++u) {
                    const uint32_t w = load_word<DT>(qrow, w0 + u, d);
                    acc = dot_word<DT>(w, w, acc);
                }
            }
        }
        qq[j] = wave_allsum(acc);
    }

    float mn[NQ], mx[NQ];
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
        mn[j] = __builtin_huge_valf();
        mx[j] = 0.0f;
    }
    const bool have_norms = a.key_sqnorms != nullptr;
    const char *kset = static_cast<const char *>(a.keys) + t.k0 * d * EB;

    for (int64_t rw = t.r0 + wave; rw < t.r1; rw += NW) {
        const void *krow = kset + rw * d * EB;
        float acc_k = 0.0f;
        float acc_q[NQ];
#pragma unroll
        for (int j = 0; j < NQ; ++j) acc_q[j] = 0.0f;
        for (int64_t c = 0; c < cpl; ++c) {
            const int64_t w0 = (lane + kWave * c) * 4;
            for (int u = 0; u < 4; ++u) {
                const uint32_t kw = load_word<DT>(krow, w0 + u, d);
                if (!have_norms) acc_k = dot_word<DT>(kw, kw, acc_k);
#pragma unroll
                for (int j = 0; j < NQ; ++j) {
                    const uint32_t qw = (j < t.nq) ? load_word<DT>(qbase + j * d * EB, w0 + u, d) : 0u;
                    acc_q[j] = dot_word<DT>(qw, kw, acc_q[j]);
                }
            }
        }
        const float kk = have_norms ? a.key_sqnorms[t.k0 + rw] : wave_allsum(acc_k);
        const bool masked = a.key_mask != nullptr && key_masked(a.key_mask, t.k0 + rw);
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
            const float dot = wave_allsum(acc_q[j]);
            const float dist = masked ? __uint_as_float(kMaskedBits) : clamp_nonneg(fmaf(-2.0f, dot, qq[j] + kk));
            if (lane == j && j < t.nq) a.dist[(t.qb + j) * a.ld + rw] = dist;
            if (!masked) {
                mn[j] = fminf(mn[j], dist);
                mx[j] = fmaxf(mx[j], dist);
            }
        }
    }
    if (a.tile_min != nullptr || a.group_min != nullptr) write_tile_extrema<NQ>(a, t, mn, mx);
}

// ------------------------------------------------------------ key norms

// ||k||^2 per row: the wave-per-row layout and word order of the distance
// kernel (so the values equal its on-the-fly norms bit for bit), over a fixed
// grid, two rows in flight per wave in register sets used in turn (half-row
// sets for 16-chunk rows), every load unconditional (rows past the end read
// row 0).  With BLOCKED (rows of at most 4 KB, enough of them to give every
// wave of the grid a block) the waves take blocks of 64 consecutive rows:
// lane i keeps the norm of the block's row i, and the block's 64 norms leave
// in one 256-byte store (a store per row, 63 lanes of it idle, held such rows
// near 70% of 8 TB/s).  Otherwise the rows stride over the waves one at a
// time, each norm stored as it is made.
template <knn_dtype DT, int CPL, bool BLOCKED>
__global__ __launch_bounds__(kDistThreads) void k_sqnorm_vec(const void *keys, int64_t n, int64_t d, float *out) {
    constexpr int EB = Elem<DT>::BYTES;
    constexpr int CPS = CPL > 8 ? 8 : CPL;  // chunks per set
    constexpr int SPR = CPL / CPS;          // sets per row
    constexpr int D = 2 * SPR;              // sets in flight: two rows
    static_assert(!BLOCKED || CPL <= 4, "blocks of short rows");
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wave_global = (static_cast<int64_t>(blockIdx.x) * kDistThreads + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (kDistThreads / kWave);
    const int nchunks = static_cast<int>(d * EB / 16);
    const int64_t row_bytes = d * EB;
    const char *base = static_cast<const char *>(keys);
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    u32x4_t kv[D][CPS];
    float acc = 0.0f;
    auto load = [&](int s, int64_t rw) __attribute__((always_inline)) {
        const int part = s % SPR;
        const char *krow = base + (rw < n ? rw : 0) * row_bytes;
#pragma unroll
        for (int c = 0; c < CPS; ++c) {
            const int ch = lane + kWave * (part * CPS + c);
            kv[s][c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(krow + 16 * (ch < nchunks ? ch : 0)));
        }
    };
    auto consume = [&](int s) __attribute__((always_inline)) {
        const int part = s % SPR;
        if (part == 0) acc = 0.0f;
#pragma unroll
        for (int c = 0; c < CPS; ++c) {
            const u32x4_t kc = lane + kWave * (part * CPS + c) < nchunks ? kv[s][c] : zero;
            const uint4 k4 = make_uint4(kc.x, kc.y, kc.z, kc.w);
            acc = dot_chunk<DT>(k4, k4, acc);
        }
    };
    if constexpr (BLOCKED) {
        // row i of this wave's block blk (i in [0, 64)); the two rows after
        // it follow in the block or start the wave's next block
        const int64_t nblk = (n + kWave - 1) / kWave;
        int64_t blk = wave_global;
        auto row_at = [&](int64_t bk, int i) __attribute__((always_inline)) {
            return i < kWave ? bk * kWave + i : (bk + nwaves) * kWave + (i - kWave);
        };
#pragma unroll
        for (int s = 0; s < D; ++s) load(s, row_at(blk, s / SPR));
        float mine = 0.0f;  // lane i: the norm of row i of the block
        for (; blk < nblk; blk += nwaves) {
            for (int i = 0; i < kWave; i += 2) {
#pragma unroll
                for (int s = 0; s < D; ++s) {
                    __builtin_amdgcn_sched_barrier(0);  // keep the sets' work apart (see the distance kernel)
                    consume(s);
                    if (s % SPR == SPR - 1) {
                        const float v = wave_allsum(acc);
                        mine = lane == i + s / SPR ? v : mine;
                    }
                    load(s, row_at(blk, i + s / SPR + 2));
                }
            }
            const int64_t r = blk * kWave + lane;
            *(r < n ? out + r : &g_dist_sink) = mine;
        }
    } else {
        int64_t row = wave_global;
#pragma unroll
        for (int s = 0; s < D; ++s) load(s, row + static_cast<int64_t>(s / SPR) * nwaves);
        for (; row < n; row += 2 * nwaves) {
#pragma unroll
            for (int s = 0; s < D; ++s) {
                __builtin_amdgcn_sched_barrier(0);  // keep the sets' work apart (see the distance kernel)
                consume(s);
                if (s % SPR == SPR - 1) {
                    const float v = wave_allsum(acc);
                    const int64_t rw = row + static_cast<int64_t>(s / SPR) * nwaves;
                    *(rw < n ? out + rw : &g_dist_sink) = v;
                }
                load(s, row + static_cast<int64_t>(s / SPR + 2) * nwaves);
            }
        }
    }
    __builtin_amdgcn_sched_barrier(0);
}

template <knn_dtype DT>
__global__ __launch_bounds__(kDistThreads) void k_sqnorm_elem(const void *keys, int64_t n, int64_t d, float *out) {
    constexpr int EB = Elem<DT>::BYTES;
    constexpr int PW = Elem<DT>::PER_WORD;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wave_global = (static_cast<int64_t>(blockIdx.x) * kDistThreads + threadIdx.x) / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (kDistThreads / kWave);
    const int64_t nwords = (d + PW - 1) / PW;
    const int64_t nchunks = (nwords + 3) / 4;
    const int64_t cpl = (nchunks + kWave - 1) / kWave;
    for (int64_t row = wave_global; row < n; row += nwaves) {
        const void *krow = static_cast<const char *>(keys) + row * d * EB;
        float acc = 0.0f;
        for (int64_t c = 0; c < cpl; ++c) {
            const int64_t w0 = (lane + kWave * c) * 4;
            for (int u = 0; u < 4; ++u) {
                const uint32_t w = load_word<DT>(krow, w0 + u, d);
                acc = dot_word<DT>(w, w, acc);
            }
        }
        acc = wave_allsum(acc);
        if (lane == 0) out[row] = acc;
    }
}

// ------------------------------------------------------------ dispatch

template <knn_dtype DT, int CPL, int NQ>
hipError_t launch_vec(const DistArgs &a, dim3 grid, hipStream_t st) {
    if constexpr (NQ * CPL <= kQueryRegChunks && CPL <= kMaxCplVec) {
        if (a.key_mask != nullptr)
            hipLaunchKernelGGL((k_dist_vec<DT, CPL, NQ, true>), grid, dim3(kDistThreads), 0, st, a);
        else
            hipLaunchKernelGGL((k_dist_vec<DT, CPL, NQ, false>), grid, dim3(kDistThreads), 0, st, a);
        return hipGetLastError();
    } else {
        return hipErrorInvalidValue;
    }
}

template <knn_dtype DT, int CPL>
hipError_t launch_vec_nq(int nq, const DistArgs &a, dim3 grid, hipStream_t st) {
    switch (nq) {
    case 1: return launch_vec<DT, CPL, 1>(a, grid, st);
    case 2: return launch_vec<DT, CPL, 2>(a, grid, st);
    case 4: return launch_vec<DT, CPL, 4>(a, grid, st);
    case 8: return launch_vec<DT, CPL, 8>(a, grid, st);
    default: return hipErrorInvalidValue;
    }
}

template <knn_dtype DT>
hipError_t launch_dist_dt(const DistPlan &p, const DistArgs &a, dim3 grid, hipStream_t st) {
    if (!p.vec) {
        switch (p.nq) {
        case 1: hipLaunchKernelGGL((k_dist_elem<DT, 1>), grid, dim3(kDistThreads), 0, st, a); break;
        case 2: hipLaunchKernelGGL((k_dist_elem<DT, 2>), grid, dim3(kDistThreads), 0, st, a); break;
        case 4: hipLaunchKernelGGL((k_dist_elem<DT, 4>), grid, dim3(kDistThreads), 0, st, a); break;
        case 8: hipLaunchKernelGGL((k_dist_elem<DT, 8>), grid, dim3(kDistThreads), 0, st, a); break;
        default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    switch (p.cpl) {
    case 1: return launch_vec_nq<DT, 1>(p.nq, a, grid, st);
    case 2: return launch_vec_nq<DT, 2>(p.nq, a, grid, st);
    case 4: return launch_vec_nq<DT, 4>(p.nq, a, grid, st);
    case 8: return launch_vec_nq<DT, 8>(p.nq, a, grid, st);
    case 16: return launch_vec_nq<DT, 16>(p.nq, a, grid, st);
    default: return hipErrorInvalidValue;
    }
}

int pow2_at_least(int64_t x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

bool vector_path_ok(int64_t d, knn_dtype dtype, const void *queries, const void *keys) {
    const int vec = vec_elems(dtype);
    if (d % vec != 0) return false;
    if ((d / vec + kWave - 1) / kWave > kMaxCplVec) return false;
    if ((reinterpret_cast<uintptr_t>(queries) & 15u) || (reinterpret_cast<uintptr_t>(keys) & 15u)) return false;
    return true;
}

}  // namespace

bool mfma_shape(int64_t d, knn_dtype dtype, int64_t max_queries) {
    return (dtype == KNN_BF16 || dtype == KNN_F16) && d % kMfmaSpan == 0 && d <= kMfmaMaxD &&
           max_queries >= kMfmaMinQueries;
}

// Key rows per distance workgroup.  Streaming path: about 1 MiB of keys,
// fewer (down to 16 rows) when the launch would otherwise have under 2048
// workgroups: with more workgroups than fit at once, each XCD's dispatcher
// hands the later ones to the CUs that finish first, which evens out the
// tail (measured at 64Ki x 4096 bf16: 77 us at 2048 workgroups against
// 80.5 us at 512).  Matrix-core path: whole passes, enough of them for a deep
// pipeline.  A multiple of 8 rows.
// Depends on sizes only, so the workspace size does not depend on pointers.
int dist_tile_rows(int64_t d, knn_dtype dtype, int64_t S, int64_t max_keys, int64_t max_queries) {
    if (mfma_shape(d, dtype, max_queries)) return mfma_tile_rows(d);
    const int64_t step = 8;
    const int64_t row_bytes = d * elem_bytes(dtype);
    int64_t rpt = (1024 * 1024) / (row_bytes > 0 ? row_bytes : 1);
    if (rpt > 4096) rpt = 4096;
    rpt = (rpt + step - 1) / step * step;
    if (rpt < step) rpt = step;
    while (rpt > 2 * step && S * ((max_keys + rpt - 1) / rpt) < 2048) rpt = (rpt / 2 + step - 1) / step * step;
    return static_cast<int>(rpt);
}

DistPlan plan_distances(int64_t d, knn_dtype dtype, int64_t max_queries, const void *queries,
                        const void *keys) {
    DistPlan p{};
    const int vec = vec_elems(dtype);
    p.vec = vector_path_ok(d, dtype, queries, keys);
    const int64_t mq = max_queries < 1 ? 1 : max_queries;
    p.mfma = p.vec && mfma_shape(d, dtype, max_queries);
    if (p.mfma) {
        const int64_t per = mq < 128 ? mq : 128;
        int blocks = 1;
        while (blocks * 16 < per) blocks <<= 1;
        p.mq = blocks;
        p.cpl = 0;
        p.nq = blocks * 16;
        p.groups = (mq + p.nq - 1) / p.nq;
        return p;
    }
    if (p.vec) {
        p.cpl = pow2_at_least((d / vec + kWave - 1) / kWave);
        int nq = 8;
        while (nq > 1 && (nq * p.cpl > kQueryRegChunks || nq / 2 >= mq)) nq >>= 1;
        p.nq = nq;
    } else {
        p.cpl = 0;
        int nq = 8;
        while (nq > 1 && nq / 2 >= mq) nq >>= 1;
        p.nq = nq;
    }
    p.rows_per_tile = 0;  // set by the caller from the workspace layout
    p.tiles_per_set = 0;
    const int64_t groups = (mq + p.nq - 1) / p.nq;
    p.groups = groups;
    return p;
}

hipError_t launch_distances(const DistPlan &plan, knn_dtype dtype, const DistArgs &args, int64_t S,
                            hipStream_t stream) {
    if (plan.mfma && plan.packed) return launch_distances_packed(plan.mq, dtype, args, S, plan.groups, stream);
    if (plan.mfma) return launch_distances_mfma(plan.mq, dtype, args, S, plan.groups, stream);
    if (plan.packed) return hipErrorInvalidValue;  // packed keys are read by the matrix-core kernels only
    const int64_t nblocks = S * plan.tiles_per_set;
    if (nblocks > 0x7fffffffLL || plan.groups > 65535) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(nblocks), static_cast<unsigned>(plan.groups));
    switch (dtype) {
    case KNN_F32: return launch_dist_dt<KNN_F32>(plan, args, grid, stream);
    case KNN_BF16: return launch_dist_dt<KNN_BF16>(plan, args, grid, stream);
    case KNN_F16: return launch_dist_dt<KNN_F16>(plan, args, grid, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_key_sqnorms(const void *keys, int64_t n, int64_t d, knn_dtype dtype, float *out,
                              hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const bool vec = vector_path_ok(d, dtype, keys, keys);
    const int cpl = vec ? pow2_at_least((d / vec_elems(dtype) + kWave - 1) / kWave) : 0;
    // the vector kernel: enough rows per wave for its pipeline (at most 1024 workgroups, four per CU)
    const int64_t max_blocks = vec ? 1024 : 65536;
    // blocks of 64 short rows where they fill every wave of that grid
    const bool blocked = vec && cpl <= 4 && n >= kWave * kWavesPerDistBlock * max_blocks;
    const int64_t waves_needed = blocked ? (n + kWave - 1) / kWave : n;  // a wave per block, or per row
    int64_t blocks = (waves_needed + kWavesPerDistBlock - 1) / kWavesPerDistBlock;
    if (blocks > max_blocks) blocks = max_blocks;
    const dim3 grid(static_cast<unsigned>(blocks));
#define KNN_SQN(DT)                                                                                 \
    do {                                                                                            \
        if (!vec) {                                                                                 \
            hipLaunchKernelGGL((k_sqnorm_elem<DT>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); \
        } else {                                                                                    \
            switch (cpl * 2 + (blocked ? 1 : 0)) {                                                  \
            case 2: hipLaunchKernelGGL((k_sqnorm_vec<DT, 1, false>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); break; \
            case 3: hipLaunchKernelGGL((k_sqnorm_vec<DT, 1, true>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); break; \
            case 4: hipLaunchKernelGGL((k_sqnorm_vec<DT, 2, false>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); break; \
            case 5: hipLaunchKernelGGL((k_sqnorm_vec<DT, 2, true>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); break; \
            case 8: hipLaunchKernelGGL((k_sqnorm_vec<DT, 4, false>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); break; \
            case 9: hipLaunchKernelGGL((k_sqnorm_vec<DT, 4, true>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); break; \
            case 16: hipLaunchKernelGGL((k_sqnorm_vec<DT, 8, false>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); break; \
            case 32: hipLaunchKernelGGL((k_sqnorm_vec<DT, 16, false>), grid, dim3(kDistThreads), 0, stream, keys, n, d, out); break; \
            default: return hipErrorInvalidValue;                                                   \
            }                                                                                       \
        }                                                                                           \
    } while (0)
    switch (dtype) {
    case KNN_F32: KNN_SQN(KNN_F32); break;
    case KNN_BF16: KNN_SQN(KNN_BF16); break;
    case KNN_F16: KNN_SQN(KNN_F16); break;
    default: return hipErrorInvalidValue;
    }
#undef KNN_SQN
    return hipGetLastError();
}

}  // namespace knnlm
