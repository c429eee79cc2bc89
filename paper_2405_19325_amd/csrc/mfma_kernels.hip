// Distance stage for query batches: d(q, k) = ||q||^2 - 2 q.k + ||k||^2, the
// squared L2 distance whose negative is the paper's similarity (Section 2.2),
// with the q.k term on the gfx950 matrix cores.
//
// When many queries share one key set (speculative verification scores every
// draft position of a sequence against that sequence's store), the dot
// products form a dense [queries x d] . [d x keys] contraction: every key
// element is used by up to 128 queries, so streaming the keys from HBM once
// needs up to 128 flop per byte -- beyond the vector ALUs, within the
// matrix cores.  A workgroup of 4 waves takes passes of 128 keys of one set
// (two blocks of 16 per wave) against up to 128 of the set's queries (MQ
// blocks of 16), walking d in spans of 128 elements (256 bytes of a row).
//
// Each span of the pass's keys and queries goes HBM -> registers -> LDS -> the
// matrix cores.  The global loads are coalesced: 16 lanes read one row's
// 256-byte span, a wave instruction four whole rows.  The LDS copy is
// swizzled -- chunk c (16 bytes) of row n sits at slot n * 16 + (c ^ (n % 16))
// -- so that both the row-wise writes and the fragment reads (lane l reads
// row l % 16, chunk 4 * step + l / 16) touch every bank once.  In MFMA step c
// lane l holds key (or query) row l % 16 and elements 32c + 8 (l / 16) .. +8
// of the span -- the same elements for both operands, so the contraction is
// exact up to fp32 rounding -- for v_mfma_f32_16x16x32 (bf16 or f16, fp32
// accumulate).  Two LDS buffers alternate: while the matrix cores work on
// span t, span t + 1 is written to the other buffer, and the next NS spans
// load into NS register sets (NS = 2 to 4, as many as the shape's registers
// allow at two waves per SIMD).  The loads are never guarded by a
// branch, since a branch around loads makes the compiler wait for every load
// in flight: rows past the data read the tile's first row, and steps past the
// tile's end re-read its last span (from L2).
#include "knnlm_internal.h"
#include "mfma_device.h"

namespace knnlm {

namespace {

constexpr int kTileQuantum = 256;  // tile rows are multiples of the largest pass (256 keys)

// Where the epilogue stores the (discarded) distances of rows past the tile or
// query slots past the group: one word per device, written, never read.
__device__ float g_mfma_sink;

constexpr int kSpan = kMfmaSpan;  // d is a multiple of this (the largest span)

// MQ: 16-query blocks per workgroup; WK x WQ waves: WK groups split the
// pass's PK / 16 key blocks, WQ groups split the query blocks (MQ / WQ each);
// NS: register sets of prefetched spans (NS spans in flight); NORMS: ||k||^2
// comes precomputed; PK keys per pass and SPAN elements of d per pipeline
// step.  A wide query block re-stages its span in LDS once per pass, so
// 128-query workgroups take 256-key passes of 64-element spans (the same
// matrix-core work per step as 128 keys x 128 elements, with a quarter less
// loaded and written to LDS per step, a third less read from it).
//
// FM (the fused select of query batches on long rows): 0 every tile, the
// distances written; 1 only the sample pieces (the first sample_rows rows of
// every sample_every-th tile), the distances written; 2 every row outside the
// sample pieces, and instead of the distances each query's candidates -- keys
// whose distance bits are below the query's threshold -- are staged in LDS
// and appended to the query's list once the tile is done (the list's count is
// true even past its capacity; a full LDS stage sets the fallback word).
template <knn_dtype DT, int MQ, int WK, int WQ, int NS, bool NORMS, int PK, int SPAN, int FM = 0>
__global__ __launch_bounds__(WK * WQ * kWave, 1) void k_dist_mfma(DistArgs a, int64_t n_tiles, int64_t groups) {
    constexpr int QW = WQ;
    constexpr int kChunks = SPAN * 2 / 16;               // 16-byte chunks per row and span
    constexpr int KSTEPS = SPAN / 32;                    // MFMA steps per span
    constexpr int KBW = PK / 16 / WK;                    // key blocks per wave
    constexpr int kThreads = WK * WQ * kWave;
    constexpr int QB = MQ * 16;
    constexpr int MQW = MQ / QW;                         // query blocks per wave
    constexpr int KCH = PK * kChunks / kThreads;         // key chunks per thread and step
    constexpr int QCH = QB * kChunks / kThreads;         // query chunks per thread and step
    static_assert(MQ % QW == 0 && (PK / 16) % WK == 0 && KCH >= 1 && QCH >= 1, "whole blocks and chunks");
    static_assert(SPAN % 32 == 0 && kSpan % SPAN == 0 && kChunks <= 16, "whole MFMA steps, spans dividing d");
    // native 4 x u32 vectors throughout, so that every 16-byte LDS access is
    // one ds_read_b128 / ds_write_b128 (a struct is split by the compiler)
    __shared__ __align__(16) u32x4_t klds[2][PK * kChunks];
    __shared__ __align__(16) u32x4_t qlds[2][QB * kChunks];
    __shared__ uint32_t smin[QB], smax[QB];
    constexpr int kStage = FM == 2 ? 1024 : 1;  // candidates staged per tile (about 120 at 128 x 4096 keys)
    __shared__ uint64_t stage_key[kStage];
    __shared__ uint8_t stage_q[kStage];
    __shared__ uint32_t stage_n;
    static_assert(FM != 2 || QB <= 256, "a staged query fits a byte");

    if constexpr (FM == 0) {
        if (a.gate != nullptr && *a.gate != a.gate_run) return;
    }
    // Consecutive workgroups land on different XCDs (round robin over 8).  The
    // query groups of one key tile are numbered 8 apart, so they run on one XCD
    // at about the same time and all but the first read the tile from its L2.
    const int64_t L = blockIdx.x;
    const int64_t grp = (L >> 3) % groups;
    const int64_t tl = ((L >> 3) / groups) * 8 + (L & 7);
    if (tl >= n_tiles) return;
    const int64_t tiles = a.tiles_per_set;
    const int64_t se = FM == 0 ? 1 : a.sample_every;
    const int64_t per_set = FM == 1 ? (tiles + se - 1) / se : tiles;  // tiles (sample pieces) per set
    const int64_t s = tl / per_set;
    const int64_t tile = FM == 1 ? (tl - s * per_set) * se : tl - s * per_set;
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    const int64_t qb = a.query_offsets[s] + grp * QB;
    const int64_t qe = a.query_offsets[s + 1];
    // this workgroup's rows [r0, r1): the tile, its sample piece (FM 1), or the tile past its piece (FM 2)
    int64_t r0 = tile * a.rows_per_tile;
    const int64_t rend = r0 + (FM == 1 ? a.sample_rows : a.rows_per_tile);
    if (FM == 2 && tile % se == 0) r0 += a.sample_rows;
    if (qb >= qe || r0 >= N) return;  // uniform over the block
    const int nq = static_cast<int>(qe - qb < QB ? qe - qb : QB);
    const int64_t r1 = rend < N ? rend : N;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = (tid / kWave) / QW;  // this wave's group of key blocks
    const int jq = ((tid / kWave) % QW) * MQW;  // its first query block
    const int g = lane >> 4, lr = lane & 15;
    const int64_t row_bytes = a.d * 2;
    const int64_t nspan = a.d / SPAN;
    const int64_t npass = (r1 - r0 + PK - 1) / PK;
    const int64_t T = npass * nspan;  // pipeline steps of this tile
    const char *qbase = static_cast<const char *>(a.queries) + qb * row_bytes;
    const char *kset = static_cast<const char *>(a.keys) + k0 * row_bytes;

    for (int q = tid; q < QB; q += kThreads) {
        smin[q] = 0xffffffffu;
        smax[q] = 0u;
    }
    if (FM == 2 && tid == 0) stage_n = 0u;
    // FM 2: the thresholds of this lane's query rows (jq + j) * 16 + lr (0 past the group: nothing passes)
    uint32_t thr_l[MQW];
#pragma unroll
    for (int j = 0; j < MQW; ++j) {
        const int q = (jq + j) * 16 + lr;
        thr_l[j] = (FM == 2 && q < nq) ? a.cand_thr[qb + q] : 0u;
    }

    // Loads: chunk i of this thread is row i * R + tid / kChunks of the pass
    // (keys) or of the query block, 16-byte column tid % kChunks of the span
    // (R = kThreads / kChunks rows per chunk index, a multiple of 16, so its
    // LDS slot swz(i * R + rsub, col) is i * R * kChunks + slot0).
    const int col = tid & (kChunks - 1);
    const int rsub = tid / kChunks;
    const int slot0 = swz<kChunks>(rsub, col);
    constexpr int kRowsPerChunk = kThreads / kChunks;
    static_assert(kRowsPerChunk % 16 == 0, "the swizzle repeats every 16 rows");

    // Addresses: a uniform base per step plus a 32-bit offset per chunk (a
    // tile is at most 4096 rows of at most 128 KiB).
    // NS register sets take the steps in turn, so that NS steps are in flight
    // while the matrix cores work on another.
    u32x4_t kr[NS][KCH], qr_[NS][QCH];
    const char *ktile = kset + r0 * row_bytes;
    const uint32_t nrows = static_cast<uint32_t>(r1 - r0);
    const uint32_t rb = static_cast<uint32_t>(row_bytes);
    uint32_t qoff[QCH];
#pragma unroll
    for (int i = 0; i < QCH; ++i) {
        const int qrow = i * kRowsPerChunk + rsub;
        qoff[i] = static_cast<uint32_t>(qrow < nq ? qrow : 0) * rb + static_cast<uint32_t>(col * 16);
    }
    const uint32_t ns = static_cast<uint32_t>(nspan);  // steps fit 32 bits: at most 32 passes of 512 spans
    auto load = [&](int set, int64_t t) __attribute__((always_inline)) {
        const uint32_t p = static_cast<uint32_t>(t) / ns, sp = static_cast<uint32_t>(t) - p * ns;
        const char *kspan = ktile + static_cast<int64_t>(sp) * (2 * SPAN);
        const char *qspan = qbase + static_cast<int64_t>(sp) * (2 * SPAN);
        const uint32_t prow = p * PK + static_cast<uint32_t>(rsub);
#pragma unroll
        for (int i = 0; i < KCH; ++i) {
            const uint32_t rr = prow + static_cast<uint32_t>(i * kRowsPerChunk);
            const uint32_t off = (rr < nrows ? rr : 0u) * rb + static_cast<uint32_t>(col * 16);
            kr[set][i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(kspan + off));
        }
#pragma unroll
        for (int i = 0; i < QCH; ++i) qr_[set][i] = *reinterpret_cast<const u32x4_t *>(qspan + qoff[i]);
    };
    auto write = [&](int set, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < KCH; ++i) klds[buf][i * kRowsPerChunk * kChunks + slot0] = kr[set][i];
#pragma unroll
        for (int i = 0; i < QCH; ++i) qlds[buf][i * kRowsPerChunk * kChunks + slot0] = qr_[set][i];
    };

    f32x4_t acc[MQW][KBW];
    float kkp[KBW], qqp[MQW];
#pragma unroll
    for (int j = 0; j < MQW; ++j) qqp[j] = 0.0f;  // ||q||^2 partials: the first pass adds them up, later passes reuse them
    auto clear = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < MQW; ++j)
#pragma unroll
            for (int kb = 0; kb < KBW; ++kb) acc[j][kb] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) kkp[kb] = 0.0f;
    };
    clear();

    // The matrix cores over one span in LDS buffer buf (with qn_pass, also
    // the query norms); the span's MFMA steps unrolled, so that the next
    // step's fragment reads overlap this step's MFMAs.
    auto compute = [&](int buf, bool qn_pass) __attribute__((always_inline)) {
#pragma unroll
        for (int c = 0; c < KSTEPS; ++c) {
            const int ch = (4 * c + g) ^ (lr & (kChunks - 1));
            u32x4_t bk[KBW], af[MQW];
#pragma unroll
            for (int kb = 0; kb < KBW; ++kb) bk[kb] = klds[buf][((wave * KBW + kb) * 16 + lr) * kChunks + ch];
#pragma unroll
            for (int j = 0; j < MQW; ++j) af[j] = qlds[buf][((jq + j) * 16 + lr) * kChunks + ch];
#pragma unroll
            for (int j = 0; j < MQW; ++j)
#pragma unroll
                for (int kb = 0; kb < KBW; ++kb) acc[j][kb] = mfma16<DT>(af[j], bk[kb], acc[j][kb]);
            if constexpr (!NORMS) {
#pragma unroll
                for (int kb = 0; kb < KBW; ++kb) kkp[kb] = dot_vec<DT>(bk[kb], kkp[kb]);
            }
            if (qn_pass) {
#pragma unroll
                for (int j = 0; j < MQW; ++j) qqp[j] = dot_vec<DT>(af[j], qqp[j]);
            }
        }
    };

    // Distances of pass p: lane (g, lr) holds dot(query (jq + j)*16 + 4g + i,
    // key c0 + (wave*KBW + kb)*16 + lr) in acc[j][kb][i].
    auto epilogue = [&](int64_t p) __attribute__((always_inline)) {
        const int64_t c0 = r0 + p * PK;
        float kk[KBW];
        bool mk[KBW];  // masked key rows (Section 3.4): distance +infinity, no part in the extrema
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
            const int64_t row = c0 + (wave * KBW + kb) * 16 + lr;
            kk[kb] = NORMS ? (row < r1 ? a.key_sqnorms[k0 + row] : 0.0f) : group4_sum(kkp[kb]);
            mk[kb] = a.key_mask != nullptr && row < r1 && key_masked(a.key_mask, k0 + row);
        }
        if constexpr (FM == 2) {
            // candidates: distance bits below the query's threshold, appended to
            // the LDS stage a wave at a time (one LDS atomic per wave that has any)
#pragma unroll
            for (int j = 0; j < MQW; ++j) {
                const float qsum = group4_sum(qqp[j]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int q = (jq + j) * 16 + g * 4 + i;
                    const float qn = __shfl(qsum, g * 4 + i);
                    const uint32_t th = __shfl(thr_l[j], g * 4 + i);
#pragma unroll
                    for (int kb = 0; kb < KBW; ++kb) {
                        const int64_t row = c0 + (wave * KBW + kb) * 16 + lr;
                        const float dist = mk[kb] ? __uint_as_float(kMaskedBits)
                                                  : clamp_nonneg(fmaf(-2.0f, acc[j][kb][i], qn + kk[kb]));
                        const bool c = q < nq && row < r1 && __float_as_uint(dist) < th;
                        const uint64_t bal = __ballot(c);
                        if (bal != 0ull) {
                            const int first = __ffsll(static_cast<unsigned long long>(bal)) - 1;
                            uint32_t base = 0u;
                            if (lane == first) base = atomicAdd(&stage_n, static_cast<uint32_t>(__popcll(bal)));
                            base = readlane_u32(base, first);
                            if (c) {
                                const uint32_t p = base + static_cast<uint32_t>(
                                                              __popcll(bal & ((1ull << lane) - 1ull)));
                                if (p < static_cast<uint32_t>(kStage)) {
                                    stage_key[p] = (static_cast<uint64_t>(__float_as_uint(dist)) << 32) |
                                                   static_cast<uint32_t>(row);
                                    stage_q[p] = static_cast<uint8_t>(q);
                                }
                            }
                        }
                    }
                }
            }
            clear();
            return;
        }
        // the pass's extrema of each query fold into the tile's (LDS atomics) here,
        // so that no per-lane extrema stay live through the main loop
#pragma unroll
        for (int j = 0; j < MQW; ++j) {
            const float qsum = group4_sum(qqp[j]);  // ||q||^2 of query (jq + j)*16 + lr
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int q = (jq + j) * 16 + g * 4 + i;
                const float qn = __shfl(qsum, g * 4 + i);
                float tmn = __builtin_huge_valf(), tmx = 0.0f;
#pragma unroll
                for (int kb = 0; kb < KBW; ++kb) {
                    const int64_t row = c0 + (wave * KBW + kb) * 16 + lr;
                    const float dist = mk[kb] ? __uint_as_float(kMaskedBits)
                                              : clamp_nonneg(fmaf(-2.0f, acc[j][kb][i], qn + kk[kb]));
                    const bool ok = q < nq && row < r1;
                    // no branch around the store (nor any other memory operation in the loop)
                    *(ok ? a.dist + (qb + q) * a.ld + row : &g_mfma_sink) = dist;
                    tmn = ok && !mk[kb] ? fminf(tmn, dist) : tmn;
                    tmx = ok && !mk[kb] ? fmaxf(tmx, dist) : tmx;
                }
                tmn = row16_min(tmn);
                tmx = row16_max(tmx);
                if (lr == 0 && q < nq) {
                    atomicMin(&smin[q], __float_as_uint(tmn));
                    atomicMax(&smax[q], __float_as_uint(tmx));
                }
            }
        }
        clear();
    };

    // Step t: the matrix cores on span t (LDS buffer t % 2); span t + 1 goes
    // from its register set (t + 1) % NS to the other LDS buffer, and that set
    // starts loading span t + NS + 1; the barrier orders the LDS buffers
    // between the waves.  Steps past the tile's last span load that span
    // again (from L2) and write a buffer no one reads, and the step count is
    // padded to a multiple of NS with steps whose products are never stored,
    // so that no branch guards the loads.
    auto step = [&](int64_t t, int set) __attribute__((always_inline)) {
        compute(static_cast<int>(t & 1), t < nspan);
        write(set, static_cast<int>((t + 1) & 1));
        load(set, t + NS + 1 < T ? t + NS + 1 : T - 1);
        __syncthreads();
    };
    // after step t: the epilogue of its pass when t is the pass's last span (a
    // padding step is pass npass: rows past r1, nothing is stored)
    auto pass_end = [&](int64_t t) __attribute__((always_inline)) {
        const uint32_t p = static_cast<uint32_t>(t) / ns;
        if (static_cast<uint32_t>(t) - p * ns == ns - 1) epilogue(p);
    };
    load(0, 0);
    write(0, 0);
#pragma unroll
    for (int k = 1; k <= NS; ++k) load(k % NS, k < T ? k : T - 1);
    __syncthreads();
    for (int64_t t = 0; t < T; t += NS) {
#pragma unroll
        for (int k = 0; k < NS; ++k) {
            step(t + k, (k + 1) % NS);
            pass_end(t + k);
        }
    }

    if constexpr (FM == 2) {
        // the staged candidates to their queries' lists (no loads are in flight any more)
        __syncthreads();
        const uint32_t n = stage_n;
        if (n > static_cast<uint32_t>(kStage) && tid == 0) *a.fallback = 1u;
        const uint32_t m = n < static_cast<uint32_t>(kStage) ? n : static_cast<uint32_t>(kStage);
        for (uint32_t e = tid; e < m; e += kThreads) {
            const int64_t qq = qb + stage_q[e];
            const uint32_t pos = atomicAdd(a.cand_count + qq, 1u);
            if (pos < static_cast<uint32_t>(kFusedCap)) a.cand_list[qq * kFusedCap + pos] = stage_key[e];
        }
        return;
    }
    // the tile's extrema of each query (folded in by every pass's epilogue)
    if (a.tile_min != nullptr) {
        __syncthreads();
        for (int q = tid; q < nq; q += kThreads) {
            a.tile_min[(qb + q) * tiles + tile] = __uint_as_float(smin[q]);
            a.tile_max[(qb + q) * tiles + tile] = __uint_as_float(smax[q]);
        }
    }
}

template <knn_dtype DT, bool NORMS>
hipError_t launch_mq(int mq, const DistArgs &a, int64_t n_tiles, int64_t groups, dim3 grid, hipStream_t st,
                     int fm) {
    const dim3 b4(4 * kWave), b8(8 * kWave);
    if (fm != 0) {  // the fused select: 128-query workgroups only
        if (mq != 8) return hipErrorInvalidValue;
        if (fm == 1)
            hipLaunchKernelGGL((k_dist_mfma<DT, 8, 4, 2, 2, NORMS, 256, 64, 1>), grid, b8, 0, st, a, n_tiles, groups);
        else
            hipLaunchKernelGGL((k_dist_mfma<DT, 8, 4, 2, 2, NORMS, 256, 64, 2>), grid, b8, 0, st, a, n_tiles, groups);
        return hipGetLastError();
    }
    switch (mq) {
    case 1: hipLaunchKernelGGL((k_dist_mfma<DT, 1, 4, 1, 4, NORMS, 128, 128>), grid, b4, 0, st, a, n_tiles, groups); break;
    case 2: hipLaunchKernelGGL((k_dist_mfma<DT, 2, 4, 1, 3, NORMS, 128, 128>), grid, b4, 0, st, a, n_tiles, groups); break;
    case 4: hipLaunchKernelGGL((k_dist_mfma<DT, 4, 4, 1, 3, NORMS, 128, 128>), grid, b4, 0, st, a, n_tiles, groups); break;
    case 8: hipLaunchKernelGGL((k_dist_mfma<DT, 8, 4, 2, 2, NORMS, 256, 64>), grid, b8, 0, st, a, n_tiles, groups); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <knn_dtype DT>
hipError_t launch_dt(int mq, const DistArgs &a, int64_t n_tiles, int64_t groups, dim3 grid, hipStream_t st, int fm) {
    return a.key_sqnorms != nullptr ? launch_mq<DT, true>(mq, a, n_tiles, groups, grid, st, fm)
                                    : launch_mq<DT, false>(mq, a, n_tiles, groups, grid, st, fm);
}

}  // namespace

// Key rows per workgroup: at least 256, and enough that a tile runs at least
// 64 pipeline steps of 128 keys x 128 elements, at most 4096 rows; always a
// multiple of 256, so that both pass sizes divide it.
int mfma_tile_rows(int64_t d) {
    const int64_t nspan = d / kSpan > 0 ? d / kSpan : 1;
    int64_t rows = (64 + nspan - 1) / nspan * 128;
    rows = (rows + kTileQuantum - 1) / kTileQuantum * kTileQuantum;
    if (rows < kTileQuantum) rows = kTileQuantum;
    if (rows > 4096) rows = 4096;
    return static_cast<int>(rows);
}

hipError_t launch_distances_mfma(int mq, knn_dtype dtype, const DistArgs &args, int64_t S, int64_t groups,
                                 hipStream_t stream, int fm) {
    if (groups < 1 || args.rows_per_tile % kTileQuantum != 0 || args.d % kSpan != 0) return hipErrorInvalidConfiguration;
    if (fm != 0 && (args.sample_every < 1 || args.sample_rows < kTileQuantum || args.sample_rows % kTileQuantum != 0 ||
                    args.sample_rows > args.rows_per_tile))
        return hipErrorInvalidConfiguration;
    if (fm == 2 && (args.cand_thr == nullptr || args.cand_count == nullptr || args.cand_list == nullptr ||
                    args.fallback == nullptr))
        return hipErrorInvalidValue;
    const int64_t per_set = fm == 1 ? (args.tiles_per_set + args.sample_every - 1) / args.sample_every
                                    : args.tiles_per_set;
    const int64_t n_tiles = S * per_set;
    const int64_t nblocks = (n_tiles + 7) / 8 * 8 * groups;
    if (nblocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(nblocks));
    switch (dtype) {
    case KNN_BF16: return launch_dt<KNN_BF16>(mq, args, n_tiles, groups, grid, stream, fm);
    case KNN_F16: return launch_dt<KNN_F16>(mq, args, n_tiles, groups, grid, stream, fm);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace knnlm
