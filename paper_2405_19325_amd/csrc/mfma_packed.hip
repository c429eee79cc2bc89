// Distance stage for query batches over keys in the packed layout: the same
// d(q, k) = ||q||^2 - 2 q.k + ||k||^2 (paper Section 2.2, the negative of the
// similarity s) as the row-major matrix-core kernel, with bit-identical
// results, read from a copy of the key store laid out in the order the matrix
// cores consume it.
//
// The packed layout (knn_pack_keys) cuts the [n, d] key matrix into blocks of
// 16 consecutive rows; block b holds, for each 32-element step c of d, one
// KiB in which lane l of a wave finds row 16 b + l % 16, elements
// 32 c + 8 (l / 16) .. +8 -- exactly the B operand of v_mfma_f32_16x16x32 for
// that step -- followed by the 16 rows' ||k||^2 in fp32 (32 d + 64 bytes per
// block).  One 16-byte load per lane then reads one contiguous KiB straight
// into the B registers: no LDS staging of keys, and every block is one
// contiguous stream (the row-major kernel's coalesced loads cover 256 bytes of
// each of 4 rows per instruction; loading B fragments straight from row-major
// keys would read 64 bytes of each of 16 rows per instruction, which streams
// markedly slower from HBM).  The stored norms are summed in the order the
// row-major kernel sums them on the fly (each lane its fragments' words in
// step order, then the four lane groups as (g0 + g1) + (g2 + g3)), so they
// are the same bits; caller-given norms replace them as in every other path.
//
// A wave takes KBW key blocks of a pass (NW x KBW x 16 keys) against all of
// the workgroup's MQ query blocks and walks d in steps of 64 elements (two
// MFMA steps).  Its keys load NS steps ahead into a ring of register sets.
// The queries (A operand) come from
//   QM = 0: global memory, loaded into the same ring (16-query groups: the
//           set's queries stay in L2, a quarter of the key bytes per step);
//   QM = 1: two LDS span buffers that all waves fill together, one barrier
//           per step (larger groups: their A fragments are read by every wave,
//           which would multiply L2 traffic).  Each thread's share of a step's
//           query span loads into the same ring set as that step's keys: the
//           memory counter completes loads in order, so a separate, shallower
//           query prefetch would make every wait for it a wait for all older
//           key loads as well, and the key ring would be as shallow as the
//           query prefetch (measured at 128 queries x 8.4 M keys of d = 1024:
//           4.0 ms with a two-step query prefetch, 3.0 ms in the key ring);
//   QM = 2: (128-query groups, four dividing the steps per pass) each step's
//           span loads straight into one of four LDS buffers three steps
//           ahead, so no registers hold it and the barrier that ends a step
//           waits only for loads issued two steps before (the kernel counts
//           those waits itself: the loads are assembly, load_to_lds_16); the
//           loop is unrolled over the four buffers, so every buffer address is
//           fixed (2-3% faster than QM 1 at the shape above; a barrier every
//           second step over eight buffers spilled registers and was no faster).
// Every step does the same MFMAs in the same k order as the row-major kernel,
// and ||k||^2 and ||q||^2 are accumulated over the same fragments in the same
// order, so every distance equals the row-major kernel's bit for bit.
//
// A tile of rows [r0, r1) of set s covers the packed blocks holding global
// rows k0 + r0 .. k0 + r1 - 1; when k0 is not a multiple of 16 the first and
// last blocks hold rows of a neighbouring tile or set, which are computed and
// discarded (stored into a sink word, left out of every extremum and list).
// Loads are never guarded by a branch (a branch around loads makes the
// compiler wait for every load in flight): blocks past the tile read the
// tile's first block, steps past the end re-read the last step.
#include "knnlm_internal.h"
#include "mfma_device.h"

namespace knnlm {

namespace {

// Where the epilogue stores the distances of rows outside the tile or query
// slots past the group: one word per device, written, never read.
__device__ float g_packed_sink;
// The mask word read when no key mask is given (no key masked).
__device__ uint32_t g_packed_no_mask;

constexpr int kPkSpan = 64;                 // elements of d per pipeline step
constexpr int kPkChunks = kPkSpan * 2 / 16;  // 16-byte chunks per row and step (LDS ring)
constexpr int kBlockRows = 16;
// QM 2: query spans load straight into LDS kPkQAhead steps ahead, into a ring of
// kPkQBufs span buffers (each span's buffer is reloaded only after the barrier
// that ends its step).
constexpr int kPkQAhead = 3;
constexpr int kPkQBufs = kPkQAhead + 1;

// Bytes of one packed block of 16 rows of d 16-bit elements: fragments, then norms.
__host__ __device__ constexpr int64_t packed_block_bytes(int64_t d) { return 32 * d + 4 * kBlockRows; }

template <knn_dtype DT, int MQ, int KBW, int NW, int NS, int QM, int FM>
__global__ __launch_bounds__(NW * kWave, 8 / NW) void k_dist_packed(DistArgs a, int64_t n_tiles, int64_t groups) {
    constexpr int NT = NW * kWave;
    constexpr int QB = MQ * 16;
    constexpr int PB = NW * KBW;  // key blocks per pass
    constexpr int QCH = QM != 0 ? QB * kPkChunks / NT : 1;
    static_assert(QM == 0 || (QB * kPkChunks) % NT == 0, "whole query chunks per thread");
    static_assert(QM != 1 || NS % 2 == 0, "the LDS ring alternates with the step's parity");
    static_assert(FM == 0 || MQ == 8, "the fused select runs on 128-query groups");
    __shared__ __align__(16) u32x4_t qlds[QM == 1 ? 2 : 1][QM == 1 ? QB * kPkChunks : 1];
    // QM 2: four span buffers (the loop is unrolled over them)
    static_assert(kPkQBufs == 4, "four span buffers");
    constexpr int QSZ = QM == 2 ? QB * kPkChunks : 1;
    __shared__ __align__(16) u32x4_t qb0[QSZ], qb1[QSZ], qb2[QSZ], qb3[QSZ];
    auto qbuf = [&](int i) __attribute__((always_inline)) { return i == 0 ? qb0 : i == 1 ? qb1 : i == 2 ? qb2 : qb3; };
    __shared__ uint32_t smin[QB], smax[QB];
    // ||q||^2 of the group's queries (written by every wave after each pass:
    // every wave sums the same A fragments in the same order) and, for FM 2,
    // their thresholds, read by the epilogue four queries at a time
    __shared__ __align__(16) float sqn[QB];
    __shared__ __align__(16) uint32_t sthr[FM == 2 ? QB : 4];
    constexpr int kStage = FM == 2 ? 1024 : 1;  // candidates staged per tile
    __shared__ uint64_t stage_key[kStage];
    __shared__ uint8_t stage_q[kStage];
    __shared__ uint32_t stage_n;
    static_assert(FM != 2 || QB <= 256, "a staged query fits a byte");

    if constexpr (FM == 0) {
        if (a.gate != nullptr && *a.gate != a.gate_run) return;
    }
    // Consecutive workgroups land on different XCDs (round robin over 8); the
    // query groups of one tile are numbered 8 apart, so they run on one XCD.
    const int64_t L = blockIdx.x;
    const int64_t grp = (L >> 3) % groups;
    const int64_t tl = ((L >> 3) / groups) * 8 + (L & 7);
    if (tl >= n_tiles) return;
    const int64_t tiles = a.tiles_per_set;
    const int64_t se = FM == 0 ? 1 : a.sample_every;
    // FM 1 takes one sample piece, FM 2 one whole sampling group of se tiles
    // (it writes no per-tile extrema, and long streams per workgroup run
    // faster: fewer pipeline fills and drains), FM 0 one tile
    const int64_t per_set = FM != 0 ? (tiles + se - 1) / se : tiles;
    const int64_t s = tl / per_set;
    const int64_t tile = FM != 0 ? (tl - s * per_set) * se : tl - s * per_set;
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    const int64_t qb = a.query_offsets[s] + grp * QB;
    const int64_t qe = a.query_offsets[s + 1];
    // this workgroup's rows [r0, r1): the tile, its sample piece (FM 1), or the
    // group's tiles past the piece at the start of its first (FM 2)
    int64_t r0 = tile * a.rows_per_tile;
    const int64_t rend = r0 + (FM == 1 ? a.sample_rows : FM == 2 ? se * a.rows_per_tile : a.rows_per_tile);
    if (FM == 2) r0 += a.sample_rows;
    if (qb >= qe || r0 >= N) return;  // uniform over the block
    const int nq = static_cast<int>(qe - qb < QB ? qe - qb : QB);
    const int64_t r1 = rend < N ? rend : N;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int g = lane >> 4, lr = lane & 15;
    const uint32_t rb = static_cast<uint32_t>(a.d * 2);  // bytes per row
    const uint32_t blk_bytes = static_cast<uint32_t>(packed_block_bytes(a.d));
    const uint32_t nspan = static_cast<uint32_t>(a.d / kPkSpan);
    // the packed blocks of global rows k0 + r0 .. k0 + r1 - 1
    const int64_t b0 = (k0 + r0) >> 4;
    const uint32_t nblk = static_cast<uint32_t>(((k0 + r1 + 15) >> 4) - b0);
    const uint32_t npass = (nblk + PB - 1) / PB;
    const uint32_t T = npass * nspan;  // pipeline steps
    const char *ptile = static_cast<const char *>(a.keys) + b0 * static_cast<int64_t>(blk_bytes);
    const char *qbase = static_cast<const char *>(a.queries) + qb * static_cast<int64_t>(rb);
    // local row (within the set) of the first row of block 0
    const int64_t lrow0 = b0 * kBlockRows - k0;
    // ||k||^2 of global row gr is nbase[((gr >> 4) - b0) * nstride + (gr & 15)]:
    // the caller's norms, or those stored in the packed blocks
    const float *nbase = a.key_sqnorms != nullptr ? a.key_sqnorms + b0 * kBlockRows
                                                  : reinterpret_cast<const float *>(ptile + 32 * a.d);
    const int64_t nstride = a.key_sqnorms != nullptr ? kBlockRows : static_cast<int64_t>(blk_bytes / 4);

    for (int q = tid; q < QB; q += NT) {
        smin[q] = 0xffffffffu;
        smax[q] = 0u;
    }
    if (FM == 2 && tid == 0) stage_n = 0u;
    if constexpr (FM == 2) {  // thresholds (0 past the group: nothing passes)
        for (int q = tid; q < QB; q += NT) sthr[q] = q < nq ? a.cand_thr[qb + q] : 0u;
    }

    // Register ring: set `set` holds one step's B fragments of this wave's
    // KBW blocks (two MFMA steps each) and, for QM 0, the A fragments.
    u32x4_t kr[NS][KBW][2];
    u32x4_t ar[QM == 0 ? NS : 1][QM == 0 ? MQ : 1][2];
    // QM 1: the step's query span, chunk i of this thread being row e / 8,
    // column e % 8 (e = i * NT + tid), bound for swizzled LDS slot swz(row, column)
    u32x4_t qr[QM == 1 ? NS : 1][QCH];
    uint32_t qso[QCH];
    int qslot[QCH];
#pragma unroll
    for (int i = 0; i < QCH; ++i) {
        const int e = i * NT + tid;
        if constexpr (QM == 2) {
            // LDS slot e (lane-consecutive, as the direct load writes them) holds the
            // chunk that the swizzle puts there: row e / 8, column (e % 8) ^ (row % 8)
            const int n = e / kPkChunks, c = (e % kPkChunks) ^ (n & (kPkChunks - 1));
            qso[i] = static_cast<uint32_t>(n < nq ? n : 0) * rb + static_cast<uint32_t>(c * 16);
            qslot[i] = e;
        } else {
            const int n = e / kPkChunks, c = e % kPkChunks;
            qso[i] = static_cast<uint32_t>(n < nq ? n : 0) * rb + static_cast<uint32_t>(c * 16);
            qslot[i] = swz<kPkChunks>(n, c);
        }
    }
    uint32_t qoff[MQ];  // QM 0: query row j * 16 + lr (the group's first past its end), this lane's 16 bytes
#pragma unroll
    for (int j = 0; j < MQ; ++j) {
        const int q = j * 16 + lr;
        qoff[j] = static_cast<uint32_t>(q < nq ? q : 0) * rb + static_cast<uint32_t>(g * 16);
    }
    auto load = [&](int set, uint32_t t) __attribute__((always_inline)) {
        const uint32_t p = t / nspan, sp = t - p * nspan;
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
            const uint32_t bi = p * PB + static_cast<uint32_t>(wave * KBW + kb);
            const uint32_t off = (bi < nblk ? bi : 0u) * blk_bytes + sp * 2048u + static_cast<uint32_t>(lane * 16);
#pragma unroll
            for (int c = 0; c < 2; ++c)
                kr[set][kb][c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(ptile + off + c * 1024));
        }
        if constexpr (QM == 0) {
#pragma unroll
            for (int j = 0; j < MQ; ++j)
#pragma unroll
                for (int c = 0; c < 2; ++c)
                    ar[set][j][c] = *reinterpret_cast<const u32x4_t *>(qbase + qoff[j] + sp * 128u + c * 64);
        } else {
#pragma unroll
            for (int i = 0; i < QCH; ++i) qr[set][i] = *reinterpret_cast<const u32x4_t *>(qbase + qso[i] + sp * 128u);
        }
    };
    auto qwrite = [&](int set, int buf) __attribute__((always_inline)) {
        if constexpr (QM == 1) {
#pragma unroll
            for (int i = 0; i < QCH; ++i) qlds[buf][qslot[i]] = qr[set][i];
        }
    };
    // QM 2: step t's query span straight into LDS buffer t % kPkQBufs; every
    // wave fills 64 consecutive slots per instruction (the LDS address is the
    // wave's, each lane's data lands 16 bytes after the previous lane's)
    auto qload = [&](uint32_t t, int b) __attribute__((always_inline)) {
        if constexpr (QM == 2) {
            const uint32_t sp = t % nspan;
            u32x4_t *buf = qbuf(b);
#pragma unroll
            for (int i = 0; i < QCH; ++i)
                load_to_lds_16(qbase + qso[i] + sp * 128u, buf + (i * NT + wave * kWave));
        }
    };

    f32x4_t acc[MQ][KBW];
    float qqp[MQ];
    // Per-pass row data for the epilogue, loaded one group of steps ahead and
    // unconditionally (rows outside the tile read its first row): ||k||^2 and
    // the mask word of each of this lane's key rows.
    float kn[KBW];
    uint32_t mw[KBW];
    auto row_of = [&](uint32_t p, int kb) __attribute__((always_inline)) {
        return lrow0 + static_cast<int64_t>(p * PB + static_cast<uint32_t>(wave * KBW + kb)) * kBlockRows + lr;
    };
    auto load_rows = [&](uint32_t t) __attribute__((always_inline)) {
        const uint32_t p = t / nspan;
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
            const int64_t row = row_of(p, kb);
            const int64_t gr = k0 + (row >= r0 && row < r1 ? row : r0);
            kn[kb] = nbase[((gr >> 4) - b0) * nstride + (gr & 15)];
            const uint32_t *mp = a.key_mask != nullptr ? a.key_mask + (gr >> 5) : &g_packed_no_mask;
            mw[kb] = *mp;
        }
    };
#pragma unroll
    for (int j = 0; j < MQ; ++j) qqp[j] = 0.0f;  // ||q||^2 partials: the first pass adds them up
    auto clear = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < MQ; ++j)
#pragma unroll
            for (int kb = 0; kb < KBW; ++kb) acc[j][kb] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    };
    clear();

    // Step t: the two MFMA steps of the span over set `set` (A from the ring
    // or from LDS buffer buf); with qn_pass, the query norms too.
    auto compute = [&](int set, int buf, bool qn_pass) __attribute__((always_inline)) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            u32x4_t af[MQ];
#pragma unroll
            for (int j = 0; j < MQ; ++j) {
                if constexpr (QM == 2) af[j] = qbuf(buf)[swz<kPkChunks>(j * 16 + lr, c * 4 + g)];
                else if constexpr (QM == 1) af[j] = qlds[buf][swz<kPkChunks>(j * 16 + lr, c * 4 + g)];
                else af[j] = ar[set][j][c];
            }
#pragma unroll
            for (int j = 0; j < MQ; ++j)
#pragma unroll
                for (int kb = 0; kb < KBW; ++kb) acc[j][kb] = mfma16<DT>(af[j], kr[set][kb][c], acc[j][kb]);
            if (qn_pass) {
#pragma unroll
                for (int j = 0; j < MQ; ++j) qqp[j] = dot_vec<DT>(af[j], qqp[j]);
            }
        }
    };

    // Distances of pass p: lane (g, lr) holds dot(query j*16 + 4g + i, the
    // key of row lr of this wave's block kb) in acc[j][kb][i].
    auto epilogue = [&](uint32_t p) __attribute__((always_inline)) {
        float kk[KBW];
        bool ok_row[KBW], mk[KBW];  // the row is this tile's; masked (Section 3.4: distance +infinity)
        int64_t row[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
            row[kb] = row_of(p, kb);
            ok_row[kb] = row[kb] >= r0 && row[kb] < r1;
            kk[kb] = kn[kb];
            mk[kb] = ok_row[kb] && ((mw[kb] >> ((k0 + row[kb]) & 31)) & 1u) != 0u;
        }
        // ||q||^2 of this lane's rows j * 16 + lr to LDS; this wave reads back those of
        // rows j * 16 + 4 g .. + 3, the queries whose products it holds (LDS
        // operations of one wave complete in order)
#pragma unroll
        for (int j = 0; j < MQ; ++j) {
            const float qsum = group4_sum(qqp[j]);  // every lane takes part in the exchange
            if (g == 0) sqn[j * 16 + lr] = qsum;
        }
        auto dist_of = [&](int j, int kb, int i, float qn) __attribute__((always_inline)) {
            return mk[kb] ? __uint_as_float(kMaskedBits) : clamp_nonneg(fmaf(-2.0f, acc[j][kb][i], qn + kk[kb]));
        };
        if constexpr (FM == 2) {
            // candidates: distance bits below the query's threshold.  They are
            // rare (about 1.2 r of a row's keys), so one ballot first tells
            // whether any lane of the wave holds one in this pass.
            bool any = false;
#pragma unroll
            for (int j = 0; j < MQ; ++j) {
                const f32x4_t qn4 = *reinterpret_cast<const f32x4_t *>(&sqn[j * 16 + 4 * g]);
                const u32x4_t th4 = *reinterpret_cast<const u32x4_t *>(&sthr[j * 16 + 4 * g]);
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int kb = 0; kb < KBW; ++kb)
                        any |= ok_row[kb] && __float_as_uint(dist_of(j, kb, i, qn4[i])) < th4[i];
            }
            if (__ballot(any) != 0ull) {
                // append them to the LDS stage a wave at a time (one LDS atomic per
                // wave that has any); queries past the group have threshold 0
#pragma unroll
                for (int j = 0; j < MQ; ++j) {
                    const f32x4_t qn4 = *reinterpret_cast<const f32x4_t *>(&sqn[j * 16 + 4 * g]);
                    const u32x4_t th4 = *reinterpret_cast<const u32x4_t *>(&sthr[j * 16 + 4 * g]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int q = j * 16 + g * 4 + i;
#pragma unroll
                        for (int kb = 0; kb < KBW; ++kb) {
                            const float dist = dist_of(j, kb, i, qn4[i]);
                            const bool c = ok_row[kb] && __float_as_uint(dist) < th4[i];
                            const uint64_t bal = __ballot(c);
                            if (bal != 0ull) {
                                const int first = __ffsll(static_cast<unsigned long long>(bal)) - 1;
                                uint32_t base = 0u;
                                if (lane == first) base = atomicAdd(&stage_n, static_cast<uint32_t>(__popcll(bal)));
                                base = readlane_u32(base, first);
                                if (c) {
                                    const uint32_t pos =
                                        base + static_cast<uint32_t>(__popcll(bal & ((1ull << lane) - 1ull)));
                                    if (pos < static_cast<uint32_t>(kStage)) {
                                        stage_key[pos] = (static_cast<uint64_t>(__float_as_uint(dist)) << 32) |
                                                         static_cast<uint32_t>(row[kb]);
                                        stage_q[pos] = static_cast<uint8_t>(q);
                                    }
                                }
                            }
                        }
                    }
                }
            }
            clear();
            return;
        }
        // the pass's extrema of each query fold into the tile's (LDS atomics)
#pragma unroll
        for (int j = 0; j < MQ; ++j) {
            const f32x4_t qn4 = *reinterpret_cast<const f32x4_t *>(&sqn[j * 16 + 4 * g]);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int q = j * 16 + g * 4 + i;
                float tmn = __builtin_huge_valf(), tmx = 0.0f;
#pragma unroll
                for (int kb = 0; kb < KBW; ++kb) {
                    const float dist = dist_of(j, kb, i, qn4[i]);
                    const bool ok = q < nq && ok_row[kb];
                    // no branch around the store
                    *(ok ? a.dist + (qb + q) * a.ld + row[kb] : &g_packed_sink) = dist;
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

    // Step t: the matrix cores on set t % NS (queries from LDS buffer t % 2),
    // then the set reloads step t + NS; with the LDS buffers, the next step's
    // query span goes from its ring set to the other buffer, and the barrier
    // orders the buffers.
    // Steps past the last one re-read it, and the step count is padded to a
    // multiple of NS with steps whose products are never stored.  A pass is a
    // whole number of groups of NS steps (the host launches NS dividing the
    // steps per pass), so the epilogue -- one copy of it -- runs after a group.
    // prologue
#pragma unroll
    for (int k = 0; k < NS; ++k) load(k, static_cast<uint32_t>(k) < T ? static_cast<uint32_t>(k) : T - 1);
    load_rows(NS - 1);
    if constexpr (QM == 1) qwrite(0, 0);
    if constexpr (QM == 2) {
#pragma unroll
        for (int k = 0; k < kPkQAhead; ++k) qload(static_cast<uint32_t>(k) < T ? static_cast<uint32_t>(k) : T - 1, k);
        __builtin_amdgcn_s_waitcnt(kVmcntZero);  // the direct loads are known to no register dependence
    }
    __syncthreads();  // the query span buffers, the extrema and the stage counter are set
    // QM 2 unrolls over the four span buffers (the host launches it when four divide the steps per pass)
    constexpr int U = QM == 2 ? kPkQBufs : NS;
    static_assert(U % NS == 0, "whole ring turns per loop body");
    for (uint32_t t0 = 0; t0 < T; t0 += U) {
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const uint32_t t = t0 + static_cast<uint32_t>(k);
            compute(k % NS, QM == 2 ? k : (k & 1), t < nspan);
            const uint32_t tn = t + NS;
            load(k % NS, tn < T ? tn : T - 1);
            if constexpr (QM == 1) {
                qwrite((k + 1) % NS, (k + 1) & 1);
                __syncthreads();
            }
            if constexpr (QM == 2) {
                // span t + kPkQAhead; then span t + 1 (loaded kPkQAhead - 1 steps ago) must
                // have landed: every step issues the same loads (KBW x 2 key fragments,
                // QCH query chunks), so at least that many per newer step are still
                // allowed in flight
                const uint32_t tq = t + kPkQAhead;
                qload(tq < T ? tq : T - 1, (k + kPkQAhead) % kPkQBufs);
                __builtin_amdgcn_s_waitcnt(vmcnt_encoding<(kPkQAhead - 1) * (2 * KBW + QCH)>());
                // a bare barrier: a fenced one would wait for every load in flight,
                // those of the spans ahead included; no memory access moves across it
                asm volatile("" ::: "memory");
                __builtin_amdgcn_s_barrier();
                asm volatile("" ::: "memory");
            }
        }
        const uint32_t te = t0 + U;  // steps done
        if (te % nspan == 0) epilogue(te / nspan - 1);
        load_rows(te + NS - 1);  // the row data of the next group's pass
    }

    if constexpr (FM == 2) {
        // the staged candidates to their queries' lists (no loads are in flight any more)
        __syncthreads();
        const uint32_t n = stage_n;
        if (n > static_cast<uint32_t>(kStage) && tid == 0) *a.fallback = 1u;
        const uint32_t m = n < static_cast<uint32_t>(kStage) ? n : static_cast<uint32_t>(kStage);
        for (uint32_t e = tid; e < m; e += NT) {
            const int64_t qq = qb + stage_q[e];
            const uint32_t pos = atomicAdd(a.cand_count + qq, 1u);
            if (pos < static_cast<uint32_t>(kFusedCap)) a.cand_list[qq * kFusedCap + pos] = stage_key[e];
        }
        return;
    }
    // the tile's extrema of each query (folded in by every pass's epilogue)
    if (a.tile_min != nullptr) {
        __syncthreads();
        for (int q = tid; q < nq; q += NT) {
            a.tile_min[(qb + q) * tiles + tile] = __uint_as_float(smin[q]);
            a.tile_max[(qb + q) * tiles + tile] = __uint_as_float(smax[q]);
        }
    }
}

// The packed copy.  Thread i writes 16-byte chunk i of the fragments: chunk
// (b * d / 32 + c) * 64 + l is row 16 b + l % 16, elements 32 c + 8 (l / 16) .. +8
// of the row-major keys (zeros for rows past n), at byte (c * 64 + l) * 16 of
// block b.
__global__ __launch_bounds__(256) void k_pack_fragments(const u32x4_t *keys, int64_t n, int64_t d, char *packed,
                                                        int64_t chunks) {
    const int64_t steps = d / 32;      // 32-element steps per row
    const int64_t row_chunks = d / 8;  // 16-byte chunks per row
    const int64_t bb = packed_block_bytes(d);
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < chunks;
         i += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t l = i & 63, bc = i >> 6;
        const int64_t b = bc / steps, c = bc - b * steps;
        const int64_t row = b * kBlockRows + (l & 15);
        const u32x4_t zero = {0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4_t *>(packed + b * bb + (c * 64 + l) * 16) =
            row < n ? keys[row * row_chunks + c * 4 + (l >> 4)] : zero;
    }
}

// ||k||^2 of every row into its block, in the matrix-core kernels' order:
// four threads per row, thread g summing the words of elements 32 c + 8 g .. +8
// for c = 0, 1, ... (dot2), then (g0 + g1) + (g2 + g3).  Rows past n get 0.
template <knn_dtype DT>
__global__ __launch_bounds__(256) void k_pack_norms(const u32x4_t *keys, int64_t n, int64_t d, char *packed,
                                                    int64_t rows) {
    const int64_t steps = d / 32;
    const int64_t row_chunks = d / 8;
    const int64_t bb = packed_block_bytes(d);
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < 4 * rows;
         i += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t row = i >> 2;
        const int g = static_cast<int>(i & 3);
        float p = 0.0f;
        if (row < n) {
            const u32x4_t *kr = keys + row * row_chunks + g;
            for (int64_t c = 0; c < steps; ++c) p = dot_vec<DT>(kr[4 * c], p);
        }
        p += __shfl_xor(p, 1);  // g0 + g1, g2 + g3 (the grid covers whole waves: every lane takes part)
        p += __shfl_xor(p, 2);  // (g0 + g1) + (g2 + g3)
        if (g == 0 && row < rows)
            reinterpret_cast<float *>(packed + (row / kBlockRows) * bb + 32 * d)[row % kBlockRows] = p;
    }
}

// Ring depth NS of each group size, used when NS divides the steps per pass
// (d / 64, always even); other passes take a ring of two.  Groups of 64 and
// 128 queries take two key blocks per wave and a ring of two: every A
// fragment read from LDS then serves 32 keys, which halves the LDS reads per
// key that bound the 128-query kernel (measured on random fp16 data at 128
// queries x 8.4 M keys of d = 1024, stand-alone: 3.3 ms against 4.1 ms with
// one block per wave and a ring of four).
template <int MQ>
constexpr int packed_ring() { return MQ >= 4 ? 2 : 4; }

template <knn_dtype DT, int MQ, int KBW, int NW, int QM, int FM>
void launch_packed_ns(bool deep, const DistArgs &a, int64_t n_tiles, int64_t groups, dim3 grid, hipStream_t st) {
    const dim3 block(NW * kWave);
    if (deep)
        hipLaunchKernelGGL((k_dist_packed<DT, MQ, KBW, NW, packed_ring<MQ>(), QM, FM>), grid, block, 0, st, a,
                           n_tiles, groups);
    else
        hipLaunchKernelGGL((k_dist_packed<DT, MQ, KBW, NW, 2, QM, FM>), grid, block, 0, st, a, n_tiles, groups);
}

template <knn_dtype DT>
hipError_t launch_packed_mq(int mq, const DistArgs &a, int64_t n_tiles, int64_t groups, dim3 grid, hipStream_t st,
                            int fm) {
    const int64_t nspan = a.d / kPkSpan;
    const bool direct = nspan % kPkQBufs == 0;  // 128-query groups: query spans loaded straight into LDS
    if (fm != 0) {  // the fused select: 128-query workgroups only
        if (mq != 8) return hipErrorInvalidValue;
        const bool deep = nspan % packed_ring<8>() == 0;
        if (direct && fm == 1) launch_packed_ns<DT, 8, 2, 8, 2, 1>(deep, a, n_tiles, groups, grid, st);
        else if (direct) launch_packed_ns<DT, 8, 2, 8, 2, 2>(deep, a, n_tiles, groups, grid, st);
        else if (fm == 1) launch_packed_ns<DT, 8, 2, 8, 1, 1>(deep, a, n_tiles, groups, grid, st);
        else launch_packed_ns<DT, 8, 2, 8, 1, 2>(deep, a, n_tiles, groups, grid, st);
        return hipGetLastError();
    }
    switch (mq) {
    case 1: launch_packed_ns<DT, 1, 4, 4, 0, 0>(nspan % packed_ring<1>() == 0, a, n_tiles, groups, grid, st); break;
    case 2: launch_packed_ns<DT, 2, 2, 4, 1, 0>(nspan % packed_ring<2>() == 0, a, n_tiles, groups, grid, st); break;
    case 4: launch_packed_ns<DT, 4, 2, 8, 1, 0>(nspan % packed_ring<4>() == 0, a, n_tiles, groups, grid, st); break;
    case 8:
        if (direct) launch_packed_ns<DT, 8, 2, 8, 2, 0>(nspan % packed_ring<8>() == 0, a, n_tiles, groups, grid, st);
        else launch_packed_ns<DT, 8, 2, 8, 1, 0>(nspan % packed_ring<8>() == 0, a, n_tiles, groups, grid, st);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_distances_packed(int mq, knn_dtype dtype, const DistArgs &args, int64_t S, int64_t groups,
                                   hipStream_t stream, int fm) {
    if (groups < 1 || args.rows_per_tile % kBlockRows != 0 || args.d % kPkSpan != 0)
        return hipErrorInvalidConfiguration;
    if (fm != 0 && (args.sample_every < 1 || args.sample_rows < kBlockRows || args.sample_rows % kBlockRows != 0 ||
                    args.sample_rows > args.rows_per_tile))
        return hipErrorInvalidConfiguration;
    if (fm == 2 && (args.cand_thr == nullptr || args.cand_count == nullptr || args.cand_list == nullptr ||
                    args.fallback == nullptr))
        return hipErrorInvalidValue;
    // a workgroup's rows (a tile, or a sampling group of tiles for fm 2) span at most
    // rows / 16 + 1 blocks: their byte offsets fit 32 bits
    const int64_t wg_rows = static_cast<int64_t>(args.rows_per_tile) * (fm == 2 ? args.sample_every : 1);
    if ((wg_rows / kBlockRows + 2) * packed_block_bytes(args.d) > 0xffffffffLL) return hipErrorInvalidConfiguration;
    const int64_t per_set = fm != 0 ? (args.tiles_per_set + args.sample_every - 1) / args.sample_every
                                    : args.tiles_per_set;
    const int64_t n_tiles = S * per_set;
    const int64_t nblocks = (n_tiles + 7) / 8 * 8 * groups;
    if (nblocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(nblocks));
    switch (dtype) {
    case KNN_BF16: return launch_packed_mq<KNN_BF16>(mq, args, n_tiles, groups, grid, stream, fm);
    case KNN_F16: return launch_packed_mq<KNN_F16>(mq, args, n_tiles, groups, grid, stream, fm);
    default: return hipErrorInvalidValue;
    }
}

int64_t packed_key_bytes(int64_t n, int64_t d) { return (n + kBlockRows - 1) / kBlockRows * packed_block_bytes(d); }

hipError_t launch_pack_keys(const void *keys, int64_t n, int64_t d, knn_dtype dtype, void *packed,
                            hipStream_t stream) {
    const int64_t nblk = (n + kBlockRows - 1) / kBlockRows;
    const int64_t chunks = nblk * kBlockRows * d / 8;
    if (chunks == 0) return hipSuccess;
    int64_t blocks = (chunks + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    const u32x4_t *k = static_cast<const u32x4_t *>(keys);
    char *out = static_cast<char *>(packed);
    hipLaunchKernelGGL(k_pack_fragments, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, k, n, d, out,
                       chunks);
    const int64_t rows = nblk * kBlockRows;
    int64_t nb = (4 * rows + 255) / 256;
    if (nb > 4096) nb = 4096;
    if (dtype == KNN_BF16)
        hipLaunchKernelGGL(k_pack_norms<KNN_BF16>, dim3(static_cast<unsigned>(nb)), dim3(256), 0, stream, k, n, d, out,
                           rows);
    else
        hipLaunchKernelGGL(k_pack_norms<KNN_F16>, dim3(static_cast<unsigned>(nb)), dim3(256), 0, stream, k, n, d, out,
                           rows);
    return hipGetLastError();
}

}  // namespace knnlm
