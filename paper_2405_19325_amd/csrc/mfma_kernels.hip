// Distance stage for query batches: d(q, k) = ||q||^2 - 2 q.k + ||k||^2, the
// squared L2 distance whose negative is the paper's similarity (Section 2.2),
// with the q.k term on the gfx950 matrix cores.
//
// When many queries share one key set (speculative verification scores every
// draft position of a sequence against that sequence's store), the dot
// products form a dense [queries x d] . [d x keys] contraction: every key
// element is used by up to 128 queries, so streaming the keys from HBM once
// needs up to 128 flop per byte -- beyond the vector ALUs, within the
// matrix cores.  A workgroup of 4 waves takes passes of 4 * KB blocks of 16
// keys of one set (KB per wave) against up to 128 of the set's queries (MQ
// blocks of 16).  d is walked in spans of 128 elements.  In MFMA step c of a
// span, lane l holds key (or query) row l % 16 and elements 32c + 8 (l / 16)
// .. +8 -- the same elements for both operands, so the contraction is exact
// up to fp32 rounding -- and one 16-byte non-temporal load per (key block, c)
// reads 64 contiguous bytes of each of 16 rows.  The workgroup stages each
// span of its queries (read from cache: every workgroup of the set shares
// them) in LDS in exactly the A-operand lane order, so staging and reading
// are contiguous 1 KB accesses.  The next span's keys and queries load while
// v_mfma_f32_16x16x32 (bf16 or f16, fp32 accumulate) runs over the current
// one for every (query block, key block) pair; every load is unconditional,
// since a branch around loads makes the compiler wait for all loads in flight.
//
// ||k||^2 (unless precomputed) and ||q||^2 are dot2 chains over the same
// elements.  The summation order differs from the matrix cores', so unlike the
// streaming kernel a query equal to a key gives a distance of a few ulps of
// ||q||^2 + ||k||^2 rather than exactly 0 (clamped at 0 from below).
#include <type_traits>

#include "knnlm_device.h"
#include "knnlm_internal.h"

namespace knnlm {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kMfmaWaves = 4;
// Key rows per distance tile: a multiple of every variant's keys per pass
// (kMfmaWaves * KB * 16 for KB = 2 or 4).
constexpr int kMfmaTileRows = 256;

template <knn_dtype DT>
__device__ __forceinline__ f32x4_t mfma16(const uint4 a, const uint4 b, f32x4_t c) {
    if constexpr (DT == KNN_BF16) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                       c, 0, 0, 0);
    } else {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b),
                                                      c, 0, 0, 0);
    }
}

// min / max over the 16 lanes of a row (every lane of the row gets it).
__device__ __forceinline__ float row16_min(float v) {
    v = fminf(v, dpp_f32<0xB1>(v));
    v = fminf(v, dpp_f32<0x4E>(v));
    v = fminf(v, dpp_f32<0x141>(v));
    return fminf(v, dpp_f32<0x140>(v));
}

__device__ __forceinline__ float row16_max(float v) {
    v = fmaxf(v, dpp_f32<0xB1>(v));
    v = fmaxf(v, dpp_f32<0x4E>(v));
    v = fmaxf(v, dpp_f32<0x141>(v));
    return fmaxf(v, dpp_f32<0x140>(v));
}

// Sum over the four lanes l % 16 == const (lane groups): every one of them gets it.
__device__ __forceinline__ float group4_sum(float v) {
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}

constexpr int kSpan = kMfmaSpan;          // elements of d per pipeline step (256 bytes of a row)
constexpr int kFragBytes = kWave * 16;    // one MFMA operand fragment: 64 lanes x 16 bytes

// MQ: 16-query blocks per workgroup; KB: 16-key blocks per wave and pass;
// NORMS: ||k||^2 comes precomputed; OCC: waves per SIMD the registers must
// allow (measured best: 4 for one query block, 2 otherwise).
template <knn_dtype DT, int MQ, int KB, bool NORMS, int OCC>
__global__ __launch_bounds__(kMfmaWaves * kWave, OCC) void k_dist_mfma(DistArgs a, int64_t n_tiles, int64_t groups) {
    constexpr int QB = MQ * 16;
    constexpr int KEYS = kMfmaWaves * KB * 16;  // keys per pass
    // Staged query span, double-buffered.  Fragment (j, c) -- rows j*16 .. +16,
    // elements 32c .. +32 of the span -- sits lane-major at (j * 4 + c) * kFragBytes,
    // exactly as the MFMA A operand wants it, so staging and reading are both
    // contiguous 1 KB accesses.
    __shared__ __align__(16) unsigned char qlds[2][MQ * 4 * kFragBytes];
    __shared__ float sqq[kMfmaWaves][QB];
    __shared__ uint32_t smin[QB], smax[QB];

    // Consecutive workgroups land on different XCDs (round robin over 8).  The
    // query groups of one key tile are numbered 8 apart, so they run on one XCD
    // at about the same time and all but the first read the tile from its L2.
    const int64_t L = blockIdx.x;
    const int64_t grp = (L >> 3) % groups;
    const int64_t tl = ((L >> 3) / groups) * 8 + (L & 7);
    if (tl >= n_tiles) return;
    const int64_t tiles = a.tiles_per_set;
    const int64_t s = tl / tiles;
    const int64_t tile = tl - s * tiles;
    const int64_t k0 = a.key_offsets[s];
    int64_t N = a.key_offsets[s + 1] - k0;
    if (N > a.ld) N = a.ld;
    const int64_t qb = a.query_offsets[s] + grp * QB;
    const int64_t qe = a.query_offsets[s + 1];
    const int64_t r0 = tile * a.rows_per_tile;
    if (qb >= qe || r0 >= N) return;  // uniform over the block
    const int nq = static_cast<int>(qe - qb < QB ? qe - qb : QB);
    const int64_t r1 = (r0 + a.rows_per_tile < N) ? r0 + a.rows_per_tile : N;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int g = lane >> 4, lr = lane & 15;
    const int64_t row_bytes = a.d * 2;
    const int64_t nspan = a.d / kSpan;
    const char *qbase = static_cast<const char *>(a.queries) + qb * row_bytes;
    const char *kset = static_cast<const char *>(a.keys) + k0 * row_bytes;

    for (int q = tid; q < QB; q += kMfmaWaves * kWave) {
        smin[q] = 0xffffffffu;
        smax[q] = 0u;
    }

    // Every load is unconditional (d is a multiple of kSpan; a query row or
    // key row past the data reads row 0 of the block or tile instead, and the
    // results of those lanes are never used), so that no branch makes the
    // compiler wait for the loads already in flight.
    //
    // Query staging: wave `wave` stages fragments (m, wave) of a span -- query
    // row m*16 + lr, elements 32*wave + 8g .. +8 -- and its lanes sum the
    // squares of what they stage (||q||^2, completed over lanes and waves).
    const char *qptr[MQ];
#pragma unroll
    for (int m = 0; m < MQ; ++m) {
        const int qr = m * 16 + lr;
        qptr[m] = qbase + (qr < nq ? qr : 0) * row_bytes + 64 * wave + 16 * g;
    }

    for (int64_t c0 = r0; c0 < r1; c0 += KEYS) {
        float qqp[MQ];
#pragma unroll
        for (int m = 0; m < MQ; ++m) qqp[m] = 0.0f;
        auto load_q = [&](int64_t sp, uint4 (&qn)[MQ]) {
#pragma unroll
            for (int m = 0; m < MQ; ++m) qn[m] = *reinterpret_cast<const uint4 *>(qptr[m] + sp * (2 * kSpan));
        };
        auto stage_q = [&](int buf, const uint4 (&qn)[MQ]) {
#pragma unroll
            for (int m = 0; m < MQ; ++m) {
                *reinterpret_cast<uint4 *>(&qlds[buf][((m * 4 + wave) * kWave + lane) * 16]) = qn[m];
                qqp[m] = dot_chunk<DT>(qn[m], qn[m], qqp[m]);
            }
        };
        // Key chunk (kb, c) of span sp for this lane: row wrow + 16 kb, elements
        // 32c + 8g .. +8, so one load instruction reads 64 contiguous bytes of
        // each of 16 rows.
        const int64_t wrow = c0 + wave * (KB * 16) + lr;
        const char *kptr[KB];  // this lane's byte 16g of its row in each key block
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            const int64_t row = wrow + kb * 16;
            kptr[kb] = kset + (row < r1 ? row : r0) * row_bytes + 16 * g;
        }
        auto load_k = [&](int64_t sp, int kb, int c) {
            return load_stream(reinterpret_cast<const uint4 *>(kptr[kb] + sp * (2 * kSpan) + 64 * c));
        };

        f32x4_t acc[MQ][KB];
#pragma unroll
        for (int j = 0; j < MQ; ++j)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) acc[j][kb] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        float kkp[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) kkp[kb] = 0.0f;

        uint4 bk[KB][4];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int c = 0; c < 4; ++c) bk[kb][c] = load_k(0, kb, c);
        {
            uint4 qn[MQ];
            load_q(0, qn);
            stage_q(0, qn);
        }
        __syncthreads();

        // One span; with MORE the next one's keys and queries load meanwhile.
        // The last span is peeled off so that the loop body has no branch (a
        // branch around loads makes the compiler wait for every load in flight).
        auto span = [&](int64_t sp, auto more_tag) {
            constexpr bool MORE = decltype(more_tag)::value;
            const int cur = static_cast<int>(sp & 1);
            uint4 qn[MQ];
            if constexpr (MORE) load_q(sp + 1, qn);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                uint4 af[MQ];
#pragma unroll
                for (int j = 0; j < MQ; ++j)
                    af[j] = *reinterpret_cast<const uint4 *>(&qlds[cur][((j * 4 + c) * kWave + lane) * 16]);
#pragma unroll
                for (int j = 0; j < MQ; ++j)
#pragma unroll
                    for (int kb = 0; kb < KB; ++kb) acc[j][kb] = mfma16<DT>(af[j], bk[kb][c], acc[j][kb]);
                if constexpr (!NORMS) {
#pragma unroll
                    for (int kb = 0; kb < KB; ++kb) kkp[kb] = dot_chunk<DT>(bk[kb][c], bk[kb][c], kkp[kb]);
                }
                // chunk c of this span is consumed: start loading it for the next
                if constexpr (MORE) {
#pragma unroll
                    for (int kb = 0; kb < KB; ++kb) bk[kb][c] = load_k(sp + 1, kb, c);
                }
            }
            if constexpr (MORE) stage_q(cur ^ 1, qn);
            __syncthreads();
        };
        for (int64_t sp = 0; sp + 1 < nspan; ++sp) span(sp, std::true_type{});
        span(nspan - 1, std::false_type{});

        // ||q||^2 for the epilogue: lane (g, lr) needs query j*16 + 4g + i;
        // lanes g share a row, waves share the rest.
#pragma unroll
        for (int m = 0; m < MQ; ++m) {
            const float t = group4_sum(qqp[m]);
            if (g == 0) sqq[wave][m * 16 + lr] = t;
        }
        __syncthreads();
        float qsel[MQ][4];
#pragma unroll
        for (int j = 0; j < MQ; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int q = j * 16 + g * 4 + i;
                float t = sqq[0][q];
#pragma unroll
                for (int w = 1; w < kMfmaWaves; ++w) t += sqq[w][q];
                qsel[j][i] = t;
            }

        // Epilogue: lane (g, lr) holds dot(query j*16 + 4g + i, key wrow + 16 kb)
        // in acc[j][kb][i].
        float kk[KB];
        bool mk[KB];  // masked key rows (Section 3.4): distance +infinity, no part in the extrema
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            const int64_t row = wrow + kb * 16;
            kk[kb] = NORMS ? (row < r1 ? a.key_sqnorms[k0 + row] : 0.0f) : group4_sum(kkp[kb]);
            mk[kb] = a.key_mask != nullptr && row < r1 && key_masked(a.key_mask, k0 + row);
        }
#pragma unroll
        for (int j = 0; j < MQ; ++j) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int q = j * 16 + g * 4 + i;
                float mn = __builtin_huge_valf(), mx = 0.0f;
#pragma unroll
                for (int kb = 0; kb < KB; ++kb) {
                    const int64_t row = wrow + kb * 16;
                    const float dist = mk[kb] ? __uint_as_float(kMaskedBits)
                                              : clamp_nonneg(fmaf(-2.0f, acc[j][kb][i], qsel[j][i] + kk[kb]));
                    const bool ok = q < nq && row < r1;
                    if (ok) a.dist[(qb + q) * a.ld + row] = dist;
                    if (ok && !mk[kb]) {
                        mn = fminf(mn, dist);
                        mx = fmaxf(mx, dist);
                    }
                }
                mn = row16_min(mn);
                mx = row16_max(mx);
                if (lr == 0 && q < nq) {
                    atomicMin(&smin[q], __float_as_uint(mn));
                    atomicMax(&smax[q], __float_as_uint(mx));
                }
            }
        }
        __syncthreads();  // sqq and the query buffers are reused by the next pass
    }

    if (a.tile_min != nullptr) {
        __syncthreads();
        for (int q = tid; q < nq; q += kMfmaWaves * kWave) {
            a.tile_min[(qb + q) * tiles + tile] = __uint_as_float(smin[q]);
            a.tile_max[(qb + q) * tiles + tile] = __uint_as_float(smax[q]);
        }
    }
}

template <knn_dtype DT, bool NORMS>
hipError_t launch_mq(int mq, const DistArgs &a, int64_t n_tiles, int64_t groups, dim3 grid, hipStream_t st) {
    const dim3 block(kMfmaWaves * kWave);
    switch (mq) {
    case 1: hipLaunchKernelGGL((k_dist_mfma<DT, 1, 2, NORMS, 4>), grid, block, 0, st, a, n_tiles, groups); break;
    case 2: hipLaunchKernelGGL((k_dist_mfma<DT, 2, 4, NORMS, 2>), grid, block, 0, st, a, n_tiles, groups); break;
    case 4: hipLaunchKernelGGL((k_dist_mfma<DT, 4, 2, NORMS, 2>), grid, block, 0, st, a, n_tiles, groups); break;
    case 8: hipLaunchKernelGGL((k_dist_mfma<DT, 8, 2, NORMS, 2>), grid, block, 0, st, a, n_tiles, groups); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <knn_dtype DT>
hipError_t launch_dt(int mq, const DistArgs &a, int64_t n_tiles, int64_t groups, dim3 grid, hipStream_t st) {
    return a.key_sqnorms != nullptr ? launch_mq<DT, true>(mq, a, n_tiles, groups, grid, st)
                                    : launch_mq<DT, false>(mq, a, n_tiles, groups, grid, st);
}

}  // namespace

int mfma_keys_per_pass() { return kMfmaTileRows; }

hipError_t launch_distances_mfma(int mq, knn_dtype dtype, const DistArgs &args, int64_t S, int64_t groups,
                                 hipStream_t stream) {
    const int64_t n_tiles = S * args.tiles_per_set;
    if (groups < 1 || args.rows_per_tile % kMfmaTileRows != 0) return hipErrorInvalidConfiguration;
    const int64_t nblocks = (n_tiles + 7) / 8 * 8 * groups;
    if (nblocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const dim3 grid(static_cast<unsigned>(nblocks));
    switch (dtype) {
    case KNN_BF16: return launch_dt<KNN_BF16>(mq, args, n_tiles, groups, grid, stream);
    case KNN_F16: return launch_dt<KNN_F16>(mq, args, n_tiles, groups, grid, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace knnlm
