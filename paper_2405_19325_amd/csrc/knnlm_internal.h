// Internal interfaces between the C ABI (knnlm_api.hip) and the kernels:
// shared constants and the distance stage (the select and mixture stages are
// in select_internal.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "knnlm.h"

namespace knnlm {

constexpr int kWave = 64;           // CDNA wavefront width
constexpr int kDistThreads = 256;   // distance workgroup: 4 waves
constexpr int kSelectThreads = 1024;
constexpr int kSelectBinsLog2 = 11; // 2048-bin histogram per refinement pass
constexpr int kSelectBins = 1 << kSelectBinsLog2;
constexpr int kMaxCplVec = 16;      // 16-byte chunks per lane on the vector path (d <= 1024*VEC)

inline int elem_bytes(knn_dtype t) { return t == KNN_F32 ? 4 : 2; }
inline int vec_elems(knn_dtype t) { return 16 / elem_bytes(t); }

// How the distance kernel covers the (set, key tile, query group) space.
struct DistPlan {
    bool mfma;              // query batches: q.k on the matrix cores (16-bit elements, >= 16 queries per set)
    bool packed;            // MFMA path: the keys are the packed copy (knn_pack_keys)
    int mq;                 // MFMA path: 16-query blocks per workgroup (1, 2, 4 or 8)
    bool vec;               // 16-byte loads (d % VEC == 0, aligned rows) vs element loads
    int cpl;                // chunks per lane (vector path), power of two <= kMaxCplVec
    int nq;                 // queries per workgroup (1, 2, 4 or 8)
    int rows_per_tile;      // key rows per workgroup (from the workspace layout)
    int64_t tiles_per_set;  // ceil(max_keys / rows_per_tile)
    int64_t groups;         // ceil(max_queries / nq)
};

struct DistArgs {
    const void *queries;
    const void *keys;
    const float *key_sqnorms;    // may be null
    const int64_t *key_offsets;
    const int64_t *query_offsets;
    int64_t d;
    int64_t ld;                  // row stride of dist (>= max keys per set)
    float *dist;                 // [B, ld]
    float *tile_min;             // [B, tiles_per_set] or null
    float *tile_max;
    int64_t tiles_per_set;
    int rows_per_tile;
    const uint32_t *key_mask;    // bit (i & 31) of word i >> 5 set: global key row i is masked; or null
    // Gate: unless null, the launch does nothing when *gate != gate_run.
    const uint32_t *gate;
    uint32_t gate_run;
    // The fused select of query batches on long rows (launch_distances_fused):
    int sample_rows;             // rows of a sample piece, a multiple of 256
    int sample_every;            // tiles t with t % sample_every == 0 start with a sample piece
    const uint32_t *cand_thr;    // [B] a key is a candidate of query b when its distance bits are below this
    uint32_t *cand_count;        // [B] candidates listed so far
    uint64_t *cand_list;         // [B, kFusedCap] (distance bits << 32 | local key index)
    uint32_t *fallback;          // set to 1 when a candidate cannot be kept
    // Streaming kernels: per query, the smallest unmasked distance of each
    // wave's rows of each tile (group 4 t + w: rows r0 + w, r0 + w + 4, ... of
    // tile t), [B, groups_per_set]; or null.
    float *group_min;
    int64_t groups_per_set;
    // Words the select stage expects zero (its cross-workgroup counters),
    // cleared by the launch's first workgroup; or null.
    uint32_t *zero_words;
    int64_t n_zero_words;
};

// Candidates per query of the fused select (the wide select's list capacity).
constexpr int kFusedCap = 4096;

// A masked key row is at distance +infinity (bits kMaskedBits), above every
// real distance, and stays out of the per-tile extrema.
constexpr uint32_t kMaskedBits = 0x7f800000u;
__device__ __forceinline__ bool key_masked(const uint32_t *mask, int64_t g) {
    return ((mask[g >> 5] >> (g & 31)) & 1u) != 0u;
}

DistPlan plan_distances(int64_t d, knn_dtype dtype, int64_t max_queries, const void *queries,
                        const void *keys);

// The matrix-core path serves 16-bit keys with d % kMfmaSpan == 0 and
// d <= kMfmaMaxD when at least kMfmaMinQueries queries share a key set.
constexpr int kMfmaMinQueries = 16;
constexpr int kMfmaSpan = 128;
constexpr int64_t kMfmaMaxD = 65536;  // a 4096-row tile stays under 2^31 bytes
bool mfma_shape(int64_t d, knn_dtype dtype, int64_t max_queries);
int mfma_tile_rows(int64_t d);
int dist_tile_rows(int64_t d, knn_dtype dtype, int64_t S, int64_t max_keys, int64_t max_queries);

hipError_t launch_distances(const DistPlan &plan, knn_dtype dtype, const DistArgs &args, int64_t S,
                            hipStream_t stream);
// fm: 0 every tile, distances written; 1 the sample pieces only, distances
// written; 2 every row outside the sample pieces, candidates listed instead of
// distances written (mq 8 only).
hipError_t launch_distances_mfma(int mq, knn_dtype dtype, const DistArgs &args, int64_t S, int64_t groups,
                                 hipStream_t stream, int fm = 0);
// The same stages over keys in the packed layout (mfma_packed.hip).
hipError_t launch_distances_packed(int mq, knn_dtype dtype, const DistArgs &args, int64_t S, int64_t groups,
                                   hipStream_t stream, int fm = 0);
// Bytes of the packed copy of n rows of d 16-bit elements: blocks of 16 rows
// (the last one padded), each its fragments and then its rows' ||k||^2.
int64_t packed_key_bytes(int64_t n, int64_t d);
hipError_t launch_pack_keys(const void *keys, int64_t n, int64_t d, knn_dtype dtype, void *packed,
                            hipStream_t stream);
hipError_t launch_key_sqnorms(const void *keys, int64_t n, int64_t d, knn_dtype dtype, float *out,
                              hipStream_t stream);
}  // namespace knnlm
