// Internal interfaces between the C ABI (knnlm_api.hip) and the kernels.
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
    int mq;                 // MFMA path: 16-query blocks per workgroup (1, 2, 4 or 8)
    bool vec;               // 16-byte loads (d % VEC == 0, aligned rows) vs element loads
    int cpl;                // chunks per lane (vector path), power of two <= kMaxCplVec
    int nq;                 // queries per workgroup (1, 2, 4 or 8)
    int rows;               // rows per wave iteration
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
};

// A masked key row is at distance +infinity (bits kMaskedBits), above every
// real distance, and stays out of the per-tile extrema.
constexpr uint32_t kMaskedBits = 0x7f800000u;
__device__ __forceinline__ bool key_masked(const uint32_t *mask, int64_t g) {
    return ((mask[g >> 5] >> (g & 31)) & 1u) != 0u;
}

struct SelectArgs {
    const float *dist;           // [B, ld]
    const float *tile_min;       // [B, tiles_per_set] or null
    const float *tile_max;
    const int64_t *key_offsets;
    const int64_t *query_offsets;
    int64_t S;
    int64_t ld;
    int64_t tiles_per_set;
    int rows_per_tile;
    int r;
    int32_t *ids;                // [B, r]
    float *dists;                // [B, r]
    uint64_t *cand;              // split select: [B, parts, kSplitKeys] candidate keys, or null
    uint32_t *part_count;        // split select: [B, parts] candidates per part
    uint32_t *part_min;          // split select: [B, parts] smallest candidate distance bits per part
    uint32_t *part_thr;          // split select: [B] threshold on the distance bits
};

struct MixArgs {
    const int32_t *ids;          // [B, r]
    const float *dists;          // [B, r]
    const int32_t *values;
    const int64_t *key_offsets;
    const int64_t *query_offsets;
    const float *p_lm;           // [B, V]
    float *p_m;                  // [B, V]
    int64_t S;
    int64_t V;
    int r;
    float mu;
    float lambda;                // weight of p_LM (rrc == 0)
    int rrc;                     // 1: a weight per query from relative retrieval confidence
    float alpha, tau;            // its parameters (rrc == 1; tau > 0)
    float *lambda_out;           // [B] the weight each query used, or null (rrc == 1)
    // Decoding outputs of a NEST step (rrc == 1; all null, or next_token,
    // p_max, span_key and use_span given):
    const int32_t *draft;        // [B] the draft token each row checks, or null
    float *p_draft;              // [B] p_M(draft[b]) (0 for a token outside [0, V)); with draft
    float *p_max;                // [B] max_w p_M(w)
    int32_t *next_token;         // [B] the lowest w with p_M(w) = p_max
    int32_t *span_key;           // [B] the nearest neighbour in pi whose value is next_token, or -1
    int32_t *use_span;           // [B] 1 if lambda_t <= delta and span_key >= 0
    float delta;
};

hipError_t launch_spec_verify(const float *p_max, const float *p_draft, const int32_t *next_token,
                              const int64_t *draft_offsets, int64_t n_drafts, float gamma, const float *uniforms,
                              int32_t *n_accept, int32_t *out_token, hipStream_t stream);

DistPlan plan_distances(int64_t d, knn_dtype dtype, int64_t max_queries, const void *queries,
                        const void *keys);

// The matrix-core path serves 16-bit keys with d % kMfmaSpan == 0 when at
// least kMfmaMinQueries queries share a key set.
constexpr int kMfmaMinQueries = 16;
constexpr int kMfmaSpan = 128;
bool mfma_shape(int64_t d, knn_dtype dtype, int64_t max_queries);
int mfma_keys_per_pass();
int dist_tile_rows(int64_t d, knn_dtype dtype, int64_t S, int64_t max_keys, int64_t max_queries);

hipError_t launch_distances(const DistPlan &plan, knn_dtype dtype, const DistArgs &args, int64_t S,
                            hipStream_t stream);
hipError_t launch_distances_mfma(int mq, knn_dtype dtype, const DistArgs &args, int64_t S, int64_t groups,
                                 hipStream_t stream);
hipError_t launch_key_sqnorms(const void *keys, int64_t n, int64_t d, knn_dtype dtype, float *out,
                              hipStream_t stream);
int select_capacity(int r);
// Split select: rows of at most kSplitMaxN keys are cut into parts of
// kSplitKeys keys, one workgroup each, when r <= kSplitMaxR and the parts of
// all queries fit in one pass of the chip.  Returns the parts per query, or 0
// when a query's row is selected by a single workgroup.
constexpr int kSplitKeys = 4096;
constexpr int kSplitCap = 4096;
constexpr int64_t kSplitMaxN = 65536;
constexpr int kSplitMaxR = 1024;
constexpr int64_t kSplitMaxBlocks = 256;
int select_split_parts(int64_t B, int64_t ld, int r);
hipError_t launch_select(const SelectArgs &args, int64_t B, hipStream_t stream);
hipError_t launch_select_mix(const SelectArgs &args, const MixArgs &mix, int64_t B, hipStream_t stream);
hipError_t launch_mix(const MixArgs &args, int64_t B, hipStream_t stream);

}  // namespace knnlm
