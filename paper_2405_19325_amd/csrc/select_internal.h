// Internal interfaces of the select, mixture and verification stages.
#pragma once

#include "knnlm_internal.h"

namespace knnlm {

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
    // Split select from group minima: the smallest unmasked distance of every
    // group of group_rows keys of a row ([B, groups_per_set], written by the
    // distance stage; group 4 t + w: rows 4 group_rows t + w + 4 e, e <
    // group_rows), or null.
    const float *group_min;
    int64_t groups_per_set;
    int group_rows;
    // Gate: unless null, a wide-select launch does nothing when *gate != gate_run.
    const uint32_t *gate;
    uint32_t gate_run;
};

// The fused select of query batches on long rows (the 128-query matrix-core
// distance kernel): a threshold per query from sampled keys, candidates
// listed by the distance kernel itself, so that the distance matrix is
// written only when the sample misjudges a query (the fallback word).
struct FusedArgs {
    int sample_rows;     // the first sample_rows rows of every sample_every-th tile are the sample
    int sample_every;
    uint32_t *thr;       // [B] threshold on the distance bits
    uint32_t *count;     // [B] candidates listed (true even past kFusedCap)
    uint64_t *list;      // [B, kFusedCap] (distance bits << 32 | local key index)
    uint32_t *fallback;  // 0: the lists hold every query's pi; 1: the distance matrix is written and selected
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
    // Split select whose finish writes each row in slices (NEST outputs):
    // [B] each, the row's largest entry key and its workgroup count, cleared
    // by the parts kernel or (no parts kernel) by the distance stage; or null.
    uint64_t *best;
    uint32_t *ticket;
};

hipError_t launch_spec_verify(const float *p_max, const float *p_draft, const int32_t *next_token,
                              const int64_t *draft_offsets, int64_t n_drafts, float gamma, const float *uniforms,
                              int32_t *n_accept, int32_t *out_token, hipStream_t stream);

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
// Split select from group minima (no parts kernel): the rows per key group
// (4 or 8) when a batch of split rows is served by the streaming distance
// kernels with rows_per_tile = 4 * group rows and every row of ld keys has at
// least 2 r groups; else 0.  The finish reads each row's group minima, takes
// as threshold the end of the histogram bin holding the r-th smallest (so at
// least r keys lie below it), and gathers the keys of the groups below it.
constexpr int kGroupMaxPerRow = 4 * kSelectThreads * 4;  // 16384: four 16-byte loads per thread
int select_group_rows(int64_t B, int64_t ld, int r, int rows_per_tile, bool streaming);
// Wide select: rows longer than kSplitMaxN keys are cut into parts (their
// candidate lists use the split layout, [B, parts, kSplitKeys]) when r <= 2048
// and the row has at least 2 r distance tiles; returns the parts per query
// (at most 64), or 0.
constexpr int64_t kWideBlocks = 2048;  // workgroups the wide select aims at
int select_wide_parts(int64_t B, int64_t ld, int r, int64_t tiles_per_set);
hipError_t launch_select(const SelectArgs &args, int64_t B, hipStream_t stream);
hipError_t launch_select_mix(const SelectArgs &args, const MixArgs &mix, int64_t B, hipStream_t stream);
hipError_t launch_mix(const MixArgs &args, int64_t B, hipStream_t stream);
// Fused select, after the sample pieces' distances (launch_distances_mfma fm 1):
// each query's threshold and the sample's candidates; clears the fallback word.
hipError_t launch_fused_threshold(const SelectArgs &args, const FusedArgs &f, int64_t B, hipStream_t stream);
// After the filter launch (fm 2): the fallback word is set if any query's
// candidate count lies outside [min(r, N), kFusedCap].
hipError_t launch_fused_check(const SelectArgs &args, const FusedArgs &f, int64_t B, hipStream_t stream);
// Select (and mixture) after the fused distance stage: from the lists when the
// fallback word is 0, else by the wide select over the distance matrix.
hipError_t launch_select_fused(const SelectArgs &args, const MixArgs *mix, const FusedArgs &f, int64_t B,
                               hipStream_t stream);
// Stores v into *word (a one-thread kernel, so that graph capture records no memset).
hipError_t launch_set_word(uint32_t *word, uint32_t v, hipStream_t stream);

}  // namespace knnlm
