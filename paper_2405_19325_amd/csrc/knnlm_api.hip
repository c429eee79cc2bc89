// C ABI of the kNN-LM mixture step: host-side validation, workspace layout and
// the launches of the three stages on the caller's stream.
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "knnlm.h"
#include "select_internal.h"

// The workspace of knn_lm_mixture_noalloc: one array per GPU, held from the
// library's load until the process ends.  Host code never uses its name as an
// address (on the host it is only a stand-in for the symbol): the device
// address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[KNNLM_NOALLOC_SCRATCH_BYTES];

namespace {

using namespace knnlm;

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool valid_dtype(knn_dtype t) { return t == KNN_F32 || t == KNN_BF16 || t == KNN_F16; }

// The element type of a dtype argument, and whether it carries the packed-keys flag.
knn_dtype base_dtype(knn_dtype t) { return static_cast<knn_dtype>(static_cast<int>(t) & ~static_cast<int>(KNN_KEYS_PACKED)); }
bool packed_flag(knn_dtype t) { return (static_cast<int>(t) & static_cast<int>(KNN_KEYS_PACKED)) != 0; }

struct Layout {
    int rows_per_tile;
    int64_t tiles_per_set;
    int64_t ld;  // distance row stride = tiles_per_set * rows_per_tile
    int split_parts;  // > 0: the select runs split over parts, short rows or long (candidate lists and counts below)
    // The fused select (128-query batches on long rows): candidates listed by the
    // distance kernel from a threshold sampled per query; the distance matrix is
    // written only when the sample misjudges a query (the fallback word).
    bool fused;
    int sample_rows, sample_every;
    // Split select from group minima (the streaming distance kernels write
    // each wave's smallest distance; no parts kernel): rows per group, or 0.
    int group_rows;
    size_t off_dist, off_tmin, off_tmax, off_cand, off_count, off_thr, off_best, off_ticket, off_fallback, off_gmin,
        total;
};

// Whether a batch takes the fused select: the 128-query matrix-core kernel
// (more than 64 queries on a set) on rows long enough for the wide select.
bool fused_shape(int64_t B, int64_t d, knn_dtype dtype, int64_t max_queries, int64_t ld, int32_t r,
                 int64_t tiles_per_set) {
    return mfma_shape(d, dtype, max_queries) && max_queries > 64 && r <= kSplitMaxR &&
           select_split_parts(B, ld, r) == 0 && select_wide_parts(B, ld, r, tiles_per_set) > 0;
}

Layout layout(int64_t B, int64_t d, int64_t S, int64_t max_keys, int64_t max_queries, knn_dtype dtype, int32_t r) {
    Layout L{};
    L.rows_per_tile = dist_tile_rows(d, dtype, S, max_keys, max_queries);
    L.tiles_per_set = (max_keys + L.rows_per_tile - 1) / L.rows_per_tile;
    if (L.tiles_per_set < 1) L.tiles_per_set = 1;
    L.ld = L.tiles_per_set * L.rows_per_tile;
    L.off_dist = 0;
    L.off_tmin = align_up(L.off_dist + sizeof(float) * static_cast<size_t>(B) * static_cast<size_t>(L.ld));
    L.off_tmax = align_up(L.off_tmin + sizeof(float) * static_cast<size_t>(B) * static_cast<size_t>(L.tiles_per_set));
    L.off_cand = align_up(L.off_tmax + sizeof(float) * static_cast<size_t>(B) * static_cast<size_t>(L.tiles_per_set));
    L.split_parts = select_split_parts(B, L.ld, r);
    if (L.split_parts == 0) L.split_parts = select_wide_parts(B, L.ld, r, L.tiles_per_set);
    const size_t np = static_cast<size_t>(L.split_parts) * static_cast<size_t>(B);  // 0 unless split or wide
    L.off_count = align_up(L.off_cand + sizeof(uint64_t) * kSplitKeys * np);
    L.off_thr = align_up(L.off_count + 2 * sizeof(uint32_t) * np);  // counts, then minima
    const size_t per_row = L.split_parts > 0 ? static_cast<size_t>(B) : 0;  // split or wide: thresholds, NEST words
    L.off_best = align_up(L.off_thr + sizeof(uint32_t) * per_row);
    L.off_ticket = align_up(L.off_best + sizeof(uint64_t) * per_row);
    L.off_fallback = align_up(L.off_ticket + sizeof(uint32_t) * per_row);
    L.fused = fused_shape(B, d, dtype, max_queries, L.ld, r, L.tiles_per_set);
    // The sample: the first sample_rows rows (whole 256-key passes) of every
    // sample_every-th tile, 1/64 of the keys, in pieces small enough that the
    // sample launch fills the chip.  (1/64 keeps about 2,300 candidates per
    // query for r = 1024 against about 1,900 at 1/32, both well inside the
    // lists, and halves the sample pass and the threshold kernel's reads.)
    L.sample_rows = L.rows_per_tile / 8 > 256 ? L.rows_per_tile / 8 : 256;
    L.sample_every = 64 * L.sample_rows / L.rows_per_tile > 1 ? 64 * L.sample_rows / L.rows_per_tile : 1;
    L.group_rows = select_group_rows(B, L.ld, r, L.rows_per_tile, !mfma_shape(d, dtype, max_queries));
    L.off_gmin = align_up(L.off_fallback + (L.fused ? sizeof(uint32_t) : 0));
    const size_t gmin_words = L.group_rows > 0 ? static_cast<size_t>(B) * static_cast<size_t>(4 * L.tiles_per_set) : 0;
    L.total = align_up(L.off_gmin + sizeof(float) * gmin_words);
    return L;
}

bool finite_pos(float x) { return isfinite(x) && x > 0.0f; }

knn_status check_sizes(int64_t B, int64_t d, int64_t V, int64_t S, int64_t total_keys,
                       int64_t min_keys, int64_t max_keys, int64_t max_queries, knn_dtype dtype,
                       int32_t r, bool need_vocab) {
    if (B < 1 || d < 1 || S < 1 || total_keys < 1 || max_queries < 1) return KNN_ERR_INVALID_ARG;
    if (need_vocab && V < 1) return KNN_ERR_INVALID_ARG;
    if (!valid_dtype(dtype)) return KNN_ERR_INVALID_ARG;
    if (min_keys < 0 || max_keys < 1 || min_keys > max_keys || max_keys > total_keys || max_queries > B)
        return KNN_ERR_INVALID_ARG;
    if (r < 1) return KNN_ERR_INVALID_ARG;
    if (B > 0x7fffffffLL || max_keys > 0x7fffffffLL) return KNN_ERR_UNSUPPORTED;
    if (r > KNNLM_MAX_R) return KNN_ERR_UNSUPPORTED;
    if (need_vocab && V > 0x7fffffffLL) return KNN_ERR_UNSUPPORTED;
    if (d > (int64_t(1) << 40) / elem_bytes(dtype)) return KNN_ERR_UNSUPPORTED;
    if (r > min_keys) return KNN_ERR_R_EXCEEDS_N;
    const Layout L = layout(B, d, S, max_keys, max_queries, dtype, r);
    if (S * L.tiles_per_set > 0x7fffffffLL) return KNN_ERR_UNSUPPORTED;
    if (max_queries > 65535) return KNN_ERR_UNSUPPORTED;  // query groups per set on grid.y
    return KNN_OK;
}

knn_status check_scalars(float mu, float lambda) {
    if (!finite_pos(mu)) return KNN_ERR_INVALID_ARG;
    if (!(lambda >= 0.0f && lambda <= 1.0f)) return KNN_ERR_INVALID_ARG;
    return KNN_OK;
}

// Relative retrieval confidence: alpha finite, tau > 0 and finite.
knn_status check_rrc(float alpha, float tau) {
    if (!isfinite(alpha)) return KNN_ERR_INVALID_ARG;
    if (!finite_pos(tau)) return KNN_ERR_INVALID_ARG;
    return KNN_OK;
}

knn_status status_of(hipError_t e) { return e == hipSuccess ? KNN_OK : KNN_ERR_HIP; }

struct Call {
    const void *queries;
    const void *keys;
    const float *key_sqnorms;
    const int32_t *values;
    const int64_t *key_offsets;
    const int64_t *query_offsets;
    const float *p_lm;
    int64_t B, d, V, S, total_keys, min_keys, max_keys, max_queries;
    knn_dtype dtype;     // element type (the packed flag stripped)
    bool packed;         // keys: the packed copy (knn_pack_keys)
    int32_t r;
    float mu, lambda;
    int rrc;             // 1: lambda_t per query (eq. rrc) instead of lambda
    float alpha, tau;
    float *lambda_out;   // [B] lambda_t, or null
    const uint32_t *key_mask;  // masked key rows, or null
    // NEST decoding outputs (all null unless a NEST step)
    const int32_t *draft;
    float *p_draft, *p_max;
    int32_t *next_token, *span_key, *use_span;
    float delta;
    float *p_m;
    int32_t *nbr_ids;
    float *nbr_dists;
    void *workspace;
    size_t workspace_bytes;
};

knn_status validate_part(const Call &c, int part) {
    knn_status st = check_sizes(c.B, c.d, c.V, c.S, c.total_keys, c.min_keys, c.max_keys, c.max_queries,
                                c.dtype, c.r, part == 0 || part == KNN_PART_MIX || part == KNN_PART_SELECT_MIX);
    if (st != KNN_OK) return st;
    if (!c.key_offsets || !c.query_offsets) return KNN_ERR_INVALID_ARG;
    const bool dist = part == 0 || part == KNN_PART_DISTANCES;
    const bool sel = part == 0 || part == KNN_PART_SELECT || part == KNN_PART_SELECT_MIX;
    const bool mix = part == 0 || part == KNN_PART_MIX || part == KNN_PART_SELECT_MIX;
    if (dist && (!c.queries || !c.keys)) return KNN_ERR_INVALID_ARG;
    if (c.packed) {  // packed keys: 16-bit elements, read by the matrix-core kernels only
        if (c.dtype != KNN_BF16 && c.dtype != KNN_F16) return KNN_ERR_INVALID_ARG;
        if (dist && !plan_distances(c.d, c.dtype, c.max_queries, c.queries, c.keys).mfma) return KNN_ERR_UNSUPPORTED;
    }
    if ((sel || mix) && (!c.nbr_ids || !c.nbr_dists)) return KNN_ERR_INVALID_ARG;
    if (mix && (!c.values || !c.p_lm || !c.p_m)) return KNN_ERR_INVALID_ARG;
    if (mix && (st = check_scalars(c.mu, c.lambda)) != KNN_OK) return st;
    if (mix && c.rrc && (st = check_rrc(c.alpha, c.tau)) != KNN_OK) return st;
    if (c.next_token || c.p_max || c.span_key || c.use_span || c.draft || c.p_draft) {
        if (!c.rrc || !c.next_token || !c.p_max || !c.span_key || !c.use_span) return KNN_ERR_INVALID_ARG;
        if ((c.draft == nullptr) != (c.p_draft == nullptr)) return KNN_ERR_INVALID_ARG;
        if (!isfinite(c.delta)) return KNN_ERR_INVALID_ARG;
    }
    if (dist || sel) {
        if (!c.workspace) return KNN_ERR_WORKSPACE;
        if (reinterpret_cast<uintptr_t>(c.workspace) % kAlign) return KNN_ERR_WORKSPACE;
        const Layout L = layout(c.B, c.d, c.S, c.max_keys, c.max_queries, c.dtype, c.r);
        if (c.workspace_bytes < L.total) return KNN_ERR_WORKSPACE;
    }
    return KNN_OK;
}

MixArgs mix_args(const Call &c) {
    MixArgs a{};
    a.ids = c.nbr_ids;
    a.dists = c.nbr_dists;
    a.values = c.values;
    a.key_offsets = c.key_offsets;
    a.query_offsets = c.query_offsets;
    a.p_lm = c.p_lm;
    a.p_m = c.p_m;
    a.S = c.S;
    a.V = c.V;
    a.r = c.r;
    a.mu = c.mu;
    a.lambda = c.lambda;
    a.rrc = c.rrc;
    a.alpha = c.alpha;
    a.tau = c.tau;
    a.lambda_out = c.lambda_out;
    a.draft = c.draft;
    a.p_draft = c.p_draft;
    a.p_max = c.p_max;
    a.next_token = c.next_token;
    a.span_key = c.span_key;
    a.use_span = c.use_span;
    a.delta = c.delta;
    return a;
}

// The select stage's view of the workspace.
SelectArgs select_args(const Call &c, const Layout &L, char *ws) {
    SelectArgs a{};
    a.dist = ws ? reinterpret_cast<float *>(ws + L.off_dist) : nullptr;
    a.tile_min = ws ? reinterpret_cast<float *>(ws + L.off_tmin) : nullptr;
    a.tile_max = ws ? reinterpret_cast<float *>(ws + L.off_tmax) : nullptr;
    a.key_offsets = c.key_offsets;
    a.query_offsets = c.query_offsets;
    a.S = c.S;
    a.ld = L.ld;
    a.tiles_per_set = L.tiles_per_set;
    a.rows_per_tile = L.rows_per_tile;
    a.r = c.r;
    a.ids = c.nbr_ids;
    a.dists = c.nbr_dists;
    uint32_t *part_count = (ws && L.split_parts > 0) ? reinterpret_cast<uint32_t *>(ws + L.off_count) : nullptr;
    a.cand = (ws && L.split_parts > 0) ? reinterpret_cast<uint64_t *>(ws + L.off_cand) : nullptr;
    a.part_count = part_count;
    a.part_min = part_count ? part_count + L.split_parts * c.B : nullptr;
    a.part_thr = (ws && L.split_parts > 0) ? reinterpret_cast<uint32_t *>(ws + L.off_thr) : nullptr;
    a.group_min = (ws && L.group_rows > 0) ? reinterpret_cast<const float *>(ws + L.off_gmin) : nullptr;
    a.groups_per_set = 4 * L.tiles_per_set;
    a.group_rows = L.group_rows;
    return a;
}

// The fused select's lists share the wide select's candidate region (one list
// of kFusedCap per query; the wide select runs on it only after a fallback).
FusedArgs fused_args(const Layout &L, char *ws) {
    FusedArgs f{};
    f.sample_rows = L.sample_rows;
    f.sample_every = L.sample_every;
    f.list = reinterpret_cast<uint64_t *>(ws + L.off_cand);
    f.count = reinterpret_cast<uint32_t *>(ws + L.off_count);
    f.thr = reinterpret_cast<uint32_t *>(ws + L.off_thr);
    f.fallback = reinterpret_cast<uint32_t *>(ws + L.off_fallback);
    return f;
}

knn_status run_part(const Call &c, int part, hipStream_t stream) {
    const Layout L = layout(c.B, c.d, c.S, c.max_keys, c.max_queries, c.dtype, c.r);
    char *ws = static_cast<char *>(c.workspace);
    float *dist = ws ? reinterpret_cast<float *>(ws + L.off_dist) : nullptr;
    float *tmin = ws ? reinterpret_cast<float *>(ws + L.off_tmin) : nullptr;
    float *tmax = ws ? reinterpret_cast<float *>(ws + L.off_tmax) : nullptr;
    if (part == KNN_PART_DISTANCES) {
        DistPlan p = plan_distances(c.d, c.dtype, c.max_queries, c.queries, c.keys);
        p.packed = c.packed;
        p.rows_per_tile = L.rows_per_tile;
        p.tiles_per_set = L.tiles_per_set;
        DistArgs a{};
        a.queries = c.queries;
        a.keys = c.keys;
        a.key_sqnorms = c.key_sqnorms;
        a.key_offsets = c.key_offsets;
        a.query_offsets = c.query_offsets;
        a.d = c.d;
        a.ld = L.ld;
        a.dist = dist;
        a.tile_min = tmin;
        a.tile_max = tmax;
        a.tiles_per_set = L.tiles_per_set;
        a.rows_per_tile = L.rows_per_tile;
        a.key_mask = c.key_mask;
        if (ws && L.group_rows > 0) {  // the group minima, and the sliced finish's counters cleared
            a.group_min = reinterpret_cast<float *>(ws + L.off_gmin);
            a.groups_per_set = 4 * L.tiles_per_set;
            a.zero_words = reinterpret_cast<uint32_t *>(ws + L.off_best);
            a.n_zero_words = static_cast<int64_t>((L.off_ticket + sizeof(uint32_t) * c.B - L.off_best) / sizeof(uint32_t));
        }
        if (!L.fused) return status_of(launch_distances(p, c.dtype, a, c.S, stream));
        uint32_t *fallback = reinterpret_cast<uint32_t *>(ws + L.off_fallback);
        if (!(p.mfma && p.mq == 8)) {  // (misaligned rows) the whole matrix, selected by the wide select
            knn_status st = status_of(launch_distances(p, c.dtype, a, c.S, stream));
            return st != KNN_OK ? st : status_of(launch_set_word(fallback, 1u, stream));
        }
        // The sample pieces' distances, each query's threshold and the sample's
        // candidates, the rest of the rows listing candidates only, the count
        // check, and (only if a query's count is off) the whole matrix.
        const FusedArgs f = fused_args(L, ws);
        a.sample_rows = L.sample_rows;
        a.sample_every = L.sample_every;
        a.cand_thr = f.thr;
        a.cand_count = f.count;
        a.cand_list = f.list;
        a.fallback = f.fallback;
        const SelectArgs sa = select_args(c, L, ws);
        auto mfma = [&](int fm) {
            return p.packed ? launch_distances_packed(p.mq, c.dtype, a, c.S, p.groups, stream, fm)
                            : launch_distances_mfma(p.mq, c.dtype, a, c.S, p.groups, stream, fm);
        };
        hipError_t e = mfma(1);
        if (e == hipSuccess) e = launch_fused_threshold(sa, f, c.B, stream);
        if (e == hipSuccess) e = mfma(2);
        if (e == hipSuccess) e = launch_fused_check(sa, f, c.B, stream);
        if (e == hipSuccess) {
            a.gate = fallback;
            a.gate_run = 1u;
            e = mfma(0);
        }
        return status_of(e);
    }
    if (part == KNN_PART_SELECT || part == KNN_PART_SELECT_MIX) {
        const SelectArgs a = select_args(c, L, ws);
        if (L.fused) {
            const FusedArgs f = fused_args(L, ws);
            if (part == KNN_PART_SELECT) return status_of(launch_select_fused(a, nullptr, f, c.B, stream));
            const MixArgs mx = mix_args(c);
            return status_of(launch_select_fused(a, &mx, f, c.B, stream));
        }
        if (part == KNN_PART_SELECT) return status_of(launch_select(a, c.B, stream));
        MixArgs mx = mix_args(c);
        if (ws && L.split_parts > 0) {
            mx.best = reinterpret_cast<uint64_t *>(ws + L.off_best);
            mx.ticket = reinterpret_cast<uint32_t *>(ws + L.off_ticket);
        }
        return status_of(launch_select_mix(a, mx, c.B, stream));
    }
    if (part == KNN_PART_MIX) return status_of(launch_mix(mix_args(c), c.B, stream));
    return KNN_ERR_INVALID_ARG;
}

Call make_call(const void *queries, const void *keys, const float *key_sqnorms, const int32_t *values,
               const int64_t *key_offsets, const int64_t *query_offsets, const float *p_lm, int64_t B,
               int64_t d, int64_t V, int64_t S, int64_t total_keys, int64_t min_keys, int64_t max_keys,
               int64_t max_queries, knn_dtype dtype, int32_t r, float mu, float lambda, float *p_m,
               int32_t *nbr_ids, float *nbr_dists, void *workspace, size_t workspace_bytes) {
    Call c;
    c.queries = queries;
    c.keys = keys;
    c.key_sqnorms = key_sqnorms;
    c.values = values;
    c.key_offsets = key_offsets;
    c.query_offsets = query_offsets;
    c.p_lm = p_lm;
    c.B = B;
    c.d = d;
    c.V = V;
    c.S = S;
    c.total_keys = total_keys;
    c.min_keys = min_keys;
    c.max_keys = max_keys;
    c.max_queries = max_queries;
    c.dtype = base_dtype(dtype);
    c.packed = packed_flag(dtype);
    c.r = r;
    c.mu = mu;
    c.lambda = lambda;
    c.rrc = 0;
    c.alpha = 0.0f;
    c.tau = 1.0f;
    c.lambda_out = nullptr;
    c.key_mask = nullptr;
    c.draft = nullptr;
    c.p_draft = nullptr;
    c.p_max = nullptr;
    c.next_token = nullptr;
    c.span_key = nullptr;
    c.use_span = nullptr;
    c.delta = 0.5f;
    c.p_m = p_m;
    c.nbr_ids = nbr_ids;
    c.nbr_dists = nbr_dists;
    c.workspace = workspace;
    c.workspace_bytes = workspace_bytes;
    return c;
}

// Device address of `scratch` on the current device, resolved on the first
// call made with that device current and kept for later calls.
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxScratchDevices];

knn_status scratch_of_current_device(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return KNN_ERR_HIP;
    if (dev < 0 || dev >= kMaxScratchDevices) return KNN_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return KNN_ERR_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return KNN_OK;
}

}  // namespace

extern "C" {

knn_status knn_lm_mixture(const void *queries, const void *keys, const float *key_sqnorms,
                          const int32_t *values, const int64_t *key_offsets,
                          const int64_t *query_offsets, const float *p_lm, int64_t B, int64_t d,
                          int64_t V, int64_t S, int64_t total_keys, int64_t min_keys_per_set,
                          int64_t max_keys_per_set, int64_t max_queries_per_set, knn_dtype dtype,
                          int32_t r, float mu, float lambda, float *p_m, int32_t *nbr_ids,
                          float *nbr_dists, void *workspace, size_t workspace_bytes, void *stream) {
    const Call c = make_call(queries, keys, key_sqnorms, values, key_offsets, query_offsets, p_lm, B, d, V, S,
                             total_keys, min_keys_per_set, max_keys_per_set, max_queries_per_set, dtype, r, mu,
                             lambda, p_m, nbr_ids, nbr_dists, workspace, workspace_bytes);
    knn_status st = validate_part(c, 0);
    if (st != KNN_OK) return st;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    st = run_part(c, KNN_PART_DISTANCES, hs);
    if (st != KNN_OK) return st;
    return run_part(c, KNN_PART_SELECT_MIX, hs);
}

knn_status knn_lm_mixture_noalloc(const void *queries, const void *keys, const float *key_sqnorms,
                                  const int32_t *values, const int64_t *key_offsets,
                                  const int64_t *query_offsets, const float *p_lm, int64_t B, int64_t d,
                                  int64_t V, int64_t S, int64_t total_keys, int64_t min_keys_per_set,
                                  int64_t max_keys_per_set, int64_t max_queries_per_set, knn_dtype dtype,
                                  int32_t r, float mu, float lambda, float *p_m, int32_t *nbr_ids,
                                  float *nbr_dists, void *stream) {
    knn_status st = check_sizes(B, d, V, S, total_keys, min_keys_per_set, max_keys_per_set, max_queries_per_set,
                                base_dtype(dtype), r, true);
    if (st != KNN_OK) return st;
    const size_t need = layout(B, d, S, max_keys_per_set, max_queries_per_set, base_dtype(dtype), r).total;
    if (need > static_cast<size_t>(KNNLM_NOALLOC_SCRATCH_BYTES)) return KNN_ERR_WORKSPACE;
    void *ws = nullptr;
    if ((st = scratch_of_current_device(&ws)) != KNN_OK) return st;
    return knn_lm_mixture(queries, keys, key_sqnorms, values, key_offsets, query_offsets, p_lm, B, d, V, S,
                          total_keys, min_keys_per_set, max_keys_per_set, max_queries_per_set, dtype, r, mu, lambda,
                          p_m, nbr_ids, nbr_dists, ws, static_cast<size_t>(KNNLM_NOALLOC_SCRATCH_BYTES), stream);
}

knn_status knn_lm_mixture_rrc(const void *queries, const void *keys, const float *key_sqnorms,
                              const int32_t *values, const int64_t *key_offsets,
                              const int64_t *query_offsets, const float *p_lm, int64_t B, int64_t d,
                              int64_t V, int64_t S, int64_t total_keys, int64_t min_keys_per_set,
                              int64_t max_keys_per_set, int64_t max_queries_per_set, knn_dtype dtype,
                              int32_t r, float mu, float alpha, float tau, float *lambda_out, float *p_m,
                              int32_t *nbr_ids, float *nbr_dists, void *workspace, size_t workspace_bytes,
                              void *stream) {
    Call c = make_call(queries, keys, key_sqnorms, values, key_offsets, query_offsets, p_lm, B, d, V, S, total_keys,
                       min_keys_per_set, max_keys_per_set, max_queries_per_set, dtype, r, mu, 0.5f, p_m, nbr_ids,
                       nbr_dists, workspace, workspace_bytes);
    c.rrc = 1;
    c.alpha = alpha;
    c.tau = tau;
    c.lambda_out = lambda_out;
    knn_status st = validate_part(c, 0);
    if (st != KNN_OK) return st;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    st = run_part(c, KNN_PART_DISTANCES, hs);
    if (st != KNN_OK) return st;
    return run_part(c, KNN_PART_SELECT_MIX, hs);
}

knn_status knn_nest_step(const void *queries, const void *keys, const float *key_sqnorms, const int32_t *values,
                         const int64_t *key_offsets, const int64_t *query_offsets, const float *p_lm, int64_t B,
                         int64_t d, int64_t V, int64_t S, int64_t total_keys, int64_t min_keys_per_set,
                         int64_t max_keys_per_set, int64_t max_queries_per_set, knn_dtype dtype, int32_t r,
                         float mu, float alpha, float tau, float delta, const uint32_t *key_mask,
                         const int32_t *draft_tokens, float *lambda_out, float *p_m, int32_t *nbr_ids,
                         float *nbr_dists, int32_t *next_token, float *p_max, float *p_draft, int32_t *span_key,
                         int32_t *use_span, void *workspace, size_t workspace_bytes, void *stream) {
    Call c = make_call(queries, keys, key_sqnorms, values, key_offsets, query_offsets, p_lm, B, d, V, S, total_keys,
                       min_keys_per_set, max_keys_per_set, max_queries_per_set, dtype, r, mu, 0.5f, p_m, nbr_ids,
                       nbr_dists, workspace, workspace_bytes);
    c.rrc = 1;
    c.alpha = alpha;
    c.tau = tau;
    c.lambda_out = lambda_out;
    c.key_mask = key_mask;
    c.draft = draft_tokens;
    c.p_draft = p_draft;
    c.p_max = p_max;
    c.next_token = next_token;
    c.span_key = span_key;
    c.use_span = use_span;
    c.delta = delta;
    if (!next_token || !p_max || !span_key || !use_span) return KNN_ERR_INVALID_ARG;
    knn_status st = validate_part(c, 0);
    if (st != KNN_OK) return st;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    st = run_part(c, KNN_PART_DISTANCES, hs);
    if (st != KNN_OK) return st;
    return run_part(c, KNN_PART_SELECT_MIX, hs);
}

knn_status knn_spec_verify(const float *p_max, const float *p_draft, const int32_t *next_token,
                           const int64_t *draft_offsets, int64_t n_drafts, float gamma, const float *uniforms,
                           int32_t *n_accept, int32_t *out_token, void *stream) {
    if (!p_max || !p_draft || !next_token || !draft_offsets || !n_accept || !out_token) return KNN_ERR_INVALID_ARG;
    if (n_drafts < 1 || !(gamma > 0.0f && gamma <= 1.0f)) return KNN_ERR_INVALID_ARG;
    return status_of(launch_spec_verify(p_max, p_draft, next_token, draft_offsets, n_drafts, gamma, uniforms,
                                        n_accept, out_token, static_cast<hipStream_t>(stream)));
}

knn_status knn_lm_mixture_part(knn_part part, const void *queries, const void *keys,
                               const float *key_sqnorms, const int32_t *values,
                               const int64_t *key_offsets, const int64_t *query_offsets,
                               const float *p_lm, int64_t B, int64_t d, int64_t V, int64_t S,
                               int64_t total_keys, int64_t min_keys_per_set,
                               int64_t max_keys_per_set, int64_t max_queries_per_set,
                               knn_dtype dtype, int32_t r, float mu, float lambda, float *p_m,
                               int32_t *nbr_ids, float *nbr_dists, void *workspace,
                               size_t workspace_bytes, void *stream) {
    if (part != KNN_PART_DISTANCES && part != KNN_PART_SELECT && part != KNN_PART_MIX && part != KNN_PART_SELECT_MIX)
        return KNN_ERR_INVALID_ARG;
    const Call c = make_call(queries, keys, key_sqnorms, values, key_offsets, query_offsets, p_lm, B, d, V, S,
                             total_keys, min_keys_per_set, max_keys_per_set, max_queries_per_set, dtype, r, mu,
                             lambda, p_m, nbr_ids, nbr_dists, workspace, workspace_bytes);
    const knn_status st = validate_part(c, part);
    if (st != KNN_OK) return st;
    return run_part(c, part, static_cast<hipStream_t>(stream));
}

size_t knn_lm_mixture_workspace_size(int64_t B, int64_t d, int64_t V, int64_t S, int64_t total_keys,
                                     int64_t min_keys_per_set, int64_t max_keys_per_set,
                                     int64_t max_queries_per_set, knn_dtype dtype, int32_t r) {
    const knn_dtype et = base_dtype(dtype);
    if (check_sizes(B, d, V, S, total_keys, min_keys_per_set, max_keys_per_set, max_queries_per_set, et, r,
                    true) != KNN_OK)
        return 0;
    return layout(B, d, S, max_keys_per_set, max_queries_per_set, et, r).total;
}

knn_status knn_lm_mixture_validate(const void *queries, const void *keys, const int32_t *values,
                                   const int64_t *key_offsets, const int64_t *query_offsets,
                                   const float *p_lm, int64_t B, int64_t d, int64_t V, int64_t S,
                                   int64_t total_keys, int64_t min_keys_per_set,
                                   int64_t max_keys_per_set, int64_t max_queries_per_set,
                                   knn_dtype dtype, int32_t r, float mu, float lambda,
                                   const float *p_m, const int32_t *nbr_ids,
                                   const float *nbr_dists, const void *workspace,
                                   size_t workspace_bytes) {
    const Call c = make_call(queries, keys, nullptr, values, key_offsets, query_offsets, p_lm, B, d, V, S,
                             total_keys, min_keys_per_set, max_keys_per_set, max_queries_per_set, dtype, r, mu,
                             lambda, const_cast<float *>(p_m), const_cast<int32_t *>(nbr_ids),
                             const_cast<float *>(nbr_dists), const_cast<void *>(workspace), workspace_bytes);
    return validate_part(c, 0);
}

knn_status knn_distances(const void *queries, const void *keys, const float *key_sqnorms,
                         const int64_t *key_offsets, const int64_t *query_offsets, int64_t B,
                         int64_t d, int64_t S, int64_t max_keys_per_set,
                         int64_t max_queries_per_set, knn_dtype dtype, float *out, int64_t ld_out,
                         void *stream) {
    if (!queries || !keys || !key_offsets || !query_offsets || !out) return KNN_ERR_INVALID_ARG;
    if (B < 1 || d < 1 || S < 1 || max_keys_per_set < 1 || max_queries_per_set < 1 || max_queries_per_set > B)
        return KNN_ERR_INVALID_ARG;
    const bool packed = packed_flag(dtype);
    dtype = base_dtype(dtype);
    if (!valid_dtype(dtype) || ld_out < max_keys_per_set) return KNN_ERR_INVALID_ARG;
    if (packed && dtype != KNN_BF16 && dtype != KNN_F16) return KNN_ERR_INVALID_ARG;
    if (B > 0x7fffffffLL || max_keys_per_set > 0x7fffffffLL || max_queries_per_set > 65535) return KNN_ERR_UNSUPPORTED;
    DistPlan p = plan_distances(d, dtype, max_queries_per_set, queries, keys);
    if (packed && !p.mfma) return KNN_ERR_UNSUPPORTED;
    p.packed = packed;
    p.rows_per_tile = dist_tile_rows(d, dtype, S, max_keys_per_set, max_queries_per_set);
    p.tiles_per_set = (max_keys_per_set + p.rows_per_tile - 1) / p.rows_per_tile;
    if (S * p.tiles_per_set > 0x7fffffffLL || p.groups > 65535) return KNN_ERR_UNSUPPORTED;
    DistArgs a{};
    a.queries = queries;
    a.keys = keys;
    a.key_sqnorms = key_sqnorms;
    a.key_offsets = key_offsets;
    a.query_offsets = query_offsets;
    a.d = d;
    a.ld = ld_out;
    a.dist = out;
    a.tile_min = nullptr;
    a.tile_max = nullptr;
    a.tiles_per_set = p.tiles_per_set;
    a.rows_per_tile = p.rows_per_tile;
    return status_of(launch_distances(p, dtype, a, S, static_cast<hipStream_t>(stream)));
}

knn_status knn_key_sqnorms(const void *keys, int64_t n, int64_t d, knn_dtype dtype, float *out, void *stream) {
    if (!keys || !out || n < 0 || d < 1 || !valid_dtype(dtype)) return KNN_ERR_INVALID_ARG;
    return status_of(launch_key_sqnorms(keys, n, d, dtype, out, static_cast<hipStream_t>(stream)));
}

size_t knn_packed_keys_bytes(int64_t n, int64_t d, knn_dtype dtype) {
    const knn_dtype et = base_dtype(dtype);
    if (n < 1 || d < 1 || (et != KNN_BF16 && et != KNN_F16) || d % kMfmaSpan != 0 || d > kMfmaMaxD) return 0;
    if (n > (int64_t(1) << 40) / (2 * d)) return 0;
    return static_cast<size_t>(packed_key_bytes(n, d));
}

knn_status knn_pack_keys(const void *keys, int64_t n, int64_t d, knn_dtype dtype, void *packed, void *stream) {
    if (!keys || !packed) return KNN_ERR_INVALID_ARG;
    if (knn_packed_keys_bytes(n, d, dtype) == 0) return n < 1 || d < 1 ? KNN_ERR_INVALID_ARG : KNN_ERR_UNSUPPORTED;
    if ((reinterpret_cast<uintptr_t>(keys) & 15u) || (reinterpret_cast<uintptr_t>(packed) & 15u))
        return KNN_ERR_INVALID_ARG;
    return status_of(launch_pack_keys(keys, n, d, base_dtype(dtype), packed, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {

knn_status mix_call(const int32_t *nbr_ids, const float *nbr_dists, const int32_t *values, const int64_t *key_offsets,
                    const int64_t *query_offsets, const float *p_lm, int64_t B, int64_t V, int64_t S, int32_t r,
                    float mu, float lambda, int rrc, float alpha, float tau, float *lambda_out, float *p_m,
                    void *stream) {
    if (!nbr_ids || !nbr_dists || !values || !key_offsets || !query_offsets || !p_lm || !p_m)
        return KNN_ERR_INVALID_ARG;
    if (B < 1 || V < 1 || S < 1 || r < 1) return KNN_ERR_INVALID_ARG;
    if (r > KNNLM_MAX_R || B > 0x7fffffffLL || V > 0x7fffffffLL) return KNN_ERR_UNSUPPORTED;
    knn_status st = check_scalars(mu, lambda);
    if (st != KNN_OK) return st;
    if (rrc && (st = check_rrc(alpha, tau)) != KNN_OK) return st;
    MixArgs a{};
    a.ids = nbr_ids;
    a.dists = nbr_dists;
    a.values = values;
    a.key_offsets = key_offsets;
    a.query_offsets = query_offsets;
    a.p_lm = p_lm;
    a.p_m = p_m;
    a.S = S;
    a.V = V;
    a.r = r;
    a.mu = mu;
    a.lambda = lambda;
    a.rrc = rrc;
    a.alpha = alpha;
    a.tau = tau;
    a.lambda_out = lambda_out;
    return status_of(launch_mix(a, B, static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

knn_status knn_mix(const int32_t *nbr_ids, const float *nbr_dists, const int32_t *values,
                   const int64_t *key_offsets, const int64_t *query_offsets, const float *p_lm,
                   int64_t B, int64_t V, int64_t S, int32_t r, float mu, float lambda, float *p_m,
                   void *stream) {
    return mix_call(nbr_ids, nbr_dists, values, key_offsets, query_offsets, p_lm, B, V, S, r, mu, lambda, 0, 0.0f,
                    1.0f, nullptr, p_m, stream);
}

knn_status knn_mix_rrc(const int32_t *nbr_ids, const float *nbr_dists, const int32_t *values,
                       const int64_t *key_offsets, const int64_t *query_offsets, const float *p_lm,
                       int64_t B, int64_t V, int64_t S, int32_t r, float mu, float alpha, float tau,
                       float *lambda_out, float *p_m, void *stream) {
    return mix_call(nbr_ids, nbr_dists, values, key_offsets, query_offsets, p_lm, B, V, S, r, mu, 0.5f, 1, alpha,
                    tau, lambda_out, p_m, stream);
}

const char *knn_status_string(knn_status status) {
    switch (status) {
    case KNN_OK: return "ok";
    case KNN_ERR_INVALID_ARG: return "invalid argument";
    case KNN_ERR_R_EXCEEDS_N: return "r exceeds the smallest key set";
    case KNN_ERR_UNSUPPORTED: return "unsupported size or configuration";
    case KNN_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case KNN_ERR_HIP: return "HIP launch failed";
    }
    return "unknown status";
}

int knn_abi_version(void) { return KNNLM_ABI_VERSION; }

}  // extern "C"
