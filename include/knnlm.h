/*
 * knnlm.h -- C ABI of the MI355X (gfx950) kNN-LM mixture step.
 *
 * The operation (paper "Nearest Neighbor Speculative Decoding", Section 2.2,
 * paragraph "Probability interpolation", eq. non-parametric and eq. kNN-LM;
 * Section 3.1 "Second-stage kNN token search"; Appendix A): for every decoding
 * query q_t and the key/value store (K', V') built from that sequence's
 * retrieved passages,
 *
 *   s(q, k)  = -||q - k||^2                        (negative squared L2 distance)
 *   pi       = the r keys with the largest s       (ties: lower key index first)
 *   p_kNN(w) = sum_{(k_i, v_i) in pi, v_i = w} exp(mu s(q, k_i)) / sum_{pi} exp(mu s)
 *   p_M(w)   = lambda p_LM(w) + (1 - lambda) p_kNN(w)
 *
 * Data model.  B queries are grouped into S key sets.  Set s owns the query
 * rows query_offsets[s] .. query_offsets[s+1]-1 and the key rows (and values)
 * key_offsets[s] .. key_offsets[s+1]-1; neighbour ids are LOCAL row indices
 * within the query's own set.  Every matrix is row-major and dense.  Queries
 * carry the key element type (round fp32 queries to it before the call).
 *
 * Memory.  Unless a parameter says "host", every pointer is a DEVICE pointer
 * (hipMalloc'd or torch CUDA storage) on the current device.  The caller owns
 * every buffer; the library allocates and frees nothing.  Scratch space comes
 * from the caller's `workspace`, sized by knn_lm_mixture_workspace_size().
 *
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  Calls only
 * validate on the host and enqueue work; they never synchronise.  Outputs are
 * valid once the stream reaches that point.  A launch failure returns
 * KNN_ERR_HIP; a device fault surfaces at the caller's next synchronisation.
 *
 * Errors.  No call prints, throws or aborts.  Argument errors are detected on
 * the host before anything is enqueued and leave every output untouched.
 *
 * Preconditions the library does not check on the device: finite query and
 * key elements, values in [0, V), offsets monotone with key_offsets[0] = 0 and
 * query_offsets[0] = 0, and planning hints that are true.  If a hint is false
 * the results are unspecified, but every device access stays inside the
 * buffers the hints describe.
 *
 * Thread safety.  Stateless and re-entrant; concurrent calls need distinct
 * workspaces.
 */
#ifndef KNNLM_H
#define KNNLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KNNLM_ABI_VERSION 2

/* Largest r accepted (the paper retrieves r = 1024, Appendix A). */
#define KNNLM_MAX_R 4096

/* Size of the per-GPU scratch array behind knn_lm_mixture_noalloc (32 MiB). */
#define KNNLM_NOALLOC_SCRATCH_BYTES (32u << 20)

typedef enum {
    KNN_OK = 0,
    KNN_ERR_INVALID_ARG = 1,  /* null pointer, bad size, mu/lambda out of range, bad hint */
    KNN_ERR_R_EXCEEDS_N = 2,  /* r larger than the smallest key set (min_keys_per_set) */
    KNN_ERR_UNSUPPORTED = 3,  /* valid request the library does not serve (r > KNNLM_MAX_R, ...) */
    KNN_ERR_WORKSPACE = 4,    /* workspace NULL or smaller than knn_lm_mixture_workspace_size() */
    KNN_ERR_HIP = 5           /* a HIP launch failed */
} knn_status;

/*
 * Element type of queries and keys.  KNN_KEYS_PACKED, OR'ed into a 16-bit type
 * (KNN_BF16_PACKED, KNN_F16_PACKED), says that `keys` is the packed copy of
 * the key matrix written by knn_pack_keys rather than the row-major matrix;
 * queries stay row-major.  Packed keys are read by the matrix-core distance
 * kernels only, which serve calls with d % 128 == 0, d <= 65536 and
 * max_queries_per_set >= 16 (and 16-byte aligned queries and keys); a call
 * with packed keys outside that returns KNN_ERR_UNSUPPORTED.  Results are
 * bit for bit those of the same call on the row-major keys.
 */
typedef enum {
    KNN_F32 = 0,
    KNN_BF16 = 1,
    KNN_F16 = 2,
    KNN_KEYS_PACKED = 0x100,
    KNN_BF16_PACKED = 0x101,
    KNN_F16_PACKED = 0x102
} knn_dtype;

/* Stages of knn_lm_mixture, runnable one at a time by knn_lm_mixture_part().
 * knn_lm_mixture itself runs KNN_PART_DISTANCES then KNN_PART_SELECT_MIX. */
typedef enum {
    KNN_PART_DISTANCES = 1, /* squared distances of every query to its set (into the workspace) */
    KNN_PART_SELECT = 2,    /* top-r per query: nbr_ids, nbr_dists */
    KNN_PART_MIX = 3,       /* softmax over mu*s, scatter onto values, lambda-mix: p_m */
    KNN_PART_SELECT_MIX = 4 /* SELECT and MIX in one launch */
} knn_part;

/*
 * knn_lm_mixture -- the whole step (eq. non-parametric, then eq. kNN-LM).
 *
 *   queries        [B, d] dtype.
 *   keys           [total_keys, d] dtype; set s = rows key_offsets[s]..key_offsets[s+1]-1.
 *   key_sqnorms    [total_keys] fp32 ||k||^2 from knn_key_sqnorms(), or NULL to
 *                  compute them on the fly (no extra bytes read).
 *   values         [total_keys] int32 next-token id of each key, in [0, V).
 *   key_offsets    [S+1] int64, monotone, key_offsets[0] = 0, key_offsets[S] = total_keys.
 *   query_offsets  [S+1] int64, monotone, query_offsets[0] = 0, query_offsets[S] = B.
 *   p_lm           [B, V] fp32 LM next-token distribution.
 *   B, d, V, S     sizes (all >= 1).
 *   total_keys     number of key rows.
 *   min_keys_per_set, max_keys_per_set, max_queries_per_set
 *                  host planning hints: the smallest key set among sets that
 *                  own at least one query, the largest key set, and the
 *                  largest number of queries owned by one set (<= 65535).
 *   dtype          element type of queries and keys.
 *   r              neighbours per query, 1 <= r <= min(KNNLM_MAX_R, min_keys_per_set).
 *   mu             inverse temperature > 0 (the paper uses 1/sqrt(d)).
 *   lambda         weight of p_LM, in [0, 1] (lambda = 1 returns p_LM bit for bit).
 *   p_m            [B, V] fp32 out: the mixture.
 *   nbr_ids        [B, r] int32 out: local key ids of pi, ascending (distance, id).
 *   nbr_dists      [B, r] fp32 out: their squared L2 distances (>= 0), = -s.
 *   workspace      device scratch of at least knn_lm_mixture_workspace_size() bytes,
 *                  256-byte aligned; contents on entry are ignored.
 */
knn_status knn_lm_mixture(const void *queries, const void *keys, const float *key_sqnorms,
                          const int32_t *values, const int64_t *key_offsets,
                          const int64_t *query_offsets, const float *p_lm, int64_t B, int64_t d,
                          int64_t V, int64_t S, int64_t total_keys, int64_t min_keys_per_set,
                          int64_t max_keys_per_set, int64_t max_queries_per_set, knn_dtype dtype,
                          int32_t r, float mu, float lambda, float *p_m, int32_t *nbr_ids,
                          float *nbr_dists, void *workspace, size_t workspace_bytes, void *stream);

/*
 * knn_lm_mixture_noalloc -- knn_lm_mixture without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that forbid allocation).  It computes exactly what
 * knn_lm_mixture computes, with the same kernels, and allocates nothing: its
 * scratch space is a static array of KNNLM_NOALLOC_SCRATCH_BYTES in device
 * memory, one per GPU, held from the library's first use on that GPU until
 * the process ends.  Its device address is looked up on the first call with
 * that GPU current (make that first call outside graph capture).
 *
 * Arguments as knn_lm_mixture; the caller still owns every input and output.
 * If knn_lm_mixture_workspace_size() for these sizes exceeds
 * KNNLM_NOALLOC_SCRATCH_BYTES the call returns KNN_ERR_WORKSPACE and enqueues
 * nothing (32 MiB serves, e.g., 64 queries on sets of up to 65,536 keys at
 * d = 4096, or 16 queries on sets of 131,072 keys at d = 8192).
 *
 * Every call on one GPU shares that GPU's array, and nothing in it needs to
 * start at any value (each call writes what it later reads): two calls that
 * can run at the same time on one GPU (different streams without ordering)
 * race on it and give unspecified results.  Calls on one stream are ordered
 * and safe.
 */
knn_status knn_lm_mixture_noalloc(const void *queries, const void *keys, const float *key_sqnorms,
                                  const int32_t *values, const int64_t *key_offsets,
                                  const int64_t *query_offsets, const float *p_lm, int64_t B, int64_t d,
                                  int64_t V, int64_t S, int64_t total_keys, int64_t min_keys_per_set,
                                  int64_t max_keys_per_set, int64_t max_queries_per_set, knn_dtype dtype,
                                  int32_t r, float mu, float lambda, float *p_m, int32_t *nbr_ids,
                                  float *nbr_dists, void *stream);

/*
 * knn_lm_mixture_rrc -- the whole step with a weight of p_LM per query from
 * relative retrieval confidence (paper Section 3.2, eq. rrc) in place of the
 * fixed lambda: with s_i = -nbr_dists[b, i] over query b's r neighbours,
 *
 *   lambda_t(b) = sigmoid((min_i |s_i| / max_i |s_i| - alpha) / tau)
 *               = sigmoid((d_(1) / d_(r) - alpha) / tau),
 *
 * computed in fp32 from the neighbours' fp32 distances (a query whose r
 * distances are all 0 takes ratio 1), then p_M as in knn_lm_mixture with
 * lambda_t(b) for query b.  Arguments as knn_lm_mixture, and:
 *   alpha          threshold on the ratio, finite (the paper uses 0.3, or 0.2).
 *   tau            temperature > 0 (the paper uses 0.1).
 *   lambda_out     [B] fp32 out: lambda_t of each query, or NULL.
 * A bad alpha or tau returns KNN_ERR_INVALID_ARG.
 */
knn_status knn_lm_mixture_rrc(const void *queries, const void *keys, const float *key_sqnorms,
                              const int32_t *values, const int64_t *key_offsets,
                              const int64_t *query_offsets, const float *p_lm, int64_t B, int64_t d,
                              int64_t V, int64_t S, int64_t total_keys, int64_t min_keys_per_set,
                              int64_t max_keys_per_set, int64_t max_queries_per_set, knn_dtype dtype,
                              int32_t r, float mu, float alpha, float tau, float *lambda_out, float *p_m,
                              int32_t *nbr_ids, float *nbr_dists, void *workspace, size_t workspace_bytes,
                              void *stream);

/*
 * knn_nest_step -- one decoding step of NEST (paper Algorithm 1, one time
 * step, without the corpus n-gram fetch): the token search with masked keys
 * left out, p_kNN, lambda_t from relative retrieval confidence and p_M exactly
 * as knn_lm_mixture_rrc computes them, followed by the decisions the algorithm
 * takes on p_M.  Arguments as knn_lm_mixture_rrc, and:
 *   delta          span threshold of eq. span_expansion (Section 3.3), finite
 *                  (the paper uses 0.5).
 *   key_mask       [ceil(total_keys / 32)] uint32 or NULL: bit (i & 31) of word
 *                  i >> 5 set means global key row i is masked (Section 3.4,
 *                  last paragraph: the keys of an accepted span are not used
 *                  again).  A masked key is never a neighbour; if a set keeps
 *                  fewer than r unmasked keys, the remaining slots of pi hold
 *                  id -1 and distance +infinity and carry no weight (with no
 *                  neighbour at all, p_kNN = 0 and p_M = lambda_t p_LM).
 *   draft_tokens   [B] int32 or NULL: the draft token each row checks (relaxed
 *                  speculative decoding, Section 3.4); p_draft must then be given.
 *   next_token     [B] int32 out: w_t = argmax_w p_M(w), the lowest id among
 *                  equal maxima (Algorithm 1, dynamic span selection).
 *   p_max          [B] fp32 out: p_M(w_t).
 *   p_draft        [B] fp32 out or NULL: p_M(draft_tokens[b]), 0 for a token
 *                  outside [0, V).
 *   span_key       [B] int32 out: the start of the span (eq. knn_interpolation,
 *                  max-pooling read as the neighbour with the largest softmax
 *                  weight): the local id of the nearest neighbour in pi whose
 *                  value is w_t (lower id on equal distances), or -1 if none.
 *   use_span       [B] int32 out: 1 if lambda_t <= delta and span_key >= 0
 *                  (eq. span_expansion), else 0.
 * next_token, p_max, span_key and use_span are required.
 */
knn_status knn_nest_step(const void *queries, const void *keys, const float *key_sqnorms, const int32_t *values,
                         const int64_t *key_offsets, const int64_t *query_offsets, const float *p_lm, int64_t B,
                         int64_t d, int64_t V, int64_t S, int64_t total_keys, int64_t min_keys_per_set,
                         int64_t max_keys_per_set, int64_t max_queries_per_set, knn_dtype dtype, int32_t r,
                         float mu, float alpha, float tau, float delta, const uint32_t *key_mask,
                         const int32_t *draft_tokens, float *lambda_out, float *p_m, int32_t *nbr_ids,
                         float *nbr_dists, int32_t *next_token, float *p_max, float *p_draft, int32_t *span_key,
                         int32_t *use_span, void *workspace, size_t workspace_bytes, void *stream);

/*
 * knn_spec_verify -- relaxed speculative verification of drafts (Section 3.4,
 * eq. rejection, and Algorithm 1) from the per-row outputs of knn_nest_step.
 * Draft j owns rows draft_offsets[j] .. draft_offsets[j+1]-1 (int64, device,
 * monotone); row i holds p_M given the prefix and the draft tokens before
 * row i's own.  ratio_i = p_draft[i] / (gamma * p_max[i]) in fp32.  Without
 * uniforms a draft token is accepted while ratio_i > 0.5; with uniforms [rows]
 * fp32 in [0, 1) drawn by the caller, while uniforms[i] < min(1, ratio_i).
 *   n_accept    [n_drafts] int32 out: draft tokens accepted before the first rejection.
 *   out_token   [n_drafts] int32 out: next_token of the first rejected row (the
 *               replacement), or -1 if every draft token was accepted.
 * gamma in (0, 1]; n_drafts >= 1.
 */
knn_status knn_spec_verify(const float *p_max, const float *p_draft, const int32_t *next_token,
                           const int64_t *draft_offsets, int64_t n_drafts, float gamma, const float *uniforms,
                           int32_t *n_accept, int32_t *out_token, void *stream);

/*
 * knn_lm_mixture_part -- one stage of knn_lm_mixture with the same arguments.
 * KNN_PART_DISTANCES followed by either KNN_PART_SELECT_MIX or KNN_PART_SELECT
 * then KNN_PART_MIX, on one stream with one workspace, computes what
 * knn_lm_mixture computes (neighbours and distances bit for bit; p_m up to
 * the order of float additions in the scatter).  Pointers a stage does not
 * use may be NULL (DISTANCES: values, p_lm, p_m, nbr_ids, nbr_dists; SELECT:
 * queries, keys, key_sqnorms, values, p_lm, p_m; MIX: queries, keys,
 * key_sqnorms, workspace; SELECT_MIX: queries, keys, key_sqnorms).
 */
knn_status knn_lm_mixture_part(knn_part part, const void *queries, const void *keys,
                               const float *key_sqnorms, const int32_t *values,
                               const int64_t *key_offsets, const int64_t *query_offsets,
                               const float *p_lm, int64_t B, int64_t d, int64_t V, int64_t S,
                               int64_t total_keys, int64_t min_keys_per_set,
                               int64_t max_keys_per_set, int64_t max_queries_per_set,
                               knn_dtype dtype, int32_t r, float mu, float lambda, float *p_m,
                               int32_t *nbr_ids, float *nbr_dists, void *workspace,
                               size_t workspace_bytes, void *stream);

/* Bytes of workspace knn_lm_mixture needs for these sizes (0 if they are invalid). */
size_t knn_lm_mixture_workspace_size(int64_t B, int64_t d, int64_t V, int64_t S,
                                     int64_t total_keys, int64_t min_keys_per_set,
                                     int64_t max_keys_per_set, int64_t max_queries_per_set,
                                     knn_dtype dtype, int32_t r);

/*
 * knn_lm_mixture_validate -- the host-side argument checks of knn_lm_mixture,
 * without enqueuing anything.  Pointers are only tested for NULL, never
 * dereferenced, so it runs without a GPU.
 */
knn_status knn_lm_mixture_validate(const void *queries, const void *keys, const int32_t *values,
                                   const int64_t *key_offsets, const int64_t *query_offsets,
                                   const float *p_lm, int64_t B, int64_t d, int64_t V, int64_t S,
                                   int64_t total_keys, int64_t min_keys_per_set,
                                   int64_t max_keys_per_set, int64_t max_queries_per_set,
                                   knn_dtype dtype, int32_t r, float mu, float lambda,
                                   const float *p_m, const int32_t *nbr_ids,
                                   const float *nbr_dists, const void *workspace,
                                   size_t workspace_bytes);

/*
 * knn_distances -- the distance stage alone, written to a caller matrix
 * (s(q,k) = -||q-k||^2, paper Section 2.2): out[b * ld_out + i] = ||q_b - k_i||^2
 * (fp32, >= 0) for i < N of b's set, via ||q||^2 - 2 q.k + ||k||^2 with fp32
 * accumulation.  Entries i >= N of a row are not written.  Requires
 * ld_out >= max_keys_per_set.  key_sqnorms may be NULL.
 */
knn_status knn_distances(const void *queries, const void *keys, const float *key_sqnorms,
                         const int64_t *key_offsets, const int64_t *query_offsets, int64_t B,
                         int64_t d, int64_t S, int64_t max_keys_per_set,
                         int64_t max_queries_per_set, knn_dtype dtype, float *out, int64_t ld_out,
                         void *stream);

/*
 * knn_key_sqnorms -- ||k_i||^2 in fp32 for n rows of d elements.  The key store
 * is built once per input before decoding starts (paper Algorithm 1), so these
 * can be computed once per store and passed to every later call.  The
 * summation order equals the one knn_lm_mixture uses on the fly, so a query
 * equal to a key gets distance exactly 0 either way.
 */
knn_status knn_key_sqnorms(const void *keys, int64_t n, int64_t d, knn_dtype dtype, float *out,
                           void *stream);

/*
 * knn_pack_keys -- the packed copy of a key matrix for query batches on the
 * matrix cores.  Like knn_key_sqnorms it is computed once per key store (the
 * store is built before decoding starts, paper Algorithm 1) and then passed as
 * `keys` with dtype KNN_BF16_PACKED / KNN_F16_PACKED to every later call.
 *
 * Layout: the n x d row-major matrix `keys` (16-bit dtype, d % 128 == 0,
 * d <= 65536) is cut into blocks of 16 consecutive rows (the last one padded
 * with zero rows).  Block b, 32-element step c of d, occupies the 1024 bytes
 * at byte offset (b * d / 32 + c) * 1024; its 16-byte chunk l (l = 0..63) holds
 * elements 32 c + 8 (l / 16) .. 32 c + 8 (l / 16) + 7 of row 16 b + l % 16 --
 * the B operand of one 16x16x32 matrix-core step for lane l.  `packed` must
 * hold knn_packed_keys_bytes(n, d, dtype) bytes; both pointers 16-byte aligned
 * device memory, not overlapping.  Key sets keep their row offsets: a set may
 * start anywhere, not only on a block boundary.
 * Errors: KNN_ERR_INVALID_ARG for null or misaligned pointers or n, d < 1;
 * KNN_ERR_UNSUPPORTED for an fp32 dtype, d % 128 != 0 or d > 65536.
 */
knn_status knn_pack_keys(const void *keys, int64_t n, int64_t d, knn_dtype dtype, void *packed, void *stream);

/* Bytes of the packed copy of n key rows of d elements: ceil(n / 16) * 16 * d * 2,
 * or 0 where knn_pack_keys would refuse the sizes or dtype. */
size_t knn_packed_keys_bytes(int64_t n, int64_t d, knn_dtype dtype);

/*
 * knn_mix -- the softmax / scatter / mixture stage alone (eq. non-parametric
 * and eq. kNN-LM) on caller-given neighbours: for each query b of set s, the
 * r entries (nbr_ids[b, j], nbr_dists[b, j]) in any order.  An entry whose id
 * lies outside [0, N_s) is absent (as the -1 slots a masked select leaves): it
 * carries no weight and takes no part in the softmax; with no entry present
 * p_kNN = 0.  A value outside [0, V) gives its weight to no token.  p_m [B, V]
 * is written.
 */
knn_status knn_mix(const int32_t *nbr_ids, const float *nbr_dists, const int32_t *values,
                   const int64_t *key_offsets, const int64_t *query_offsets, const float *p_lm,
                   int64_t B, int64_t V, int64_t S, int32_t r, float mu, float lambda, float *p_m,
                   void *stream);

/*
 * knn_mix_rrc -- knn_mix with lambda_t per query from relative retrieval
 * confidence (Section 3.2, eq. rrc) over the query's r caller-given distances
 * (any order): sigmoid((min_j nbr_dists[b, j] / max_j nbr_dists[b, j] - alpha) / tau),
 * ratio 1 if every distance is 0.  alpha finite, tau > 0; lambda_out [B] fp32
 * out or NULL.
 */
knn_status knn_mix_rrc(const int32_t *nbr_ids, const float *nbr_dists, const int32_t *values,
                       const int64_t *key_offsets, const int64_t *query_offsets, const float *p_lm,
                       int64_t B, int64_t V, int64_t S, int32_t r, float mu, float alpha, float tau,
                       float *lambda_out, float *p_m, void *stream);

/*
 * knn_stream_read -- a measurement aid, not a step of the method: one plain
 * read of `bytes` bytes of device memory at `buf` (16-byte aligned, a multiple
 * of 16 bytes) with the same 16-byte non-temporal loads the distance stage
 * streams keys with, by 2048 workgroups each reading one contiguous piece.  Its duration is
 * the HBM read ceiling the distance stage's key streaming is compared with.
 * `sink` is a device word that is written only with negligible probability
 * (it keeps the loads from being optimised away).
 */
knn_status knn_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *stream);

/* Static text for a status code. */
const char *knn_status_string(knn_status status);

/* KNNLM_ABI_VERSION of the loaded library. */
int knn_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KNNLM_H */
