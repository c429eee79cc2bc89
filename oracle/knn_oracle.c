/*
 * CPU ORACLE for the kNN-LM mixture step -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, fp64 brute force of what the paper defines.  It is used by the
 * tests, by the smoke check and by the benchmark's CPU-baseline leg, and by
 * nothing else.  It shares no code, header, table or helper with the HIP
 * library; it is built with gcc from this one file.
 *
 * What it computes (paper, Section 2.2 "Nearest Neighbor Language Models",
 * paragraph "Probability interpolation", and Section 3.1 second-stage search):
 *
 *   1. s(q, k) = -||q - k||^2: the negative squared L2 distance, computed here
 *      directly as sum_j (q_j - k_j)^2 in fp64 from the stored element bytes
 *      widened to fp64 (eq. non-parametric and the sentence after it;
 *      Appendix A, where r = 1024 neighbours are retrieved by squared L2 distance).
 *   2. pi = the r keys of the query's own key set with the largest s, i.e. the
 *      smallest distance; equal distances are ordered by the lower key index
 *      (the paper does not say; this is the reading used throughout).
 *   3. p_kNN(w) proportional to sum over (k_i, v_i) in pi with v_i = w of
 *      exp(mu * s(q, k_i)), normalised over pi; tokens no neighbour carries get
 *      0 (eq. non-parametric).  The softmax is evaluated after subtracting the
 *      largest mu*s, which changes nothing mathematically.
 *   4. p_M = lambda * p_LM + (1 - lambda) * p_kNN (eq. kNN-LM), with p_LM the
 *      caller's fp32 row widened to fp64.
 *   5. Optionally a per-query lambda_t from relative retrieval confidence
 *      (Section 3.2, eq. rrc): sigmoid((min_i |s_i| / max_i |s_i| - alpha) / tau)
 *      over the query's r neighbours.
 *   6. Optionally a key mask (Section 3.4, last paragraph: the keys of an
 *      accepted span are never used again in that generation): a masked key
 *      is never a neighbour.  If fewer than r keys of a set are unmasked, the
 *      remaining slots of pi are absent (id -1, distance +infinity); an absent
 *      neighbour carries no weight and takes no part in the softmax or in
 *      lambda_t.
 *
 * Every function returns 0 on success and a negative code on a rejected
 * argument; nothing is printed.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F16 = 2 };

#define ORC_ERR_ARG (-1)
#define ORC_ERR_RANGE (-2)
#define ORC_ERR_NOMEM (-3)

/* ---- element widening -------------------------------------------------- */

static size_t elem_size(int dtype) {
    switch (dtype) {
    case ORC_F32: return 4;
    case ORC_BF16: return 2;
    case ORC_F16: return 2;
    default: return 0;
    }
}

/* bfloat16 is the upper half of an IEEE binary32 word. */
static double widen_bf16(uint16_t h) {
    uint32_t w = (uint32_t)h << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

/* IEEE binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
static double widen_f16(uint16_t h) {
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (expo == 0) {
        v = ldexp((double)frac, -24); /* subnormal: frac * 2^-14 * 2^-10 */
    } else if (expo == 31) {
        v = frac ? NAN : INFINITY;
    } else {
        v = ldexp(1.0 + (double)frac / 1024.0, expo - 15);
    }
    return sign ? -v : v;
}

static double widen(const void *base, int dtype, int64_t idx) {
    if (dtype == ORC_F32) {
        float f;
        memcpy(&f, (const char *)base + 4 * idx, 4);
        return (double)f;
    }
    uint16_t h;
    memcpy(&h, (const char *)base + 2 * idx, 2);
    return dtype == ORC_BF16 ? widen_bf16(h) : widen_f16(h);
}

/* Decode n stored elements to fp64 (exposed so tests can pin the decoding). */
int knn_oracle_widen(const void *src, int dtype, int64_t n, double *out) {
    if (!src || !out || n < 0 || elem_size(dtype) == 0) return ORC_ERR_ARG;
    for (int64_t i = 0; i < n; ++i) out[i] = widen(src, dtype, i);
    return 0;
}

/* ---- step 1: direct squared distances ---------------------------------- */

typedef struct {
    const double *q;   /* [d] widened query */
    const void *keys;  /* key rows of one set */
    int dtype;
    int64_t d;
    int64_t k0, k1;    /* rows [k0, k1) of the set */
    double *out;       /* [n] distances of the set */
} dist_job;

static void *dist_worker(void *arg) {
    dist_job *job = (dist_job *)arg;
    for (int64_t i = job->k0; i < job->k1; ++i) {
        double acc = 0.0;
        for (int64_t j = 0; j < job->d; ++j) {
            double diff = job->q[j] - widen(job->keys, job->dtype, i * job->d + j);
            acc += diff * diff;
        }
        job->out[i] = acc;
    }
    return NULL;
}

/* Distances of one widened query to n key rows, split over nthreads threads
 * by contiguous key ranges (threads change no arithmetic). */
static int set_distances(const double *q, const void *keys, int dtype, int64_t n, int64_t d,
                         int nthreads, double *out) {
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    if (n < (int64_t)nthreads * 64) nthreads = 1;
    dist_job jobs[256];
    pthread_t tids[256];
    int started[256] = {0};
    int64_t per = (n + nthreads - 1) / nthreads;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t].q = q;
        jobs[t].keys = keys;
        jobs[t].dtype = dtype;
        jobs[t].d = d;
        jobs[t].k0 = (int64_t)t * per < n ? (int64_t)t * per : n;
        jobs[t].k1 = jobs[t].k0 + per < n ? jobs[t].k0 + per : n;
        jobs[t].out = out;
    }
    for (int t = 1; t < nthreads; ++t) {
        started[t] = pthread_create(&tids[t], NULL, dist_worker, &jobs[t]) == 0;
        if (!started[t]) dist_worker(&jobs[t]); /* run inline if a thread cannot start */
    }
    dist_worker(&jobs[0]);
    for (int t = 1; t < nthreads; ++t)
        if (started[t]) pthread_join(tids[t], NULL);
    return 0;
}

/* All distances of nq queries to nk keys: out[i * nk + k] = ||q_i - k_k||^2. */
int knn_oracle_sqdist(const void *queries, const void *keys, int dtype, int64_t nq, int64_t nk,
                      int64_t d, int nthreads, double *out) {
    if (!queries || !keys || !out || nq < 0 || nk < 0 || d < 1 || elem_size(dtype) == 0)
        return ORC_ERR_ARG;
    double *q = (double *)malloc(sizeof(double) * (size_t)d);
    if (!q) return ORC_ERR_NOMEM;
    for (int64_t i = 0; i < nq; ++i) {
        for (int64_t j = 0; j < d; ++j) q[j] = widen(queries, dtype, i * d + j);
        set_distances(q, keys, dtype, nk, d, nthreads, out + i * nk);
    }
    free(q);
    return 0;
}

/* ---- step 2: the r nearest keys, ordered by (distance, index) ----------- */

typedef struct {
    double d;
    int64_t i;
} dist_idx;

static int by_dist_then_index(const void *a, const void *b) {
    const dist_idx *x = (const dist_idx *)a, *y = (const dist_idx *)b;
    if (x->d < y->d) return -1;
    if (x->d > y->d) return 1;
    return (x->i > y->i) - (x->i < y->i);
}

static int check_offsets(const int64_t *off, int64_t S, int64_t *total) {
    if (off[0] != 0) return 0;
    for (int64_t s = 0; s < S; ++s)
        if (off[s + 1] < off[s]) return 0;
    *total = off[S];
    return 1;
}

/*
 * For every query b (query set s owns rows query_offsets[s]..query_offsets[s+1]
 * of `queries` and key rows key_offsets[s]..key_offsets[s+1] of `keys`), write
 * the r local key indices with the smallest distance, ascending by
 * (distance, index), and their fp64 squared distances.  All arrays are host
 * memory.  Returns ORC_ERR_RANGE when a set with queries has fewer than r keys.
 *
 * key_mask (NULL: none) holds one bit per global key row, bit (i & 31) of
 * word i >> 5, 1 = masked: masked keys are left out, and slots pi cannot fill
 * from the unmasked keys get id -1 and distance +infinity.
 */
int knn_oracle_select_masked(const void *queries, const void *keys, int dtype, int64_t B, int64_t d,
                             const int64_t *key_offsets, const int64_t *query_offsets, int64_t S, int32_t r,
                             const uint32_t *key_mask, int nthreads, int32_t *out_ids, double *out_dists) {
    int64_t total_keys, total_q;
    if (!queries || !keys || !key_offsets || !query_offsets || !out_ids || !out_dists) return ORC_ERR_ARG;
    if (B < 0 || d < 1 || S < 1 || r < 1 || elem_size(dtype) == 0) return ORC_ERR_ARG;
    if (!check_offsets(key_offsets, S, &total_keys) || !check_offsets(query_offsets, S, &total_q) ||
        total_q != B)
        return ORC_ERR_ARG;
    int64_t nmax = 0;
    for (int64_t s = 0; s < S; ++s) {
        int64_t n = key_offsets[s + 1] - key_offsets[s];
        if (query_offsets[s + 1] > query_offsets[s] && n < r) return ORC_ERR_RANGE;
        if (n > nmax) nmax = n;
    }
    double *q = (double *)malloc(sizeof(double) * (size_t)d);
    double *dist = (double *)malloc(sizeof(double) * (size_t)(nmax > 0 ? nmax : 1));
    dist_idx *order = (dist_idx *)malloc(sizeof(dist_idx) * (size_t)(nmax > 0 ? nmax : 1));
    if (!q || !dist || !order) {
        free(q); free(dist); free(order);
        return ORC_ERR_NOMEM;
    }
    size_t esz = elem_size(dtype);
    for (int64_t s = 0; s < S; ++s) {
        int64_t n = key_offsets[s + 1] - key_offsets[s];
        const void *set_keys = (const char *)keys + (size_t)key_offsets[s] * (size_t)d * esz;
        for (int64_t b = query_offsets[s]; b < query_offsets[s + 1]; ++b) {
            for (int64_t j = 0; j < d; ++j) q[j] = widen(queries, dtype, b * d + j);
            set_distances(q, set_keys, dtype, n, d, nthreads, dist);
            for (int64_t i = 0; i < n; ++i) {
                order[i].d = dist[i];
                order[i].i = i;
            }
            int64_t kept = 0;  /* the unmasked keys, in index order */
            for (int64_t i = 0; i < n; ++i) {
                const int64_t g = key_offsets[s] + i;
                if (key_mask && ((key_mask[g >> 5] >> (g & 31)) & 1u)) continue;
                order[kept].d = dist[i];
                order[kept].i = i;
                ++kept;
            }
            qsort(order, (size_t)kept, sizeof(dist_idx), by_dist_then_index);
            for (int32_t j = 0; j < r; ++j) {
                out_ids[b * r + j] = j < kept ? (int32_t)order[j].i : -1;
                out_dists[b * r + j] = j < kept ? order[j].d : INFINITY;
            }
        }
    }
    free(q); free(dist); free(order);
    return 0;
}

int knn_oracle_select(const void *queries, const void *keys, int dtype, int64_t B, int64_t d,
                      const int64_t *key_offsets, const int64_t *query_offsets, int64_t S, int32_t r,
                      int nthreads, int32_t *out_ids, double *out_dists) {
    return knn_oracle_select_masked(queries, keys, dtype, B, d, key_offsets, query_offsets, S, r, NULL, nthreads,
                                    out_ids, out_dists);
}

/* ---- steps 3-4: p_kNN over pi and the lambda mixture -------------------- */

/*
 * Given, per query, r neighbour local ids with fp64 squared distances (any
 * order), form p_kNN by a softmax over mu * s = -mu * dist scattered onto the
 * neighbours' value tokens (duplicates accumulate), then
 * p_M = lambda * p_LM + (1 - lambda) * p_kNN.  out_pknn may be NULL.
 * An id of -1 is an absent neighbour (a slot a masked select could not fill):
 * it carries no weight and takes no part in the softmax; with no neighbour
 * present p_kNN is 0.  Returns ORC_ERR_RANGE for any other id outside its set
 * or a value outside [0, V).
 */
/* The mixture with a per-query weight of p_LM: lambdas[b] for query b. */
int knn_oracle_mix_lambdas(const int32_t *ids, const double *dists, const int32_t *values,
                           const int64_t *key_offsets, const int64_t *query_offsets, int64_t S, int64_t B,
                           int32_t r, const float *p_lm, int64_t V, double mu, const double *lambdas,
                           double *out_pm, double *out_pknn) {
    int64_t total_keys, total_q;
    if (!ids || !dists || !values || !key_offsets || !query_offsets || !p_lm || !lambdas || !out_pm)
        return ORC_ERR_ARG;
    if (S < 1 || B < 0 || r < 1 || V < 1 || !(mu >= 0.0)) return ORC_ERR_ARG;
    for (int64_t b = 0; b < B; ++b)
        if (!(lambdas[b] >= 0.0 && lambdas[b] <= 1.0)) return ORC_ERR_ARG;
    if (!check_offsets(key_offsets, S, &total_keys) || !check_offsets(query_offsets, S, &total_q) ||
        total_q != B)
        return ORC_ERR_ARG;
    double *pknn = (double *)malloc(sizeof(double) * (size_t)V);
    double *w = (double *)malloc(sizeof(double) * (size_t)r);
    if (!pknn || !w) {
        free(pknn); free(w);
        return ORC_ERR_NOMEM;
    }
    int rc = 0;
    for (int64_t s = 0; s < S && rc == 0; ++s) {
        int64_t n = key_offsets[s + 1] - key_offsets[s];
        for (int64_t b = query_offsets[s]; b < query_offsets[s + 1] && rc == 0; ++b) {
            const int32_t *id = ids + b * r;
            const double *dd = dists + b * r;
            const double lambda = lambdas[b];
            /* the largest mu*s over pi is -mu times the smallest distance */
            double dmin = INFINITY;
            for (int32_t j = 0; j < r; ++j)
                if (id[j] != -1 && dd[j] < dmin) dmin = dd[j];
            double z = 0.0;
            for (int32_t j = 0; j < r; ++j) {
                w[j] = id[j] == -1 ? 0.0 : exp(-mu * (dd[j] - dmin));
                z += w[j];
            }
            for (int64_t v = 0; v < V; ++v) pknn[v] = 0.0;
            for (int32_t j = 0; j < r; ++j) {
                if (id[j] == -1) continue;
                if (id[j] < 0 || id[j] >= n) { rc = ORC_ERR_RANGE; break; }
                int32_t tok = values[key_offsets[s] + id[j]];
                if (tok < 0 || tok >= V) { rc = ORC_ERR_RANGE; break; }
                pknn[tok] += w[j] / z;
            }
            for (int64_t v = 0; v < V; ++v) {
                out_pm[b * V + v] = lambda * (double)p_lm[b * V + v] + (1.0 - lambda) * pknn[v];
                if (out_pknn) out_pknn[b * V + v] = pknn[v];
            }
        }
    }
    free(pknn); free(w);
    return rc;
}

/* The mixture with one weight of p_LM for every query (eq. kNN-LM). */
int knn_oracle_mix(const int32_t *ids, const double *dists, const int32_t *values,
                   const int64_t *key_offsets, const int64_t *query_offsets, int64_t S, int64_t B,
                   int32_t r, const float *p_lm, int64_t V, double mu, double lambda, double *out_pm,
                   double *out_pknn) {
    if (!(lambda >= 0.0 && lambda <= 1.0) || B < 0) return ORC_ERR_ARG;
    double *lams = (double *)malloc(sizeof(double) * (size_t)(B > 0 ? B : 1));
    if (!lams) return ORC_ERR_NOMEM;
    for (int64_t b = 0; b < B; ++b) lams[b] = lambda;
    int rc = knn_oracle_mix_lambdas(ids, dists, values, key_offsets, query_offsets, S, B, r, p_lm, V, mu, lams,
                                    out_pm, out_pknn);
    free(lams);
    return rc;
}

/*
 * Relative retrieval confidence (Section 3.2, eq. rrc): for each query b, with
 * s_i = -dists[b * r + i] <= 0 over its r neighbours (any order),
 *   lambda_t = sigmoid((min_i |s_i| / max_i |s_i| - alpha) / tau).
 * |s_i| is the distance, so the ratio is the smallest over the largest
 * neighbour distance.  If every neighbour is at distance 0 the ratio is 0/0;
 * it is taken as 1 (the neighbours are all equally close).  tau > 0.  An
 * absent neighbour (distance +infinity, from a masked select) is left out;
 * with none present the ratio is taken as 1 as well.
 */
int knn_oracle_rrc_lambda(const double *dists, int64_t B, int32_t r, double alpha, double tau,
                          double *out_lambda) {
    if (!dists || !out_lambda || B < 0 || r < 1 || !(tau > 0.0) || !isfinite(alpha)) return ORC_ERR_ARG;
    for (int64_t b = 0; b < B; ++b) {
        double dmin = INFINITY, dmax = 0.0;
        for (int32_t j = 0; j < r; ++j) {
            double x = dists[b * r + j];
            if (isinf(x) && x > 0.0) continue;
            if (x < dmin) dmin = x;
            if (x > dmax) dmax = x;
        }
        if (dmin < 0.0 || isnan(dmin) || isnan(dmax)) return ORC_ERR_RANGE;
        double ratio = dmax > 0.0 ? dmin / dmax : 1.0;
        out_lambda[b] = 1.0 / (1.0 + exp(-(ratio - alpha) / tau));
    }
    return 0;
}

int knn_oracle_version(void) { return 1; }
