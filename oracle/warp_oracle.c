/*
 * Plain CPU oracle of the WARP search path. TEST INFRASTRUCTURE ONLY: only the
 * tests, the smoke check and the benchmark's CPU-baseline leg may load it.
 *
 * Each function follows one passage of the paper (WARP, SIGIR '25):
 *   oracle_centroid_scores  Section 4.3, S_{c,q} = C q^T
 *   oracle_select           Section 4.3, top-n_probe centroids and WARP_SELECT's
 *                           missing-similarity estimate from cumulative cluster sizes
 *   lut / token score       Section 4.4, Eq. warp_selective_sum and the table
 *                           upsilon = q_hat x omega_hat
 *   search                  Section 4.5, token-level max (r_tok) and document-level
 *                           sum with imputation (r_doc, Eq. doc_level_reduce), then
 *                           top-k; scores follow Eq. 1 without the 1/Z factor.
 *
 * Written to be read, not to be fast: full sorts, dense per-query arrays, one
 * embedding at a time. Parallel over queries, or over the tokens of one query
 * when there are fewer queries than threads (each token owns its rows).
 */
#include "warp_oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

#define ABSENT INT64_MIN

/* R(x): x in fixed point with ORACLE_FRAC_BITS fraction bits, round half to even. */
static int64_t fixed(double x) { return (int64_t)nearbyint(ldexp(x, ORACLE_FRAC_BITS)); }

/* Packed b-bit code of dimension d of one embedding's code row, most significant bits first. */
static int code_at(const uint8_t* row, int32_t nbits, int32_t d) {
    int per_byte = 8 / nbits;
    int byte = row[d / per_byte];
    int shift = 8 - nbits * (d % per_byte + 1);
    return (byte >> shift) & ((1 << nbits) - 1);
}

void oracle_centroid_scores(const float* centroids, int32_t n_c, int32_t dim, const float* q,
                            double* out) {
    for (int32_t c = 0; c < n_c; ++c) {
        double s = 0.0;
        for (int32_t d = 0; d < dim; ++d) s += (double)centroids[(int64_t)c * dim + d] * (double)q[d];
        out[c] = s;
    }
}

typedef struct {
    double s;
    int32_t id;
} scored_centroid;

/* centroid order: higher score first, lower id first among equal scores */
static int by_score_desc(const void* a, const void* b) {
    const scored_centroid* x = (const scored_centroid*)a;
    const scored_centroid* y = (const scored_centroid*)b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->id > y->id) - (x->id < y->id);
}

void oracle_select(const double* scores, const int64_t* offsets, int32_t n_c, int32_t nprobe,
                   int64_t t_prime, int32_t* sel, double* m) {
    scored_centroid* order = (scored_centroid*)malloc(sizeof(scored_centroid) * (size_t)n_c);
    for (int32_t c = 0; c < n_c; ++c) {
        order[c].s = scores[c];
        order[c].id = c;
    }
    qsort(order, (size_t)n_c, sizeof(scored_centroid), by_score_desc);
    for (int32_t j = 0; j < nprobe; ++j) sel[j] = order[j].id;
    /* first position whose inclusive cumulative size exceeds t'; the last one if none does */
    int32_t p_star = n_c - 1;
    int64_t cum = 0;
    for (int32_t p = 0; p < n_c; ++p) {
        int32_t c = order[p].id;
        cum += offsets[c + 1] - offsets[c];
        if (cum > t_prime) {
            p_star = p;
            break;
        }
    }
    *m = order[p_star].s;
    free(order);
}

/* Q(x) = round-half-even(x * 2^22): query values and bucket weights quantised to
 * 2^-22 before they are multiplied */
static int64_t quant(double x) { return (int64_t)nearbyint(ldexp(x, ORACLE_PROD_BITS)); }

/* upsilon[d][beta] = Q(q_d) * Q(omega_beta): the per-token bucket-weight table, as
 * exact integers in units of 2^-44 */
static void build_lut(const float* q, int32_t dim, const float* w, int32_t nbits, int64_t* lut) {
    int nb = 1 << nbits;
    for (int32_t d = 0; d < dim; ++d)
        for (int b = 0; b < nb; ++b) lut[d * nb + b] = quant((double)q[d]) * quant((double)w[b]);
}

/* selective sum: one table entry per dimension, summed exactly, then rounded once to
 * the 2^-26 grid (halves upward) and added to the centroid term */
static int64_t token_score(const int64_t* lut, int32_t dim, int32_t nbits, int64_t centroid_term,
                           const uint8_t* row) {
    int nb = 1 << nbits;
    int64_t v = 0;
    for (int32_t d = 0; d < dim; ++d) v += lut[d * nb + code_at(row, nbits, d)];
    /* |v| < 2^52, so v + 2^17 and its scaling by 2^-18 are exact in fp64, and
     * floor(x + 1/2) rounds x to the nearest integer, halves upward */
    const int shift = 2 * ORACLE_PROD_BITS - ORACLE_FRAC_BITS;
    return centroid_term + (int64_t)floor(ldexp((double)v + ldexp(1.0, shift - 1), -shift));
}

void oracle_token_scores(const float* q, int32_t dim, double centroid_score, const uint8_t* codes,
                         int32_t nbits, const float* bucket_weights, int64_t e0, int64_t e1,
                         int32_t* out) {
    int64_t* lut = (int64_t*)malloc(sizeof(int64_t) * (size_t)dim << nbits);
    build_lut(q, dim, bucket_weights, nbits, lut);
    int64_t row_bytes = (int64_t)dim * nbits / 8;
    for (int64_t e = e0; e < e1; ++e)
        out[e - e0] = (int32_t)token_score(lut, dim, nbits, fixed(centroid_score), codes + e * row_bytes);
    free(lut);
}

typedef struct {
    int64_t score;
    int32_t doc;
} scored_doc;

/* result order: higher score first, lower document id first among equal scores */
static int by_doc_score_desc(const void* a, const void* b) {
    const scored_doc* x = (const scored_doc*)a;
    const scored_doc* y = (const scored_doc*)b;
    if (x->score > y->score) return -1;
    if (x->score < y->score) return 1;
    return (x->doc > y->doc) - (x->doc < y->doc);
}

typedef struct {
    const float* centroids;
    int32_t n_c, dim;
    const int64_t* offsets;
    const int32_t* doc_ids;
    const uint8_t* codes;
    int32_t nbits;
    const float* w;
    int32_t n_docs;
    int32_t n_qtok, nprobe, k, flags;
    int64_t t_prime;
    const int32_t* doc_len; /* only with ORACLE_EQ1_LITERAL */
    int32_t token_threads;  /* > 1: the tokens of one query are processed in parallel */
} search_args;

static void search_one(const search_args* a, const float* query, int32_t* out_ids, int64_t* out_fixed,
                       float* out_scores, int32_t* out_count, int32_t* sel, int64_t* m_fixed,
                       uint32_t* cand_bitmap, int64_t* n_scored, int64_t* doc_fixed) {
    const int32_t T = a->n_qtok, D = a->dim, P = a->nprobe, n_docs = a->n_docs;
    const int64_t row_bytes = (int64_t)D * a->nbits / 8;
    int32_t* my_sel = (int32_t*)malloc(sizeof(int32_t) * (size_t)T * P);
    int64_t* M = (int64_t*)malloc(sizeof(int64_t) * (size_t)T);
    /* best[i][doc]: token-level max over every retrieved embedding of doc for token i */
    int64_t* best = (int64_t*)malloc(sizeof(int64_t) * (size_t)T * n_docs);
    int32_t* seen = NULL; /* retrieved embeddings per (token, doc), Eq.-1-literal reading only */
    if (a->flags & ORACLE_EQ1_LITERAL) seen = (int32_t*)calloc((size_t)T * n_docs, sizeof(int32_t));
    for (int64_t x = 0; x < (int64_t)T * n_docs; ++x) best[x] = ABSENT;
    int64_t scored = 0;

#pragma omp parallel for schedule(dynamic, 1) reduction(+ : scored) if (a->token_threads > 1) \
    num_threads(a->token_threads > 1 ? a->token_threads : 1)
    for (int32_t i = 0; i < T; ++i) {
        const float* q = query + (int64_t)i * D;
        double* S = (double*)malloc(sizeof(double) * (size_t)a->n_c);
        int64_t* lut = (int64_t*)malloc(sizeof(int64_t) * (size_t)D << a->nbits);
        /* candidate generation: centroid scores, n_probe best, missing similarity */
        double m;
        oracle_centroid_scores(a->centroids, a->n_c, D, q, S);
        oracle_select(S, a->offsets, a->n_c, P, a->t_prime, my_sel + (int64_t)i * P, &m);
        M[i] = fixed(m);
        /* decompression: selective sum over every embedding of every probed cluster */
        build_lut(q, D, a->w, a->nbits, lut);
        int64_t min_retrieved = INT64_MAX;
        for (int32_t j = 0; j < P; ++j) {
            int32_t c = my_sel[(int64_t)i * P + j];
            int64_t centroid_term = fixed(S[c]);
            for (int64_t e = a->offsets[c]; e < a->offsets[c + 1]; ++e) {
                int64_t t = token_score(lut, D, a->nbits, centroid_term, a->codes + e * row_bytes);
                int32_t doc = a->doc_ids[e];
                int64_t* cell = &best[(int64_t)i * n_docs + doc];
                if (*cell == ABSENT || t > *cell) *cell = t; /* r_tok */
                if (seen) seen[(int64_t)i * n_docs + doc] += 1;
                if (t < min_retrieved) min_retrieved = t;
                ++scored;
            }
        }
        if (a->flags & ORACLE_M_MIN_RETRIEVED) M[i] = (min_retrieved == INT64_MAX) ? 0 : min_retrieved;
        free(lut);
        free(S);
    }

    /* document-level reduction over the candidate set (docs with any retrieved token) */
    scored_doc* cand = (scored_doc*)malloc(sizeof(scored_doc) * (size_t)(n_docs > 0 ? n_docs : 1));
    int32_t n_cand = 0;
    for (int32_t doc = 0; doc < n_docs; ++doc) {
        int any = 0;
        for (int32_t i = 0; i < T; ++i) any |= best[(int64_t)i * n_docs + doc] != ABSENT;
        if (doc_fixed) doc_fixed[doc] = ABSENT;
        if (!any) continue;
        int64_t score = 0;
        for (int32_t i = 0; i < T; ++i) {
            int64_t v = best[(int64_t)i * n_docs + doc];
            if (v == ABSENT) {
                score += M[i]; /* r_doc: a missing entry takes the token's estimate */
            } else if (seen && seen[(int64_t)i * n_docs + doc] < a->doc_len[doc]) {
                score += v > M[i] ? v : M[i]; /* Eq. 1 literal: an unretrieved doc token contributes m_i */
            } else {
                score += v;
            }
        }
        if (doc_fixed) doc_fixed[doc] = score;
        if (cand_bitmap) cand_bitmap[doc >> 5] |= 1u << (doc & 31);
        cand[n_cand].score = score;
        cand[n_cand].doc = doc;
        ++n_cand;
    }
    qsort(cand, (size_t)n_cand, sizeof(scored_doc), by_doc_score_desc);
    int32_t n_out = n_cand < a->k ? n_cand : a->k;
    for (int32_t r = 0; r < a->k; ++r) {
        if (r < n_out) {
            out_ids[r] = cand[r].doc;
            out_fixed[r] = cand[r].score;
            out_scores[r] = (float)ldexp((double)cand[r].score, -ORACLE_FRAC_BITS);
        } else {
            out_ids[r] = -1;
            out_fixed[r] = INT64_MIN;
            out_scores[r] = -INFINITY;
        }
    }
    *out_count = n_out;
    if (sel) memcpy(sel, my_sel, sizeof(int32_t) * (size_t)T * P);
    if (m_fixed) memcpy(m_fixed, M, sizeof(int64_t) * (size_t)T);
    if (n_scored) *n_scored = scored;
    free(cand);
    free(seen);
    free(best);
    free(M);
    free(my_sel);
}

int oracle_search(const float* centroids, int32_t n_c, int32_t dim, const int64_t* offsets,
                  const int32_t* doc_ids, const uint8_t* codes, int32_t nbits,
                  const float* bucket_weights, int32_t n_docs, const float* queries,
                  int32_t n_queries, int32_t n_qtok, int32_t nprobe, int64_t t_prime, int32_t k,
                  int32_t flags, int32_t* out_ids, int64_t* out_fixed, float* out_scores,
                  int32_t* out_counts, int32_t* sel, int64_t* m_fixed, uint32_t* cand_bitmap,
                  int64_t* n_scored, int64_t* doc_fixed, int32_t n_threads) {
    if (n_c < 1 || dim < 1 || n_docs < 0 || n_queries < 0 || n_qtok < 1 || nprobe < 1 ||
        nprobe > n_c || k < 1 || t_prime < 0)
        return -1;
    if (!(nbits == 1 || nbits == 2 || nbits == 4 || nbits == 8) || (dim * nbits) % 8 != 0) return -1;
    int32_t* doc_len = NULL;
    if (flags & ORACLE_EQ1_LITERAL) {
        doc_len = (int32_t*)calloc((size_t)(n_docs > 0 ? n_docs : 1), sizeof(int32_t));
        for (int64_t e = 0; e < offsets[n_c]; ++e) doc_len[doc_ids[e]] += 1;
    }
    if (n_threads <= 0) n_threads = omp_get_num_procs();
    /* fewer queries than threads: one query at a time, its tokens in parallel */
    const int32_t token_threads = n_queries < n_threads ? n_threads : 1;
    search_args a = {centroids, n_c,   dim,     offsets, doc_ids, codes,   nbits,   bucket_weights,
                     n_docs,    n_qtok, nprobe, k,       flags,   t_prime, doc_len, token_threads};
    int64_t words = ((int64_t)n_docs + 31) / 32;
    if (cand_bitmap) memset(cand_bitmap, 0, sizeof(uint32_t) * (size_t)(words * n_queries));
#pragma omp parallel for schedule(dynamic, 1) num_threads(token_threads > 1 ? 1 : n_threads)
    for (int32_t qi = 0; qi < n_queries; ++qi) {
        search_one(&a, queries + (int64_t)qi * n_qtok * dim, out_ids + (int64_t)qi * k,
                   out_fixed + (int64_t)qi * k, out_scores + (int64_t)qi * k, out_counts + qi,
                   sel ? sel + (int64_t)qi * n_qtok * nprobe : NULL,
                   m_fixed ? m_fixed + (int64_t)qi * n_qtok : NULL,
                   cand_bitmap ? cand_bitmap + qi * words : NULL, n_scored ? n_scored + qi : NULL,
                   doc_fixed ? doc_fixed + (int64_t)qi * n_docs : NULL);
    }
    free(doc_len);
    return 0;
}

/* ------------------------------------------------------------------ index construction (Section 4.1) */

static int32_t nearest(const float* C, int32_t n_c, const float* x) {
    int32_t best = 0;
    double bs = 0.0;
    for (int32_t c = 0; c < n_c; ++c) {
        double s = 0.0;
        for (int d = 0; d < ORACLE_DIM; ++d) s += (double)C[(int64_t)c * ORACLE_DIM + d] * (double)x[d];
        if (c == 0 || s > bs) {
            bs = s;
            best = c;
        }
    }
    return best;
}

static int by_float(const void* a, const void* b) {
    float x = *(const float*)a, y = *(const float*)b;
    return (x > y) - (x < y);
}

int oracle_build_index(const float* tokens, const int32_t* token_docs, int64_t n, const float* init,
                       int32_t n_c, const int64_t* sample, int64_t n_sample, int32_t iterations,
                       int32_t nbits, int64_t n_quant, float* centroids, int64_t* offsets,
                       int32_t* doc_ids, uint8_t* codes, float* weights, float* cutoffs,
                       int32_t* assign, int32_t n_threads) {
    const int D = ORACLE_DIM;
    if (n < 1 || n_c < 1 || n_sample < 1 || iterations < 0 || n_quant < 1 || n_quant > n) return -1;
    if (nbits != 1 && nbits != 2 && nbits != 4 && nbits != 8) return -1;
    if (n_threads > 0) omp_set_num_threads(n_threads);
    /* the starting centroids: the caller's starting vectors, normalised */
    for (int32_t c = 0; c < n_c; ++c) {
        double ss = 0.0;
        for (int d = 0; d < D; ++d) ss += (double)init[(int64_t)c * D + d] * (double)init[(int64_t)c * D + d];
        if (!(ss > 0.0) || !isfinite(ss)) return -1;
        double norm = sqrt(ss);
        for (int d = 0; d < D; ++d) centroids[(int64_t)c * D + d] = (float)((double)init[(int64_t)c * D + d] / norm);
    }

    /* k-means on the sample */
    int32_t* sa = (int32_t*)malloc(sizeof(int32_t) * (size_t)n_sample);
    int64_t* sums = (int64_t*)malloc(sizeof(int64_t) * (size_t)n_c * D);
    int64_t* cnt = (int64_t*)malloc(sizeof(int64_t) * (size_t)n_c);
    for (int32_t it = 0; it < iterations; ++it) {
#pragma omp parallel for schedule(dynamic, 64)
        for (int64_t i = 0; i < n_sample; ++i) sa[i] = nearest(centroids, n_c, tokens + sample[i] * D);
        memset(sums, 0, sizeof(int64_t) * (size_t)n_c * D);
        memset(cnt, 0, sizeof(int64_t) * (size_t)n_c);
        for (int64_t i = 0; i < n_sample; ++i) {
            const float* x = tokens + sample[i] * D;
            cnt[sa[i]] += 1;
            for (int d = 0; d < D; ++d) sums[(int64_t)sa[i] * D + d] += (int64_t)nearbyint(ldexp((double)x[d], 30));
        }
        for (int32_t c = 0; c < n_c; ++c) {
            if (cnt[c] == 0) continue;
            double ss = 0.0;
            for (int d = 0; d < D; ++d) ss += (double)sums[(int64_t)c * D + d] * (double)sums[(int64_t)c * D + d];
            if (!(ss > 0.0)) continue;
            double norm = sqrt(ss);
            for (int d = 0; d < D; ++d) centroids[(int64_t)c * D + d] = (float)((double)sums[(int64_t)c * D + d] / norm);
        }
    }
    free(sa);
    free(sums);
    free(cnt);

    /* every token to its nearest centroid */
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t t = 0; t < n; ++t) assign[t] = nearest(centroids, n_c, tokens + t * D);

    /* quantile buckets from the residual components of tokens [0, n_quant) */
    const int64_t m = n_quant * D;
    float* r = (float*)malloc(sizeof(float) * (size_t)m);
    for (int64_t t = 0; t < n_quant; ++t)
        for (int d = 0; d < D; ++d) r[t * D + d] = tokens[t * D + d] - centroids[(int64_t)assign[t] * D + d];
    qsort(r, (size_t)m, sizeof(float), by_float);
    const int nb = 1 << nbits;
    for (int j = 1; j < nb; ++j) {
        int64_t k = (m * j + nb - 1) / nb; /* ceil(m j / 2^b) */
        cutoffs[j - 1] = r[(k < 1 ? 1 : k) - 1];
    }
    for (int j = 0; j < nb; ++j) {
        int64_t k = (m * (2 * j + 1) + 2 * nb - 1) / (2 * nb); /* ceil(m (2j+1) / 2^(b+1)) */
        weights[j] = r[(k < 1 ? 1 : k) - 1];
    }
    free(r);

    /* grouping by cluster (stable) and codes */
    int64_t* cur = (int64_t*)calloc((size_t)n_c + 1, sizeof(int64_t));
    for (int64_t t = 0; t < n; ++t) cur[assign[t] + 1] += 1;
    for (int32_t c = 0; c < n_c; ++c) cur[c + 1] += cur[c];
    memcpy(offsets, cur, sizeof(int64_t) * ((size_t)n_c + 1));
    const int64_t row_bytes = (int64_t)D * nbits / 8;
    const int per_byte = 8 / nbits;
    for (int64_t t = 0; t < n; ++t) {
        int64_t p = cur[assign[t]]++;
        doc_ids[p] = token_docs[t];
        uint8_t* row = codes + p * row_bytes;
        memset(row, 0, (size_t)row_bytes);
        for (int d = 0; d < D; ++d) {
            float x = tokens[t * D + d] - centroids[(int64_t)assign[t] * D + d];
            int code = 0;
            for (int j = 0; j < nb - 1; ++j) code += cutoffs[j] <= x;
            row[d / per_byte] |= (uint8_t)(code << (8 - nbits * (d % per_byte + 1)));
        }
    }
    free(cur);
    return 0;
}
