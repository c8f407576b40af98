/*
 * Plain CPU oracle of the WARP search path (WARP_SELECT, implicit
 * decompression, two-stage reduction, top-k).
 *
 * TEST INFRASTRUCTURE ONLY. This code exists to check the HIP engine. Only the
 * tests, the smoke check and the CPU-baseline leg of the benchmark may load it;
 * the engine never calls it and shares no code, header or table with it.
 *
 * Arithmetic (the paper does not fix one; this is the canonical reading):
 *   - centroid score S64 = sum_d (double)C[c][d] * (double)q[d], accumulated in
 *     fp64 in increasing d order (each fp32 x fp32 product is exact in fp64);
 *   - R(x) = round-half-even(x * 2^26) in fp64, converted to an integer;
 *   - Q(x) = round-half-even(x * 2^22): query values and bucket weights quantised
 *     to 2^-22; the selective sum V = sum_d Q(q[d]) * Q(w[code_d]) is an exact
 *     integer in units of 2^-44 (|V| < 2^53);
 *   - token score t = R(S64) + floor(V * 2^-18 + 1/2) (int32, units of 2^-26): the
 *     residual term is rounded to nearest with halves upward;
 *   - document score = sum over query tokens of (token max, else R(m_i)) (int64);
 *   - reported score = (float)(score * 2^-26).
 */
#ifndef WARP_ORACLE_H
#define WARP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORACLE_FRAC_BITS 26
#define ORACLE_DIM 128  /* token dimension of the index construction */
#define ORACLE_PROD_BITS 22

/* flags for oracle_search */
#define ORACLE_EQ1_LITERAL     1  /* Eq. 1 read literally: max(m_i, retrieved) when some doc token is unretrieved */
#define ORACLE_M_MIN_RETRIEVED 2  /* m_i = smallest retrieved token score of q_i (XTR's estimate) instead of t' */

/* Section 4.3: S_{c,q} = C q^T for one query token, all centroids. out[n_c]. */
void oracle_centroid_scores(const float* centroids, int32_t n_c, int32_t dim,
                            const float* q, double* out);

/* Section 4.3 (WARP_SELECT): the nprobe best centroids of one token, ordered by
 * (score desc, id asc), and the missing-similarity estimate m (score of the
 * first centroid in that order whose inclusive cumulative size exceeds t').
 * sel[nprobe]; *m receives m. */
void oracle_select(const double* scores, const int64_t* offsets, int32_t n_c,
                   int32_t nprobe, int64_t t_prime, int32_t* sel, double* m);

/* Eq. warp_selective_sum: fixed-point token scores of the embeddings
 * [e0, e1) against one query token whose centroid score for their cluster is
 * `centroid_score`. out[e1 - e0]. */
void oracle_token_scores(const float* q, int32_t dim, double centroid_score,
                         const uint8_t* codes, int32_t nbits, const float* bucket_weights,
                         int64_t e0, int64_t e1, int32_t* out);

/* Whole search. Returns 0 on success, -1 on a bad argument.
 *   out_ids [n_queries][k] (pad -1), out_fixed [n_queries][k] (pad INT64_MIN),
 *   out_scores [n_queries][k] (pad -inf), out_counts [n_queries];
 * debug outputs may be NULL:
 *   sel [n_queries][n_qtok][nprobe], m_fixed [n_queries][n_qtok],
 *   cand_bitmap [n_queries][ceil(n_docs/32)], n_scored [n_queries],
 *   doc_fixed [n_queries][n_docs] (document scores, INT64_MIN for non-candidates).
 * n_threads <= 0 means one thread per online CPU. */
int oracle_search(const float* centroids, int32_t n_c, int32_t dim,
                  const int64_t* offsets, const int32_t* doc_ids, const uint8_t* codes,
                  int32_t nbits, const float* bucket_weights, int32_t n_docs,
                  const float* queries, int32_t n_queries, int32_t n_qtok,
                  int32_t nprobe, int64_t t_prime, int32_t k, int32_t flags,
                  int32_t* out_ids, int64_t* out_fixed, float* out_scores, int32_t* out_counts,
                  int32_t* sel, int64_t* m_fixed, uint32_t* cand_bitmap, int64_t* n_scored,
                  int64_t* doc_fixed, int32_t n_threads);

/* Section 4.1 (index construction), written out plainly:
 *   start       = every starting vector init[c] normalised: (float)(init[c][d] / ||init[c]||), the
 *                 norm in fp64 (sum of squares in dimension order, IEEE sqrt); rows must be
 *                 finite and nonzero;
 *   assign(x)   = argmax_c sum_d (double)C[c][d] * (double)x[d] (dimension order), lowest c on ties;
 *   k-means     = `iterations` times: assign the sample tokens, then replace every centroid that
 *                 has tokens by normalise(sum over them of round(x * 2^30)) (int64 sums, fp64
 *                 norm in dimension order, rounded to fp32);
 *   quantiles   = of the n fp32 residual components x - C[assign(x)] of tokens [0, n_quant):
 *                 cutoff j (1 <= j < 2^b) = ceil(n j / 2^b)-th smallest,
 *                 weight j (0 <= j < 2^b) = ceil(n (2j+1) / 2^(b+1))-th smallest;
 *   codes       = per dimension the number of cutoffs <= the residual component, packed with the
 *                 first dimension in the most significant bits;
 *   layout      = embeddings grouped by cluster (offsets), input order inside a cluster.
 * Outputs: centroids [n_c][128], offsets [n_c+1], doc_ids [n], codes [n][16b], weights [2^b],
 * cutoffs [2^b - 1], assign [n]. Returns 0, or -1 on a bad argument. */
int oracle_build_index(const float* tokens, const int32_t* token_docs, int64_t n, const float* init,
                       int32_t n_c, const int64_t* sample, int64_t n_sample, int32_t iterations,
                       int32_t nbits, int64_t n_quant, float* centroids, int64_t* offsets,
                       int32_t* doc_ids, uint8_t* codes, float* weights, float* cutoffs,
                       int32_t* assign, int32_t n_threads);

#ifdef __cplusplus
}
#endif
#endif
