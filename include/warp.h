/*
 * warp.h - C ABI of the WARP multi-vector search engine for AMD Instinct MI355X
 * (gfx950).
 *
 * The engine implements the search path of WARP (Scheerer et al., SIGIR '25):
 *   1. WARP_SELECT (Section 4.3): query-token x centroid scores S = C q^T, the
 *      n_probe best centroids of every query token, and the missing-similarity
 *      estimate m_i = score of the first centroid, in score order, at which the
 *      cumulative cluster size exceeds t'.
 *   2. Implicit decompression (Section 4.4, Eq. warp_selective_sum): every
 *      embedding of every probed cluster is scored from its packed b-bit residual
 *      codes as S_{c,q_i} + sum_d upsilon_{i,d}[code_d], with the per-token table
 *      upsilon = q_hat x omega_hat.
 *   3. Two-stage reduction (Section 4.5): token-level max per (document, query
 *      token) (r_tok), then a document-level sum in which a missing entry takes
 *      m_i (r_doc, Eq. doc_level_reduce), then the top-k documents.
 *
 * Arithmetic. Centroid scores are computed in fp64 in dimension order; every
 * token score and document score is held in fixed point with
 * warp_fixed_point_bits() fraction bits (R(x) = round-half-even(x * 2^F)).
 * The table entries of Section 4.4 are exact products of query values and
 * bucket weights quantised to 2^-22 (Q(x) = round-half-even(x * 2^22)):
 *   token score  t = R(S_{c,q_i}) + floor(2^(F-44) * V + 1/2),
 *                V = sum_d Q(q_{i,d}) * Q(omega[code_d])                (int32)
 *   doc score    s = sum_i (max retrieved t, or R(m_i) if none)        (int64)
 * so every product, max and sum is exact and independent of the order of
 * evaluation.
 * The reported float score is (float)(s * 2^-F). Ties between documents are
 * broken by the lower document id; ties between centroids by the lower id.
 *
 * Index layout. Embeddings are grouped by cluster: cluster c owns embeddings
 * [cluster_offsets[c], cluster_offsets[c+1]). Each embedding has a document id
 * and dim * nbits / 8 code bytes; code bytes hold 8 / nbits dimensions each,
 * the first dimension in the most significant bits (for nbits = 4, dimension
 * 2j is bits 7..4 of byte j). Inside a cluster, embeddings should be ordered by
 * document id (results do not depend on it; throughput does).
 *
 * Errors. Every call returns WARP_OK or a negative code and never aborts. On an
 * error the outputs are unspecified and warp_last_error() describes the cause.
 *
 * Threads. Calls on one index are serialised by a lock inside the index.
 *
 * Scratch. An index grows device scratch on demand and keeps it until freed. A
 * search runs in waves of as many queries as the scratch budget holds: the value
 * of the environment variable WARP_SCRATCH_MB (MiB) if set, else 80% of the free
 * device memory. The dominant scratch is a [tokens][documents] table of token
 * maxima per wave, one slot of rows per query of the wave. Each wave tags its
 * cells with its slots' epochs, in the bits that the score range leaves spare
 * (the range follows from the bucket weights and the norm limits), so that cells
 * of earlier waves read as empty; a slot's rows are zeroed on the index's stream
 * when its epochs run out (every 7 to 15 waves that use it, for bucket weights
 * below about 0.2). With weights too large for a spare bit, and in the
 * Eq.-1-literal mode, the final reduction instead resets every cell it reads.
 *
 * Top-k. The final selection visits only the blocks of 256 documents whose best
 * score can reach the k-th, when at most WARP_TOPK_LIST_BLOCKS (default and
 * largest 4096; 0 turns this off) such blocks exist; results do not depend on it.
 *
 * Other tuning variables, none of which changes a result: WARP_MAX_SCRATCH_BYTES
 * caps an index's search scratch (a search that needs more fails with
 * WARP_ENOMEM); WARP_NARROW_MAX sets the most probing tokens of a cluster chunk
 * scored by the few-token scan (default 3 for waves of at most 16 queries, else
 * 0); WARP_SELECT_SLICES sets the workgroups per token of the centroid selection
 * (default: several per token for waves of at most 256 tokens, else one).
 */
#ifndef WARP_H
#define WARP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    WARP_OK = 0,
    WARP_EINVAL = -1,  /* an argument is out of range or inconsistent            */
    WARP_ENOMEM = -2,  /* device memory could not be allocated                   */
    WARP_EDEVICE = -3, /* no usable gfx950 device, or a HIP runtime call failed  */
    WARP_ENOTSUP = -4  /* a valid request this engine does not implement         */
};

typedef struct warp_index warp_index; /* opaque; owns all of its device memory */

/* Scoring modes (warp_set_scoring). */
enum {
    WARP_SCORING_PAPER = 0,      /* Section 4.5: a missing (token, document) entry takes m_i */
    WARP_SCORING_EQ1_LITERAL = 1 /* Eq. 1 read literally: a retrieved entry is also raised to m_i
                                    while some of the document's embeddings were not retrieved for
                                    that query token */
};

/* Number of fraction bits F of the fixed-point token and document scores (26). */
int warp_fixed_point_bits(void);

/* Thread-local description of the last non-OK return on this thread. */
const char* warp_last_error(void);

/*
 * The t' policy of Section 4.6 (hyperparameters): t' grows with the square root
 * of the number of indexed embeddings and is bounded by t'_max:
 *   *out = min(t_max, floor(c * sqrt(n_embeddings)))
 * The paper fixes neither c nor t_max; the caller passes both. Host-only, no
 * device call. WARP_EINVAL for a null out, n_embeddings < 0, c negative or not
 * finite, or t_max < 0.
 */
int warp_t_prime_policy(int64_t n_embeddings, double c, int64_t t_max, int64_t* out);

/*
 * The k-means sample size of Section 4.1 (index construction): the centroids
 * are trained on a sample of passages whose size grows with the square root of
 * the collection size:
 *   *out = min(n_passages, ceil(c * sqrt(n_passages)))
 * The paper fixes no constant; the caller passes c (ColBERTv2's recipe, which
 * the paper follows, uses 16). Which passages form the sample is the caller's
 * random draw. Host-only, no device call. WARP_EINVAL for a null out,
 * n_passages < 0, or c negative or not finite.
 */
int warp_kmeans_sample_size(int64_t n_passages, double c, int64_t* out);

/*
 * Build a device-resident index (Section 4.1's index: centroids, per-cluster
 * document ids and packed residual codes, bucket weights).
 *
 *   centroids        [n_centroids][dim] fp32, each row of unit norm (within 1e-3)
 *   n_centroids      >= 1
 *   dim              must be 128 (else WARP_ENOTSUP)
 *   cluster_offsets  [n_centroids + 1] int64: offsets[0] = 0, non-decreasing;
 *                    N = offsets[n_centroids] embeddings, N < 2^40
 *   doc_ids          [N] int32, 0 <= id < n_docs, grouped by cluster
 *   codes            [N][dim * nbits / 8] uint8, grouped by cluster
 *   nbits            1, 2, 4 or 8
 *   bucket_weights   [2^nbits] fp32, finite, |w| <= 1.99 (so that Q(w) has three
 *                    signed base-256 digits)
 *   n_docs           1 <= n_docs <= 2^24
 *   out              receives the index on WARP_OK; untouched otherwise
 *
 * warp_index_load reads host pointers; warp_index_load_device reads device
 * pointers (on the current device). Both copy: the caller keeps ownership of
 * its arrays and may free them once the call returns. Validation reads every
 * element (offsets, ids, weights, centroid norms) before anything is kept.
 */
int warp_index_load(const float* centroids, int32_t n_centroids, int32_t dim,
                    const int64_t* cluster_offsets, const int32_t* doc_ids, const uint8_t* codes,
                    int32_t nbits, const float* bucket_weights, int32_t n_docs, warp_index** out);
int warp_index_load_device(const float* centroids, int32_t n_centroids, int32_t dim,
                           const int64_t* cluster_offsets, const int32_t* doc_ids,
                           const uint8_t* codes, int32_t nbits, const float* bucket_weights,
                           int32_t n_docs, warp_index** out);

/* Free an index and all of its device memory. NULL is ignored. */
void warp_index_free(warp_index* idx);

/* Sizes of an index: any pointer may be NULL. */
int warp_index_info(const warp_index* idx, int32_t* n_centroids, int64_t* n_embeddings,
                    int32_t* n_docs, int32_t* nbits);

/*
 * Search a batch of queries (Section 4, the four retrieval steps after query
 * encoding).
 *
 *   queries      [n_queries][n_qtok][dim] fp32 host, each token of norm <= 1 + 1e-3
 *   n_queries    >= 1
 *   n_qtok       1..32 (query_maxlen = 32); every token takes part in the sum
 *   nprobe       1..n_centroids. Up to 256 the selection rescores only the
 *                centroids near its boundaries; above, it sorts every
 *                (token, centroid) score of a wave (same results, slower;
 *                WARP_ENOTSUP if n_qtok * n_centroids > 2^31)
 *   t_prime      >= 0, in embeddings
 *   k            >= 1. Up to 4096 the top-k gathers the best keys in LDS;
 *                above, it sorts every document key of a query (same results)
 *   out_doc_ids  [n_queries][k] caller-owned host; -1 past the result count
 *   out_scores   [n_queries][k] caller-owned host; -inf past the result count
 *   out_counts   [n_queries] host or NULL: min(k, number of candidate documents)
 *
 * Only candidate documents (those with at least one retrieved embedding) are
 * ranked. Blocks until the results are in host memory. If more than 1024
 * centroids of a token fall within about 3e-3 of a selection boundary (only
 * possible with degenerate centroid sets), the search is run again with the
 * selection that sorts every score, which gives the same results without that
 * limit.
 */
int warp_search(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok,
                int32_t nprobe, int64_t t_prime, int32_t k, int32_t* out_doc_ids,
                float* out_scores, int32_t* out_counts);

/*
 * As warp_search, with every pointer in device memory, enqueued on `hip_stream`
 * (a hipStream_t, NULL for the default stream); returns once the work is
 * enqueued. out_fixed_scores [n_queries][k] (int64, INT64_MIN padding) and
 * out_counts may be NULL. Query norms are checked on the device: that error,
 * and a centroid-selection overflow (more than 1024 centroids whose scores fall
 * within about 3e-3 of a selection boundary, only possible with degenerate
 * centroid sets: WARP_ENOTSUP; warp_search and warp_search_debug retry such a
 * search with the sorting selection), are reported by warp_index_sync. The index's scratch memory
 * is shared by its searches: enqueue the searches of one index on one stream.
 */
int warp_search_async(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok,
                      int32_t nprobe, int64_t t_prime, int32_t k, int32_t* out_doc_ids,
                      float* out_scores, int32_t* out_counts, int64_t* out_fixed_scores,
                      void* hip_stream);

/*
 * warp_search_async without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc). Same arguments, results and errors as
 * warp_search_async; every pointer is device memory and the work is enqueued on
 * `hip_stream`. It calls no hipMalloc or hipFree: all of its scratch lives in
 * one static device array of 256 MiB per GPU, held from the first index load on
 * that GPU until the process ends. A search takes waves of as many queries as
 * the array holds; if one query does not fit (roughly 4 * n_qtok * n_docs +
 * 2 * n_qtok * n_centroids + 8 * n_docs bytes, e.g. about 17 MB for 100k
 * documents, 1.1 GB for 8.8M; nprobe above 256 adds about 57 * n_qtok *
 * n_centroids bytes, k above 4096 about 25 * n_docs) it fails with WARP_ENOMEM
 * before enqueuing anything. Every call on a GPU shares that GPU's array, whichever index it
 * searches, and finds what the last call left there (the call clears what must
 * start at zero): calls that overlap on one GPU race, so enqueue them on one
 * stream or wait for each before the next. The index's own scratch is not
 * used, so this call and warp_search_async may alternate on an index.
 */
int warp_search_noalloc(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok,
                        int32_t nprobe, int64_t t_prime, int32_t k, int32_t* out_doc_ids,
                        float* out_scores, int32_t* out_counts, int64_t* out_fixed_scores,
                        void* hip_stream);

/* Wait for the index's outstanding work on `hip_stream` and report any deferred
 * device-side error. */
int warp_index_sync(warp_index* idx, void* hip_stream);

/*
 * warp_search plus intermediate results, all host memory (any may be NULL):
 *   out_fixed_scores [n_queries][k]                 int64 document scores (INT64_MIN padding)
 *   sel              [n_queries][n_qtok][nprobe]    probed centroids, in (score desc, id asc) order
 *   m_fixed          [n_queries][n_qtok]            R(m_i)
 *   cand_bitmap      [n_queries][ceil(n_docs/32)]   bit d%32 of word d/32: doc d is a candidate
 *   n_scored         [n_queries]                    embeddings scored (sum of probed cluster sizes)
 */
int warp_search_debug(warp_index* idx, const float* queries, int32_t n_queries, int32_t n_qtok,
                      int32_t nprobe, int64_t t_prime, int32_t k, int32_t* out_doc_ids,
                      float* out_scores, int32_t* out_counts, int64_t* out_fixed_scores,
                      int32_t* sel, int64_t* m_fixed, uint32_t* cand_bitmap, int64_t* n_scored);

/*
 * The fp32 matrix-core centroid scores that drive centroid selection, for
 * checking their error bound: out [n_tok][n_centroids] fp32 host, for host
 * queries [n_tok][dim]. Selection treats them as within 2^-13 of the fp64
 * scores and recomputes every centroid near a selection boundary in fp64.
 */
int warp_centroid_filter_scores(warp_index* idx, const float* queries, int32_t n_tok, float* out);

/*
 * Index construction on the device (Section 4.1): k-means on a sample of the
 * token embeddings, then every token encoded as a b-bit quantised residual to
 * its nearest centroid. Every pointer is device memory; the call blocks.
 *
 *   tokens           [n_tokens][128] fp32, finite, norm <= 1 + 1e-3
 *   token_docs       [n_tokens] document id of each token, in [0, n_docs)
 *   init_centroids   [n_centroids][128] fp32 starting vectors, finite and nonzero; each is
 *                    normalised (fp64 norm, sum of squares in dimension order) into a
 *                    starting centroid
 *   sample_ids       [n_sample] token ids (in [0, n_tokens)) used by k-means; Section
 *                    4.1 samples passages in proportion to the square root of the
 *                    collection size (the caller's choice)
 *   iterations       k-means steps (assign the sample, then recompute every centroid)
 *   n_quant          the residuals of tokens [0, n_quant) fit the quantile buckets
 * Outputs (caller-allocated, device):
 *   centroids        [n_centroids][128] fp32
 *   cluster_offsets  [n_centroids + 1]
 *   doc_ids          [n_tokens] and codes [n_tokens][16 * nbits]: the embeddings grouped by
 *                    cluster, in input order inside a cluster (the layout warp_index_load takes)
 *   bucket_weights   [2^nbits], bucket_cutoffs [2^nbits - 1] fp32
 *   assignment       [n_tokens] cluster of each input token, or null
 * Definitions (exact; the result does not depend on the order of evaluation):
 *   assignment = argmax_c S64(c, x), lowest id on ties (S64: fp64 dot product in
 *   dimension order); a k-means step replaces a centroid with a token by
 *   normalise(sum of round(x * 2^30)) (int64 sums, fp64 norm, rounded to fp32) and
 *   keeps a centroid without one; with r the fp32 residual components of the first
 *   n_quant tokens (n values), the cutoff j (1 <= j < 2^b) is the ceil(n j / 2^b)-th
 *   smallest and the weight j (0 <= j < 2^b) the ceil(n (2j + 1) / 2^(b+1))-th
 *   smallest; a code is the number of cutoffs <= the residual component.
 * WARP_EINVAL for an argument out of range, WARP_ENOTSUP if more than 1,024
 * centroids score within 2.5 * 2^-13 of a token's best, WARP_ENOMEM, WARP_EDEVICE.
 */
int warp_build_index(const float* tokens, const int32_t* token_docs, int64_t n_tokens, int32_t n_docs,
                     const float* init_centroids, int32_t n_centroids, const int64_t* sample_ids,
                     int64_t n_sample, int32_t iterations, int32_t nbits, int64_t n_quant, float* centroids,
                     int64_t* cluster_offsets, int32_t* doc_ids, uint8_t* codes, float* bucket_weights,
                     float* bucket_cutoffs, int32_t* assignment);

/*
 * Scoring of a (query token, document) entry (Section 4.5 versus Eq. 1).
 * WARP_SCORING_PAPER (the default) replaces only missing entries by m_i.
 * WARP_SCORING_EQ1_LITERAL reads Eq. 1 literally: a document with a retrieved
 * score v for query token i, but with some embeddings not retrieved for i (the
 * retrieved count is below the document's number of embeddings), takes
 * max(v, m_i). That mode keeps a second [tokens][documents] count table per wave
 * and more device atomics. Applies to later searches on the index.
 * WARP_EINVAL for an invalid handle or mode.
 */
int warp_set_scoring(warp_index* index, int32_t mode);

/*
 * Per-stage device time, measured with HIP events on the stream each search
 * runs on. warp_set_timing(idx, 1) starts recording and clears the totals;
 * warp_stage_timings returns, per stage, the summed milliseconds and the number
 * of launches since then, counting the searches completed by a synchronising
 * call (warp_search, warp_search_debug, warp_index_sync). Stages: [0] centroid
 * filter GEMM, [1] selection (with the wave's preparation before it: query
 * checks and digit planes, counters, and the zeroing of token-max rows whose
 * epochs ran out), [2] plan, [3] residual scan, [4] document fold, [5] top-k.
 */
int warp_set_timing(warp_index* idx, int32_t enable);
int warp_stage_timings(const warp_index* idx, double* total_ms, int64_t* launches, int32_t n);

#ifdef __cplusplus
}
#endif
#endif
