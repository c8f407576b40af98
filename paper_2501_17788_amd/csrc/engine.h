// Internal declarations shared by the engine's translation units: constants of
// the fixed-point contract, device-side layouts, and the host-side launchers
// each kernel file exports. Nothing here is part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace warp {

constexpr int kDim = 128;          // token embedding dimension
constexpr int kFrac = 26;          // fixed-point fraction bits of token and doc scores
constexpr int kMaxQtok = 32;       // query_maxlen
constexpr int kMaxProbe = 256;     // largest n_probe of the band selection; above, the sorting one
constexpr int kMaxK = 4096;        // largest k of the LDS top-k; above, every key is sorted
constexpr int kMaxDocs = 1 << 24;  // document ids packed into the low 24 bits of a sort key
constexpr int kTopkListCap = 4096;  // blocks of 256 documents the top-k's pruned passes can list
// A token-max cell holds t plus the bias of its query's epoch (an order-preserving bias, see
// cell_code); cells below the epoch's threshold hold no retrieved embedding of the wave. A
// zeroed cell holds kTokAbsent.
constexpr uint32_t kTokAbsent = 0;

// Centroid selection: the fp32 matrix-core scores are within kFilterEps of the
// fp64 scores; bins of the score histogram are wider than 2 * kFilterEps.
constexpr float kFilterEps = 1.0f / 8192.0f;
constexpr int kSelBins = 2048;
constexpr float kSelLim = 1.0625f;  // |score| <= (1 + 1e-3)^2 < kSelLim
constexpr int kSelCap = 1024;       // centroids near one selection boundary held in LDS
constexpr int kSplitTokens = 256;   // waves of at most this many tokens take the split selection
constexpr int kSplitSlice = 4096;   // fewest centroids per workgroup of the split selection
static_assert(2.0f * kSelLim / kSelBins > 2.0f * kFilterEps, "a bin must be wider than 2 eps");

// Histogram bin of a filter score: floor((f + kSelLim) * kSelBins / (2 kSelLim)),
// clamped. Monotone non-decreasing in f.
__device__ __forceinline__ int score_bin(float f) {
    const float scale = (float)kSelBins / (2.0f * kSelLim);
    int b = (int)floorf((f + kSelLim) * scale);
    return b < 0 ? 0 : (b >= kSelBins ? kSelBins - 1 : b);
}

// Residual scan on the matrix cores: a work item is (cluster, chunk of kMxChunk
// embeddings, group of up to kMxGroup probing tokens), run by kMxBlock threads.
constexpr int kMxChunk = 256;
constexpr int kMxGroup = 32;
constexpr int kMxBlock = 256;
// The persistent scan grid takes its items in batches of kScanBatch consecutive items:
// workgroup b starts with batch b, and every later batch comes from a device counter.
constexpr int kScanBatch = 4;
// In waves of at most kNarrowWave queries, chunks probed by at most kNarrowMax tokens (by
// default; WARP_NARROW_MAX) take the narrow scan (k_scan_narrow):
// one wave per chunk, with groups of kNrGroup tokens whose five digit classes are the rows
// of one matrix-core tile, so a 16-embedding tile of a group costs 6 int8 MFMAs instead of 18.
constexpr int kNarrowMax = 3;
constexpr int kNarrowWave = 16;  // waves of more queries send every chunk to the wide scan
constexpr int kNrGroup = 3;
constexpr int kQdigBytes = 3 * kDim;  // three base-256 digit planes of a query token
// Largest bucket weight magnitude: Q(omega) = round(omega * 2^22) must have three
// signed base-256 digits, i.e. lie in [-8421504, 8355711].
constexpr float kMaxWeight = 1.99f;
constexpr int kPlanBlock = 1024;  // threads of the work plan's kernels; chunks per block of its prefix sums
constexpr int kPairBlock = 8192;  // clusters per block of the pair offsets (8 per thread)
constexpr int kRecLenShift = 48;   // a chunk's length above its first embedding (< 2^40) in a list record

// Error bits the device reports through the index's flag word.
constexpr int kErrSelOverflow = 1;
constexpr int kErrSelNoCrossing = 2;
constexpr int kErrDocRange = 1 << 8;
constexpr int kErrQueryNorm = 1 << 9;

struct WaveArgs {
    // index
    const float* centroids;     // [n_c][128]
    const int64_t* offsets;     // [n_c + 1]
    const int32_t* sizes;       // [n_c]
    const int32_t* doc_ids;     // [N]
    const uint8_t* codes;       // [N][16 * nbits]
    const float* weights;       // [2^nbits]
    int32_t n_c, n_docs, nbits;
    // wave of queries
    const float* queries;       // [n_tok][128], n_tok = n_q * n_qtok
    int32_t n_q, n_qtok, nprobe, k;
    int64_t t_prime;
    // scratch
    uint16_t* filter_bins;      // [n_tok][n_c] histogram bin of each filter score
    int32_t* sel;               // [n_tok][nprobe]
    int32_t* base;              // [n_tok][nprobe]  R(S64) of the probed centroids
    int64_t* seg_pref;          // [n_tok][nprobe + 1] cumulative probed sizes
    int64_t* m_fixed;           // [n_tok]
    uint32_t* tokmax;           // [n_tok][n_docs] biased token maxima
    const uint32_t* q_epoch;    // [n_q] epoch e >= 1 of each query's token-max rows; null: cells are reset
    int32_t tok_w;              // width w of a cell's value field (epochs in the bits above it)
    uint32_t* tokcnt;           // [n_tok][n_docs] retrieved embeddings per (token, doc); only for the
                                // Eq.-1-literal scoring, else null
    const int32_t* doc_len;     // [n_docs] embeddings per document (Eq.-1-literal scoring)
    uint64_t* keys;             // [n_q][n_docs]
    uint64_t* qpart;            // [n_q][ceil(n_docs / 256)][2]: candidate count and largest key of each fold block
    int32_t* err;               // device flag word
    // cluster-major pairing
    // split selection (sel_slices > 1 workgroups per token; see launch_select)
    unsigned long long* sel_hist;  // [n_tok][kSelBins] packed (count, size) histogram, zeroed per wave
    int32_t* sel_lists;         // [n_tok][2][kSelCap] centroids of the two rescoring bands
    int32_t* sel_cnt;           // [n_tok][2] their counts (may exceed kSelCap), zeroed per wave
    int32_t sel_slices;         // workgroups per token of the split selection; 1: one workgroup
    int32_t* ccount;            // [n_c] probing tokens per cluster
    int32_t* cursor;            // [n_c] scatter cursors
    int32_t* pair_start;        // [n_c] exclusive prefix of pairs within the cluster's block of
                                // kPairBlock clusters; the cluster's first pair is this plus coff
    int64_t* coff;              // [ceil(n_c / kPairBlock)] pairs of the blocks before each block
    int32_t* plist;             // [n_tok * nprobe][2]: (wave token, R(S64) + cell bias) grouped by cluster
    int8_t* qdig;               // [n_tok][kQdigBytes] query digit planes in operand order
    // The scan's items run over the probed chunks in the index's fixed pseudo-random chunk
    // order, the token groups of one chunk consecutively, so that the equal shares of the
    // persistent grid hold similar mixes of dense and sparse chunks of all clusters.
    const int32_t* chunk_c;     // [n_chunks] cluster of each chunk of the index, in that order
    const int32_t* chunk_k;     // [n_chunks] its chunk within the cluster
    int64_t n_chunks;
    int4* list_rec;             // [n_chunks] the probed chunks of the wave, in that order: first
                                // embedding (x, y: low and high words; the chunk's length in the
                                // top bits of y), first pair of the cluster (z), probing tokens (w)
    int64_t* list_item;         // [n_chunks + 1] exclusive prefix of their items; list_item[*list_n] = total
    int64_t* list_n;            // [1] number of probed chunks of the wide scan (more than narrow_max tokens)
    int4* list_rec2;            // [n_chunks] the probed chunks of the narrow scan (1..narrow_max tokens),
                                // in the same order, with records like list_rec
    int64_t* list_n2;           // [1] their number
    int64_t* cblk;              // [3 * ceil(n_chunks / kPlanBlock)] per block of chunks: wide chunks,
                                // their items and narrow chunks before it (block sums until the
                                // prefix kernel turns them into prefixes)
    uint32_t* scan_queue;       // [1] next unclaimed batch of the scan's items
    // outputs (device; the debug ones may be null)
    int32_t* out_ids;           // [n_q][k]
    float* out_scores;          // [n_q][k]
    int64_t* out_fixed;         // [n_q][k] or null
    int32_t* out_counts;        // [n_q] or null
    int32_t* dbg_sel;           // [n_q][n_qtok][nprobe] or null
    int64_t* dbg_m;             // [n_q][n_qtok] or null
    uint32_t* dbg_bitmap;       // [n_q][ceil(n_docs / 32)] or null
    int64_t* dbg_scored;        // [n_q] or null
    int32_t scan_grid;          // persistent workgroups of the residual scan
    int32_t narrow_max;         // chunks probed by 1..narrow_max tokens take the narrow scan
    int32_t topk_list_cap;      // at most kTopkListCap; the top-k visits every block when more pass
};

// Bias and threshold of the token-max cells of wave query q: with epochs, a cell holds
// t + e 2^w + 2^(w-1) and the query's retrieved cells are those at or above e 2^w, where
// 2^(w-1) exceeds every |t| the index admits; without, t + 2^31 and every nonzero cell,
// and the fold resets what it reads.
__device__ __forceinline__ void cell_code(const WaveArgs& a, int q, uint32_t& bias, uint32_t& vmin) {
    if (!a.q_epoch) {
        bias = 1u << 31;
        vmin = 1;
        return;
    }
    vmin = a.q_epoch[q] << a.tok_w;
    bias = vmin + (1u << (a.tok_w - 1));
}

// out_bins [n_tok][n_c] u16 bins (the search path) or, if null, out_scores fp32
void launch_filter_gemm(const float* q, int32_t n_tok, const float* c, int32_t n_c, uint16_t* out_bins,
                        float* out_scores, hipStream_t s);
void launch_select(const WaveArgs& a, hipStream_t s);
void launch_scored(const WaveArgs& a, hipStream_t s);
void launch_pairing(const WaveArgs& a, hipStream_t s);
void launch_wave_prep(const WaveArgs& a, uint32_t* ep, uint32_t last, hipStream_t s);
void launch_scan_mx(const WaveArgs& a, hipStream_t s);
int scan_mx_blocks_per_cu(int nbits);
void launch_scan_narrow(const WaveArgs& a, int32_t grid, hipStream_t s);
int scan_narrow_blocks_per_cu(int nbits);
void launch_fold(const WaveArgs& a, hipStream_t s);
void launch_topk(const WaveArgs& a, hipStream_t s);
// exact whole-list paths for n_probe > kMaxProbe and k > kMaxK (device radix sorts); the
// scratch holds the bytes the *_bytes functions give
size_t select_full_bytes(int64_t n_tok, int32_t n_c);
hipError_t launch_select_full(const WaveArgs& a, void* scratch, hipStream_t s);
size_t topk_full_bytes(int32_t n_docs);
hipError_t launch_topk_full(const WaveArgs& a, void* scratch, hipStream_t s);
void launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);
void launch_zero_cells(uint32_t* p, int64_t n, hipStream_t s);  // streaming stores
void launch_check_docs(const int32_t* ids, int64_t n, int32_t n_docs, int32_t* err, hipStream_t s);
void launch_check_queries(const float* q, int64_t n_tok, int32_t* err, hipStream_t s);
void launch_doc_len(const int32_t* doc_ids, int64_t n, int32_t* doc_len, int32_t n_docs, hipStream_t s);

// index construction
constexpr int kErrArgOverflow = 1 << 10;  // more than kArgCap centroids in one token's argmax band
void launch_rows_argmax(const float* scores, int64_t n, int32_t n_c, const float* x, const float* cen,
                        int32_t* assign, int32_t* err, hipStream_t s);
void launch_gather_rows(const float* x, const int64_t* ids, int64_t n, float* out, hipStream_t s);
void launch_kmeans_accum(const float* xs, const int32_t* assign, int64_t n, unsigned long long* sums,
                         unsigned long long* counts, hipStream_t s);
void launch_kmeans_normalize(const unsigned long long* sums, const unsigned long long* counts, int32_t n_c,
                             float* cen, hipStream_t s);
void launch_normalize_rows(float* rows, int32_t n, hipStream_t s);
void launch_residuals(const float* x, const int32_t* assign, int64_t n, const float* cen, float* out,
                      hipStream_t s);
void launch_pick_quantiles(const float* sorted, int64_t n, int32_t nbits, float* cutoffs, float* weights,
                           hipStream_t s);
void launch_encode(int32_t nbits, const float* x, const int32_t* token_docs, const int32_t* assign,
                   const int64_t* perm, int64_t n, const float* cen, const float* cutoffs, uint8_t* codes,
                   int32_t* doc_ids, hipStream_t s);
void launch_count_clusters(const int32_t* assign, int64_t n, unsigned long long* counts, hipStream_t s);
void launch_iota64(int64_t* out, int64_t n, hipStream_t s);
hipError_t sort_floats(void* temp, size_t* temp_bytes, const float* in, float* out, int64_t n, hipStream_t s);
hipError_t sort_by_cluster(void* temp, size_t* temp_bytes, const int32_t* keys_in, int32_t* keys_out,
                           const int64_t* vals_in, int64_t* vals_out, int64_t n, int end_bit, hipStream_t s);
hipError_t exclusive_sum_u64(void* temp, size_t* temp_bytes, const unsigned long long* in, int64_t* out,
                             int64_t n, hipStream_t s);

}  // namespace warp
