// Document-level reduction (Section 4.5, r_doc and Eq. doc_level_reduce):
//     score[d] = sum_i (tokmax[i][d] if retrieved, else R(m_i))       (int64, exact)
// over the candidate documents (at least one retrieved token). Every split of
// the token strides gives this sum, so one pass per document computes it.
//
// One thread per (query, document); the n_qtok token rows are read with
// coalesced loads and reset to kTokAbsent for the next wave. The output is a sort
// key per document: ((score + 2^39) << 24) | (2^24 - 1 - doc), larger is
// better and equal scores order by lower document id; 0 marks a non-candidate.
#include "engine.h"

namespace warp {

__global__ __launch_bounds__(256) void k_fold(WaveArgs a) {
    const int q = blockIdx.y;
    const int64_t doc = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const bool in = doc < a.n_docs;
    bool any = false;
    if (in) {
        int64_t sum = 0;
        const int T = a.n_qtok;
        uint32_t* col = a.tokmax + (int64_t)q * T * a.n_docs + doc;
        const int64_t* m = a.m_fixed + (int64_t)q * T;
        for (int i = 0; i < T; ++i) {
            const uint32_t v = col[(int64_t)i * a.n_docs];
            if (v != kTokAbsent) {
                any = true;
                sum += (int32_t)(v ^ 0x80000000u);
                col[(int64_t)i * a.n_docs] = kTokAbsent;
            } else {
                sum += m[i];
            }
        }
        const uint64_t key =
            any ? ((uint64_t)(sum + (1ll << 39)) << 24) | (uint64_t)(kMaxDocs - 1 - (int32_t)doc) : 0;
        a.keys[(int64_t)q * a.n_docs + doc] = key;
    }
    if (a.dbg_bitmap) {
        const unsigned long long bits = __ballot(in && any);
        const int lane = threadIdx.x & 63;
        const int64_t words = (a.n_docs + 31) / 32;
        const int64_t w0 = (doc - lane) / 32;  // first word of this wave (64 docs = 2 words)
        uint32_t* row = a.dbg_bitmap + (int64_t)q * words;
        if (lane == 0 && w0 < words) row[w0] = (uint32_t)bits;
        if (lane == 32 && w0 + 1 < words) row[w0 + 1] = (uint32_t)(bits >> 32);
    }
}

void launch_fold(const WaveArgs& a, hipStream_t s) {
    dim3 grid((a.n_docs + 255) / 256, a.n_q);
    hipLaunchKernelGGL(k_fold, grid, dim3(256), 0, s, a);
}

}  // namespace warp
