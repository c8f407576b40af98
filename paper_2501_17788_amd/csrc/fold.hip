// Document-level reduction (Section 4.5, r_doc and Eq. doc_level_reduce):
//     score[d] = sum_i (tokmax[i][d] if retrieved, else R(m_i))       (int64, exact)
// over the candidate documents (at least one retrieved token). Every split of
// the token strides gives this sum, so one pass per document computes it.
//
// One thread per (query, document): the n_qtok token rows are read with coalesced
// non-temporal loads (nothing reads them again), all issued before the first is
// used. A cell at or above the query's threshold holds t plus the query's bias; a
// lower one (zeroed, or written by an earlier wave) is not retrieved (cell_code).
// With epochs the fold only reads; without, it zeroes every retrieved cell it read.
// The output is a sort key per document: ((score + 2^39) << 24) | (2^24 - 1 - doc),
// larger is better and equal scores order by lower document id; 0 marks a
// non-candidate.
#include "engine.h"

namespace warp {

__global__ __launch_bounds__(256) void k_fold(WaveArgs a) {
    const int q = blockIdx.y;
    const int64_t doc = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const bool in = doc < a.n_docs;
    bool any = false;
    uint64_t key = 0;
    if (in) {
        const int T = a.n_qtok;
        const int64_t nd = a.n_docs;
        uint32_t* col = a.tokmax + (int64_t)q * T * nd + doc;
        // R(m_i) of the query's tokens: wave-uniform, read through the scalar cache
        const auto* m = (const __attribute__((address_space(4))) int64_t*)(a.m_fixed + (int64_t)q * T);
        uint32_t* cnt = a.tokcnt ? a.tokcnt + (int64_t)q * T * nd + doc : nullptr;
        uint32_t ubias, vmin;
        cell_code(a, q, ubias, vmin);
        const int64_t bias = (int64_t)ubias;
        uint32_t v[kMaxQtok];
#pragma unroll
        for (int i = 0; i < kMaxQtok; ++i) v[i] = i < T ? __builtin_nontemporal_load(col + i * nd) : kTokAbsent;
        int64_t sum = 0;
        if (!cnt) {
#pragma unroll
            for (int i = 0; i < kMaxQtok; ++i) {
                if (i < T) {
                    any |= v[i] >= vmin;
                    sum += v[i] >= vmin ? (int64_t)v[i] - bias : m[i];
                }
            }
            if (!a.q_epoch) {
#pragma unroll
                for (int i = 0; i < kMaxQtok; ++i)
                    if (i < T && v[i] >= vmin) col[i * nd] = kTokAbsent;
            }
        } else {
            // Eq. 1 read literally: while some of the document's tokens were not retrieved
            // for this query token, the estimate m_i bounds it from below (cells are reset)
            const int32_t len = a.doc_len[doc];
            for (int i = 0; i < T; ++i) {
                const uint32_t n = cnt[i * nd];
                if (v[i] >= vmin) {
                    any = true;
                    int64_t t = (int64_t)v[i] - bias;
                    if ((int32_t)n < len && t < m[i]) t = m[i];
                    sum += t;
                    col[i * nd] = kTokAbsent;
                } else {
                    sum += m[i];
                }
                cnt[i * nd] = 0;
            }
        }
        key = any ? ((uint64_t)(sum + (1ll << 39)) << 24) | (uint64_t)(kMaxDocs - 1 - (int32_t)doc) : 0;
        a.keys[(int64_t)q * nd + doc] = key;
    }
    // candidate count and largest key of the block, for the top-k's histogram
    __shared__ unsigned long long s_max[4];
    __shared__ int s_cnt[4];
    unsigned long long kmax = key;
    for (int off = 32; off > 0; off >>= 1) {
        const unsigned long long o = __shfl_xor(kmax, off, 64);
        kmax = o > kmax ? o : kmax;
    }
    const int n_any = __popcll(__ballot(in && any));
    if ((threadIdx.x & 63) == 0) {
        s_max[threadIdx.x >> 6] = kmax;
        s_cnt[threadIdx.x >> 6] = n_any;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long m = 0;
        long long cnt = 0;
        for (int w = 0; w < 4; ++w) {
            m = s_max[w] > m ? s_max[w] : m;
            cnt += s_cnt[w];
        }
        uint64_t* part = a.qpart + 2 * ((int64_t)q * gridDim.x + blockIdx.x);
        part[0] = (uint64_t)cnt;
        part[1] = m;
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
