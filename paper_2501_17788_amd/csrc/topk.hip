// Final top-k (Section 4.5: the k best candidate documents by score).
//
// One workgroup per query over its n_docs sort keys (fold kernel): keys are
// distinct, so the K-th largest key (K = min(k, candidates)) is found exactly
// by an MSB-first radix select, 8 bits per pass, with an LDS histogram of the
// keys that match the digits fixed so far. The K keys >= that key are gathered
// and sorted in LDS; each decodes to (document id, fixed-point score).
#include "engine.h"

namespace warp {

constexpr int kTopkThreads = 1024;

__global__ __launch_bounds__(kTopkThreads) void k_topk(WaveArgs a) {
    __shared__ uint32_t hist[256];
    __shared__ unsigned long long buf[kMaxK];
    __shared__ unsigned long long s_prefix, s_mask;
    __shared__ uint32_t s_need, s_count, s_ncand;

    const int q = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t n = a.n_docs;
    const unsigned long long* keys = reinterpret_cast<const unsigned long long*>(a.keys) + (int64_t)q * n;
    if (tid == 0) {
        s_ncand = 0;
        s_count = 0;
        s_prefix = 0;
        s_mask = 0;
    }
    __syncthreads();
    uint32_t mine = 0;
    for (int64_t x = tid; x < n; x += kTopkThreads) mine += keys[x] != 0;
    atomicAdd(&s_ncand, mine);
    __syncthreads();
    const uint32_t ncand = s_ncand;
    const int K = (int)(ncand < (uint32_t)a.k ? ncand : (uint32_t)a.k);
    if (tid == 0) s_need = (uint32_t)K;
    __syncthreads();

    if (K > 0) {
        for (int shift = 56; shift >= 0; shift -= 8) {
            for (int i = tid; i < 256; i += kTopkThreads) hist[i] = 0;
            __syncthreads();
            const unsigned long long prefix = s_prefix, mask = s_mask;
            for (int64_t x = tid; x < n; x += kTopkThreads) {
                const unsigned long long key = keys[x];
                if (key != 0 && (key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1u);
            }
            __syncthreads();
            if (tid == 0) {
                uint32_t need = s_need, cum = 0;
                int digit = 0;
                for (int dgt = 255; dgt >= 0; --dgt) {
                    if (cum + hist[dgt] >= need) {
                        digit = dgt;
                        break;
                    }
                    cum += hist[dgt];
                }
                s_need = need - cum;
                s_prefix = prefix | ((unsigned long long)digit << shift);
                s_mask = mask | (255ull << shift);
            }
            __syncthreads();
        }
        const unsigned long long kth = s_prefix;  // the K-th largest key
        for (int64_t x = tid; x < n; x += kTopkThreads) {
            const unsigned long long key = keys[x];
            if (key != 0 && key >= kth) {
                const uint32_t p = atomicAdd(&s_count, 1u);
                if (p < (uint32_t)kMaxK) buf[p] = key;
            }
        }
        __syncthreads();
    }
    // bitonic sort, descending, of the K gathered keys padded with zeros
    int np = 2;
    while (np < K) np <<= 1;
    for (int i = tid; i < np; i += kTopkThreads)
        if (i >= K) buf[i] = 0;
    __syncthreads();
    if (K > 1) {
        for (int kk = 2; kk <= np; kk <<= 1) {
            for (int j = kk >> 1; j > 0; j >>= 1) {
                for (int i = tid; i < np; i += kTopkThreads) {
                    const int ixj = i ^ j;
                    if (ixj > i) {
                        const bool desc = (i & kk) == 0;
                        const unsigned long long x = buf[i], y = buf[ixj];
                        if (desc ? (x < y) : (x > y)) {
                            buf[i] = y;
                            buf[ixj] = x;
                        }
                    }
                }
                __syncthreads();
            }
        }
    }
    for (int r = tid; r < a.k; r += kTopkThreads) {
        const int64_t o = (int64_t)q * a.k + r;
        if (r < K) {
            const unsigned long long key = buf[r];
            const int32_t doc = (int32_t)(kMaxDocs - 1 - (int32_t)(key & (kMaxDocs - 1)));
            const int64_t score = (int64_t)(key >> 24) - (1ll << 39);
            a.out_ids[o] = doc;
            a.out_scores[o] = (float)((double)score * (1.0 / (double)(1 << kFrac)));
            if (a.out_fixed) a.out_fixed[o] = score;
        } else {
            a.out_ids[o] = -1;
            a.out_scores[o] = -__builtin_inff();
            if (a.out_fixed) a.out_fixed[o] = INT64_MIN;
        }
    }
    if (tid == 0 && a.out_counts) a.out_counts[q] = K;
}

void launch_topk(const WaveArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(k_topk, dim3(a.n_q), dim3(kTopkThreads), 0, s, a);
}

}  // namespace warp
