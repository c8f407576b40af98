// Final top-k (Section 4.5: the k best candidate documents by score).
//
// One workgroup per query over its n_docs sort keys (fold kernel). A key is
// ((score + 2^39) << 24) | (2^24 - 1 - doc): keys are distinct, larger is
// better, and the score is key >> 24 (offset). The fold leaves, per block of
// 256 documents, the candidate count and the largest key.
//
// With K = min(k, candidates), histograms of the blocks' largest keys (coarse, then
// fine inside the crossing bin) first give a distance D0 below the best score such
// that at least K block maxima, hence at least K keys, lie within it: every one of the
// K largest keys then lies in a block whose maximum is within D0, and the keys of any
// other block are smaller than all of these. The passes below visit only those blocks,
// listed in LDS (all blocks when more than kTopkListCap pass, or no D0 is found). The
// first pass over their keys gathers every key within D0; if at most kMaxK, these are
// ranked or sorted and the first K decoded. Otherwise the
// K largest keys are found in one or two histogram passes over the keys: bins of the
// distance below the largest score (4096 bins of 2^-6, then, inside the bin holding the
// K-th key, 4096 bins of 2^-18), after which every key at or above the bin holding the
// K-th key is gathered (at most kMaxK); each takes its rank among them as its position
// (up to kRankMax keys), or they are sorted in LDS, and the first K are decoded. When
// the K-th key lies more than 64 below the best, or its fine bin alone would overflow
// the gather buffer, an MSB-first radix select over the whole key (8 bits per pass)
// finds the K-th key exactly instead.
#include "engine.h"

namespace warp {

constexpr int kTopkThreads = 1024;
constexpr int kTopkBins = 4096;
constexpr int kCoarseShift = 20;  // coarse bin width: 2^20 units of 2^-26
constexpr int kFineShift = 8;     // fine bin width inside one coarse bin: 2^8 units
constexpr int kRankMax = 512;     // up to this many gathered keys are placed by rank, more are sorted
constexpr int kKeysInFlight = 8;  // key loads per thread in flight in every pass over the keys

// Smallest bin b with hist[0] + ... + hist[b] >= need, and the count of bins
// before it; b = -1 if the total is below need. Every thread calls it. The prefix over
// the threads' bin counts is a shuffle scan inside each wave, then over the wave totals.
__device__ void find_crossing(const uint32_t* hist, uint32_t need, uint32_t* scan, int* s_bin,
                              uint32_t* s_before) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int PER = kTopkBins / kTopkThreads;
    constexpr int NWV = kTopkThreads / 64;
    uint32_t mine = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) mine += hist[PER * tid + i];
    uint32_t incl = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t t = __shfl_up(incl, off, 64);
        if (lane >= off) incl += t;
    }
    if (lane == 63) scan[wave] = incl;  // wave totals
    if (tid == 0) *s_bin = -1;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < NWV; ++w) incl += w < wave ? scan[w] : 0;
    const uint32_t excl = incl - mine;
    if (excl < need && incl >= need) {
        uint32_t cum = excl;
        for (int i = 0; i < PER; ++i) {
            const uint32_t h = hist[PER * tid + i];
            if (cum + h >= need) {
                *s_bin = PER * tid + i;
                *s_before = cum;
                break;
            }
            cum += h;
        }
    }
    __syncthreads();
}

// Appends key to buf[*count] where pred holds, with one LDS atomic per wave for the lanes
// that call it together; positions past kMaxK are counted but not written.
__device__ __forceinline__ void append_key(bool pred, unsigned long long key, uint32_t* count,
                                           unsigned long long* buf) {
    const unsigned long long m = __ballot(pred);
    if (m == 0) return;
    const int lane = threadIdx.x & 63;
    const int leader = __builtin_ctzll(m);
    uint32_t base = 0;
    if (lane == leader) base = atomicAdd(count, (uint32_t)__popcll(m));
    base = __shfl(base, leader, 64);
    if (pred) {
        const uint32_t p = base + (uint32_t)__popcll(m & ((1ull << lane) - 1));
        if (p < (uint32_t)kMaxK) buf[p] = key;
    }
}

__global__ __launch_bounds__(kTopkThreads) void k_topk(WaveArgs a) {
    __shared__ uint32_t hist[kTopkBins];
    __shared__ uint32_t scan[kTopkThreads / 64];
    __shared__ unsigned long long buf[kMaxK];
    __shared__ int32_t blist[kTopkListCap];
    __shared__ unsigned long long s_prefix, s_mask, s_max, s_lim;
    __shared__ uint32_t s_need, s_count, s_ncand, s_before, s_nlist;
    __shared__ int s_bin;

    const int q = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t n = a.n_docs;
    const int64_t nb = (n + 255) / 256;
    const unsigned long long* keys = reinterpret_cast<const unsigned long long*>(a.keys) + (int64_t)q * n;
    const uint64_t* part = a.qpart + 2 * (int64_t)q * nb;

    // every block's (candidate count, largest key), kKeysInFlight 16-byte loads in flight per thread
    typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
    auto for_each_part = [&](auto&& f) {
        for (int64_t b0 = tid; b0 < nb; b0 += kKeysInFlight * kTopkThreads) {
            u64x2 pv[kKeysInFlight];
#pragma unroll
            for (int u = 0; u < kKeysInFlight; ++u) {
                const int64_t b = b0 + (int64_t)u * kTopkThreads;
                pv[u] = b < nb ? *reinterpret_cast<const u64x2*>(part + 2 * b) : (u64x2){0ull, 0ull};
            }
#pragma unroll
            for (int u = 0; u < kKeysInFlight; ++u) {
                const int64_t b = b0 + (int64_t)u * kTopkThreads;
                if (b < nb) f(b, pv[u].x, pv[u].y);
            }
        }
    };

    // candidates and the largest key, from the fold's per-block partials
    if (tid == 0) {
        s_ncand = 0;
        s_max = 0;
        s_count = 0;
        s_nlist = 0;
    }
    __syncthreads();
    {
        unsigned long long cnt = 0, mx = 0;
        for_each_part([&](int64_t, unsigned long long c, unsigned long long m) {
            cnt += c;
            mx = m > mx ? m : mx;
        });
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {  // one LDS atomic of each kind per wave
            cnt += __shfl_xor(cnt, off, 64);
            const unsigned long long o = __shfl_xor(mx, off, 64);
            mx = o > mx ? o : mx;
        }
        if ((tid & 63) == 0) {
            atomicAdd(&s_ncand, (uint32_t)cnt);
            atomicMax(&s_max, mx);
        }
    }
    __syncthreads();
    const uint32_t ncand = s_ncand;
    const int K = (int)(ncand < (uint32_t)a.k ? ncand : (uint32_t)a.k);
    const unsigned long long smax = s_max >> 24;  // the best (offset) score

    bool done = K == 0;
    // D0 from the block maxima: coarse bins, then fine bins inside the crossing one
    unsigned long long d0 = 0;  // 0: no pruning
    if (!done) {
        for (int i = tid; i < kTopkBins; i += kTopkThreads) hist[i] = 0;
        __syncthreads();
        for_each_part([&](int64_t, unsigned long long, unsigned long long mx) {
            const unsigned long long d = smax - (mx >> 24);
            if (mx != 0 && d < ((unsigned long long)kTopkBins << kCoarseShift)) atomicAdd(&hist[d >> kCoarseShift], 1u);
        });
        __syncthreads();
        find_crossing(hist, (uint32_t)K, scan, &s_bin, &s_before);
        const int b1 = s_bin;
        if (b1 >= 0) {
            const uint32_t need = (uint32_t)K - s_before;
            __syncthreads();
            for (int i = tid; i < kTopkBins; i += kTopkThreads) hist[i] = 0;
            __syncthreads();
            const unsigned long long base = (unsigned long long)b1 << kCoarseShift;
            for_each_part([&](int64_t, unsigned long long, unsigned long long mx) {
                const unsigned long long d = smax - (mx >> 24);
                if (mx != 0 && d >= base && d - base < (1ull << kCoarseShift))
                    atomicAdd(&hist[(d - base) >> kFineShift], 1u);
            });
            __syncthreads();
            find_crossing(hist, need, scan, &s_bin, &s_before);
            d0 = base + ((unsigned long long)(s_bin + 1) << kFineShift);  // the crossing exists
        }
        if (d0 != 0) {
            for_each_part([&](int64_t b, unsigned long long, unsigned long long mx) {
                if (mx != 0 && smax - (mx >> 24) < d0) {
                    const uint32_t p = atomicAdd(&s_nlist, 1u);
                    if (p < (uint32_t)kTopkListCap) blist[p] = (int32_t)b;
                }
            });
        }
        __syncthreads();
    }
    const uint32_t nlist = s_nlist;
    const bool pruned = d0 != 0 && nlist <= (uint32_t)a.topk_list_cap;
    // every key of the listed blocks, or of all blocks
    // (kKeysInFlight loads per thread are issued before any of their keys is used)
    auto for_each_key = [&](auto&& f) {
        const int64_t total = pruned ? (int64_t)nlist * 256 : n;
        for (int64_t j0 = tid; j0 < total; j0 += kKeysInFlight * kTopkThreads) {
            unsigned long long kv[kKeysInFlight];
#pragma unroll
            for (int u = 0; u < kKeysInFlight; ++u) {
                const int64_t j = j0 + (int64_t)u * kTopkThreads;
                const int64_t x = pruned ? (int64_t)blist[j < total ? j >> 8 : 0] * 256 + (j & 255) : j;
                kv[u] = j < total && x < n ? keys[x] : 0ull;
            }
#pragma unroll
            for (int u = 0; u < kKeysInFlight; ++u)
                if (kv[u] != 0) f(kv[u]);
        }
    };
    // level 1: coarse bins of the distance below the best score. The same pass gathers every
    // key within D0, a set that holds the K best: when it fits the buffer (kMaxK keys), they
    // are ranked or sorted directly and the passes below are skipped.
    if (!done) {
        for (int i = tid; i < kTopkBins; i += kTopkThreads) hist[i] = 0;
        __syncthreads();
        const bool spec = d0 != 0;  // uniform
        for_each_key([&](unsigned long long key) {
            const unsigned long long d = smax - (key >> 24);
            if (d < ((unsigned long long)kTopkBins << kCoarseShift)) atomicAdd(&hist[d >> kCoarseShift], 1u);
            if (spec) append_key(d < d0, key, &s_count, buf);
        });
        __syncthreads();
        if (spec && s_count <= (uint32_t)kMaxK) done = true;  // uniform
        else if (spec) {
            __syncthreads();  // every thread has read s_count
            if (tid == 0) s_count = 0;
        }
    }
    if (!done) {
        find_crossing(hist, (uint32_t)K, scan, &s_bin, &s_before);
        const int b1 = s_bin;
        if (b1 >= 0) {
            const uint32_t above = s_before;
            unsigned long long lim = 0;  // gather every key with distance < lim
            if (above + hist[b1] <= (uint32_t)kMaxK) {
                lim = (unsigned long long)(b1 + 1) << kCoarseShift;
            } else {
                // level 2: fine bins inside coarse bin b1
                __syncthreads();
                for (int i = tid; i < kTopkBins; i += kTopkThreads) hist[i] = 0;
                __syncthreads();
                const unsigned long long base = (unsigned long long)b1 << kCoarseShift;
                for_each_key([&](unsigned long long key) {
                    const unsigned long long d = smax - (key >> 24);
                    if (d >= base && d - base < (1ull << kCoarseShift))
                        atomicAdd(&hist[(d - base) >> kFineShift], 1u);
                });
                __syncthreads();
                find_crossing(hist, (uint32_t)K - above, scan, &s_bin, &s_before);
                const int b2 = s_bin;
                if (b2 >= 0 && above + s_before + hist[b2] <= (uint32_t)kMaxK)
                    lim = base + ((unsigned long long)(b2 + 1) << kFineShift);
            }
            if (tid == 0) s_lim = lim;
            __syncthreads();
            lim = s_lim;
            if (lim != 0) {
                for_each_key([&](unsigned long long key) { append_key(smax - (key >> 24) < lim, key, &s_count, buf); });
                done = true;
            }
        }
        __syncthreads();
    }
    // fallback: exact radix select of the K-th key, 8 bits per pass
    if (!done) {
        if (tid == 0) {
            s_need = (uint32_t)K;
            s_prefix = 0;
            s_mask = 0;
            s_count = 0;
        }
        __syncthreads();
        for (int shift = 56; shift >= 0; shift -= 8) {
            for (int i = tid; i < 256; i += kTopkThreads) hist[i] = 0;
            __syncthreads();
            const unsigned long long prefix = s_prefix, mask = s_mask;
            for_each_key([&](unsigned long long key) {
                if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1u);
            });
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
        for_each_key([&](unsigned long long key) { append_key(key >= kth, key, &s_count, buf); });
        __syncthreads();
    }
    const int cnt = K == 0 ? 0 : (int)(s_count < (uint32_t)kMaxK ? s_count : (uint32_t)kMaxK);
    auto emit = [&](int r, unsigned long long key) {  // output position r < K
        const int64_t o = (int64_t)q * a.k + r;
        const int32_t doc = (int32_t)(kMaxDocs - 1 - (int32_t)(key & (kMaxDocs - 1)));
        const int64_t score = (int64_t)(key >> 24) - (1ll << 39);
        a.out_ids[o] = doc;
        a.out_scores[o] = (float)((double)score * (1.0 / (double)(1 << kFrac)));
        if (a.out_fixed) a.out_fixed[o] = score;
    };
    if (cnt <= kRankMax) {
        // few gathered keys: each key's position is the number of larger ones (keys are distinct)
        for (int t = tid; t < cnt; t += kTopkThreads) {
            const unsigned long long key = buf[t];
            int r = 0;
            for (int j = 0; j < cnt; ++j) r += buf[j] > key ? 1 : 0;
            if (r < K) emit(r, key);
        }
    } else {
        // bitonic sort, descending, of the gathered keys padded with zeros; the first K are the result
        int np = 2;
        while (np < cnt) np <<= 1;
        for (int i = tid; i < np; i += kTopkThreads)
            if (i >= cnt) buf[i] = 0;
        __syncthreads();
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
        for (int r = tid; r < K; r += kTopkThreads) emit(r, buf[r]);
    }
    for (int r = K + tid; r < a.k; r += kTopkThreads) {
        const int64_t o = (int64_t)q * a.k + r;
        a.out_ids[o] = -1;
        a.out_scores[o] = -__builtin_inff();
        if (a.out_fixed) a.out_fixed[o] = INT64_MIN;
    }
    if (tid == 0 && a.out_counts) a.out_counts[q] = K;
}

void launch_topk(const WaveArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(k_topk, dim3(a.n_q), dim3(kTopkThreads), 0, s, a);
}

}  // namespace warp
