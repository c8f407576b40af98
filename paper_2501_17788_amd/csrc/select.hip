// WARP_SELECT (Section 4.3): for every query token, the n_probe centroids with
// the highest scores, ordered by (score desc, id asc), and the missing-similarity
// estimate m_i = score of the first centroid in that order whose inclusive
// cumulative cluster size exceeds t' (the last centroid when none does).
//
// The exact order is defined on fp64 scores S64 = sum_d (double)c_d (double)q_d
// taken in dimension order. The filter GEMM gives, for every (token, centroid),
// the histogram bin of its fp32 matrix-core score f (score_bin). One workgroup
// per token:
//   1. a histogram over the bins, counting centroids and summing their sizes;
//   2. from the top bin down: the bin b_P where the centroid count reaches
//      n_probe and the bin b_t where the size sum first exceeds t';
//   3. every centroid whose bin is within 2 of b_t, or at least b_P - 2, is
//      rescored in fp64 and placed in (S64 desc, id asc) order by its rank.
// Since |f - S64| <= kFilterEps and a bin is wider than 2 kFilterEps, a centroid
// three or more bins above (below) b_t scores strictly above (below) m_i, and no
// centroid below bin b_P - 2 can be among the n_probe best. Walking the rescored
// band in exact order, starting from the size of every bin above it, the first
// entry whose cumulative size exceeds t' gives m_i: entries of the band that lie
// above the true boundary reach at most the size of all bins above b_t, which
// does not exceed t'. So sel and m_i are those of the full fp64 sort.
#include "engine.h"

namespace warp {

__device__ __forceinline__ int64_t to_fixed(double x) {
    return (int64_t)__builtin_rint(x * (double)(1 << kFrac));
}

// x comes before y in (score desc, id asc) order
__device__ __forceinline__ bool before(double xs, int xi, double ys, int yi) {
    return xs > ys || (xs == ys && xi < yi);
}

constexpr int kSelThreads = 512;

// Calls place(p, r) for each of the n LDS entries p, with r the number of entries that come
// before it in (score desc, id asc) order: its position in that order, since ids are
// distinct. Each entry is ranked by a group of L lanes of one wave (the largest power of two
// up to 64 with n L <= kSelThreads, at least 1), which split the comparisons and add their
// counts; place runs on the group's first lane. Every thread calls it.
template <typename F>
__device__ __forceinline__ void rank_all(const double* s, const int* id, int n, F place) {
    int L = 64;
    while (L > 1 && n * L > kSelThreads) L >>= 1;
    const int sub = threadIdx.x & (L - 1);
    for (int p = threadIdx.x / L; p < n; p += kSelThreads / L) {  // uniform over each group
        const double xs = s[p];
        const int xi = id[p];
        int r = 0;
        for (int j = sub; j < n; j += L) r += before(s[j], id[j], xs, xi) ? 1 : 0;
        for (int off = L >> 1; off > 0; off >>= 1) r += __shfl_xor(r, off, 64);
        if (sub == 0) place(p, r);
    }
}

// fp64 centroid score, accumulated in dimension order (each product is exact), by the
// four lanes 4 m .. 4 m + 3 of a wave that share centroid c: lane part loads dimensions
// 32 part .. 32 part + 31 (one round trip for the whole row), and the running sum passes
// from lane to lane in that order. Every lane of the four returns the score; the cluster's
// size is loaded with the row.
// (one copy per calling kernel: with one copy called from both selection kernels, each took
// 97 VGPRs instead of 68)
template <bool K>
__device__ __noinline__ double score64_quad(const float* __restrict__ cen, const int32_t* __restrict__ sizes,
                                               int c, const float* qs, int part, int& size) {
    const float4* row = reinterpret_cast<const float4*>(cen + (int64_t)c * kDim) + 8 * part;
    float4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = row[k];
    size = sizes[c];
    const int lead = (threadIdx.x & 63) & ~3;
    const float* qp = qs + 32 * part;
    double s = 0.0;
#pragma unroll 1
    for (int seg = 0; seg < 4; ++seg) {
        if (part == seg) {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                float4 w = v[k];
                // keeps the fp64 conversions inside the branch (else all 32 are hoisted)
                asm volatile("" : "+v"(w.x), "+v"(w.y), "+v"(w.z), "+v"(w.w));
                s = __builtin_fma((double)w.x, (double)qp[4 * k + 0], s);
                s = __builtin_fma((double)w.y, (double)qp[4 * k + 1], s);
                s = __builtin_fma((double)w.z, (double)qp[4 * k + 2], s);
                s = __builtin_fma((double)w.w, (double)qp[4 * k + 3], s);
            }
        }
        s = __shfl(s, lead + seg, 64);
    }
    return s;
}

constexpr int kBinLoads = 8;  // 16-byte bin loads in flight per thread: 2^15 bins in one round

// Inclusive prefix sum over the block of one value per thread: shuffle scans inside
// each wave, then the wave totals through LDS (wtot: one entry per wave). Also returns
// the block total. Every thread calls it.
__device__ unsigned long long block_scan(unsigned long long v, unsigned long long* wtot,
                                         unsigned long long* total) {
    constexpr int NW = kSelThreads / 64;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const unsigned long long t = __shfl_up(v, off, 64);
        if (lane >= off) v += t;
    }
    if (lane == 63) wtot[w] = v;
    __syncthreads();
    unsigned long long base = 0, all = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        base += i < w ? wtot[i] : 0;
        all += wtot[i];
    }
    __syncthreads();  // wtot is free again
    *total = all;
    return v + base;
}

// Inclusive prefix sum of n <= 2 kSelThreads int64 values in LDS.
__device__ void block_inclusive_scan(int64_t* v, int n, unsigned long long* wtot) {
    const int i0 = 2 * threadIdx.x;
    const int64_t a = i0 < n ? v[i0] : 0, b = i0 + 1 < n ? v[i0 + 1] : 0;
    unsigned long long total;
    const unsigned long long incl = block_scan((unsigned long long)(a + b), wtot, &total);
    const int64_t excl = (int64_t)incl - (a + b);
    if (i0 < n) v[i0] = excl + a;
    if (i0 + 1 < n) v[i0 + 1] = excl + a + b;
    __syncthreads();
}

constexpr unsigned long long kCntOne = 1ull << 40;  // histogram word: (count << 40) | size sum
constexpr unsigned long long kSizeMask = kCntOne - 1;

// Calls f(c, bin) for every centroid of the token's row of bins: 16-byte loads of
// eight bins when the row is 16-byte aligned, kBinLoads loads in flight per thread.
template <typename F>
__device__ __forceinline__ void for_each_bin(const uint16_t* bins, int n_c, F f) {
    constexpr int NT = kSelThreads;
    const int tid = threadIdx.x;
    if ((n_c & 7) == 0 && ((uintptr_t)bins & 15) == 0) {
        const uint4* b4 = reinterpret_cast<const uint4*>(bins);
        const int n8 = n_c >> 3;
        for (int j0 = 0; j0 < n8; j0 += kBinLoads * NT) {
            uint4 v[kBinLoads];
#pragma unroll
            for (int u = 0; u < kBinLoads; ++u) {
                const int j = j0 + u * NT + tid;
                v[u] = j < n8 ? b4[j] : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int u = 0; u < kBinLoads; ++u) {
                const int j = j0 + u * NT + tid;
                if (j >= n8) continue;
                const unsigned w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    f(8 * j + 2 * h, (int)(w[h] & 0xFFFFu));
                    f(8 * j + 2 * h + 1, (int)(w[h] >> 16));
                }
            }
        }
    } else {
        for (int c = tid; c < n_c; c += NT) f(c, (int)bins[c]);
    }
}

// Step 2 of the selection over the token's histogram in LDS (every thread calls it, after a
// barrier that follows the histogram's last write): from the top bin down, the bin b_P where the
// centroid count reaches n_probe (-1: none) and the bin b_t where the size sum first exceeds t'
// (-1: none) with the size of every bin above it, and the lowest occupied bin.
struct SelBounds {
    int bP, bt, blo;
    unsigned long long wabove;
};
__device__ __forceinline__ SelBounds hist_bounds(const unsigned long long* hist, unsigned long long* wtot, uint32_t P,
                                                 unsigned long long tp) {
    constexpr int NT = kSelThreads;
    constexpr int PER = kSelBins / NT;
    __shared__ int s_bP, s_bt, s_blo;
    __shared__ unsigned long long s_wabove;
    const int tid = threadIdx.x;
    if (tid == 0) {  // ordered before the writes below by the block scan's barrier
        s_bP = -1;
        s_bt = -1;
        s_blo = kSelBins;
        s_wabove = 0;
    }
    // suffix sums over bins; thread tid owns bins [PER * tid, PER * tid + PER). Packed words
    // add field by field: sizes total < 2^40, counts < 2^24.
    unsigned long long own = 0;
    for (int j = 0; j < PER; ++j) own += hist[PER * tid + j];
    unsigned long long total;
    const unsigned long long incl = block_scan(own, wtot, &total);
    const unsigned long long above = total - incl;  // every bin above this thread's
    const uint32_t above_c = (uint32_t)(above >> 40), own_c = (uint32_t)(own >> 40);
    const unsigned long long above_w = above & kSizeMask, own_w = own & kSizeMask;
    if (above_c < (uint32_t)P && above_c + own_c >= (uint32_t)P) {
        uint32_t run = above_c;
        for (int j = PER - 1; j >= 0; --j) {
            run += (uint32_t)(hist[PER * tid + j] >> 40);
            if (run >= (uint32_t)P) {
                s_bP = PER * tid + j;
                break;
            }
        }
    }
    if (above_w <= tp && above_w + own_w > tp) {
        unsigned long long run = above_w;
        for (int j = PER - 1; j >= 0; --j) {
            const int b = PER * tid + j;
            const unsigned long long w = hist[b] & kSizeMask;
            if (run + w > tp) {
                s_bt = b;
                s_wabove = run;  // size of every bin above b
                break;
            }
            run += w;
        }
    }
    int lo = kSelBins;  // the lowest occupied bin: one LDS atomic per wave
    for (int j = PER - 1; j >= 0; --j)
        if (hist[PER * tid + j] >> 40) lo = PER * tid + j;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const int o = __shfl_xor(lo, off, 64);
        lo = o < lo ? o : lo;
    }
    if ((tid & 63) == 0 && lo < kSelBins) atomicMin(&s_blo, lo);
    __syncthreads();
    return SelBounds{s_bP, s_bt, s_blo, s_wabove};
}

// The bins whose centroids the selection rescores: every bin from b_P - 2 up (list A, the
// n_probe best), and b_t - 2 .. b_t + 2 (list B, the t' crossing; around the lowest occupied
// bin when the total size does not exceed t').
struct SelBand {
    int bA, lo, hi;
    bool clamp;
};
__device__ __forceinline__ SelBand sel_band(int bP, int bt, int blo) {
    SelBand r;
    r.bA = bP - 2 < 0 ? 0 : bP - 2;
    r.clamp = bt < 0;  // total size <= t': m is the lowest score
    r.lo = r.clamp ? blo : (bt - 2 < 0 ? 0 : bt - 2);
    r.hi = r.clamp ? (blo + 2 < kSelBins ? blo + 2 : kSelBins - 1) : (bt + 2 < kSelBins ? bt + 2 : kSelBins - 1);
    return r;
}

// Centroids [c0, c1) of token t's row of bins: the slice that workgroup x of S takes (slices of
// a multiple of 8 centroids, so that 16-byte loads stay aligned).
__device__ __forceinline__ void sel_slice(int n_c, int S, int x, int& c0, int& c1) {
    const int len = ((n_c + S - 1) / S + 7) & ~7;
    c0 = x * len < n_c ? x * len : n_c;
    c1 = c0 + len < n_c ? c0 + len : n_c;
}

// Split selection, for waves of few tokens (one workgroup per token would leave most of the
// GPU idle while each reads its whole row of bins twice). Grid (S, n_tok): each workgroup adds
// the histogram of its slice of the token's bins into the token's histogram in global memory
// (zeroed by the wave's preparation).
__global__ __launch_bounds__(kSelThreads) void k_select_hist(WaveArgs a) {
    __shared__ unsigned long long hist[kSelBins];
    const int t = blockIdx.y, tid = threadIdx.x;
    const int n_c = a.n_c;
    int c0, c1;
    sel_slice(n_c, gridDim.x, blockIdx.x, c0, c1);
    for (int i = tid; i < kSelBins; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    const int32_t* sizes = a.sizes + c0;
    for_each_bin(a.filter_bins + (int64_t)t * n_c + c0, c1 - c0, [&](int c, int b) {
        atomicAdd(&hist[b], kCntOne | (unsigned long long)sizes[c]);
    });
    __syncthreads();
    unsigned long long* g = a.sel_hist + (int64_t)t * kSelBins;
    for (int i = tid; i < kSelBins; i += kSelThreads)
        if (hist[i]) atomicAdd(&g[i], hist[i]);
}

// Then each workgroup reads the token's whole histogram, finds the bands, gathers the centroids
// of its slice that fall in them in LDS and appends them to the token's two lists in global
// memory with one atomic per list (the counts may exceed kSelCap; the final kernel treats that
// as the overflow it is).
__global__ __launch_bounds__(kSelThreads) void k_select_collect(WaveArgs a) {
    __shared__ unsigned long long hist[kSelBins];
    __shared__ unsigned long long wtot[kSelThreads / 64];
    __shared__ int s_list[2][kSelCap];
    __shared__ int s_n[2], s_at[2];
    const int t = blockIdx.y, tid = threadIdx.x;
    const int n_c = a.n_c;
    const unsigned long long* g = a.sel_hist + (int64_t)t * kSelBins;
    for (int i = tid; i < kSelBins; i += kSelThreads) hist[i] = g[i];
    if (tid == 0) {
        s_n[0] = 0;
        s_n[1] = 0;
    }
    __syncthreads();
    const SelBounds bd = hist_bounds(hist, wtot, (uint32_t)a.nprobe, (unsigned long long)a.t_prime);
    const SelBand band = sel_band(bd.bP, bd.bt, bd.blo);
    int c0, c1;
    sel_slice(n_c, gridDim.x, blockIdx.x, c0, c1);
    int32_t* cnt = a.sel_cnt + 2 * (int64_t)t;
    int32_t* listA = a.sel_lists + 2 * (int64_t)t * kSelCap;
    int32_t* listB = listA + kSelCap;
    for_each_bin(a.filter_bins + (int64_t)t * n_c + c0, c1 - c0, [&](int c, int b) {
        if (b >= band.bA) {
            const int p = atomicAdd(&s_n[0], 1);
            if (p < kSelCap) s_list[0][p] = c0 + c;
        }
        if (b >= band.lo && b <= band.hi) {
            const int p = atomicAdd(&s_n[1], 1);
            if (p < kSelCap) s_list[1][p] = c0 + c;
        }
    });
    __syncthreads();
    if (tid < 2) s_at[tid] = s_n[tid] ? atomicAdd(&cnt[tid], s_n[tid]) : 0;
    __syncthreads();
    for (int l = 0; l < 2; ++l) {
        const int n = s_n[l] < kSelCap ? s_n[l] : kSelCap;
        int32_t* dst = l == 0 ? listA : listB;
        for (int p = tid; p < n; p += kSelThreads)
            if (s_at[l] + p < kSelCap) dst[s_at[l] + p] = s_list[l][p];
    }
}

// SPLIT: the histogram and the band lists come from k_select_hist and k_select_collect.
template <bool SPLIT>
__global__ __launch_bounds__(kSelThreads) void k_select(WaveArgs a) {
    constexpr int NT = kSelThreads;
    __shared__ unsigned long long hist[kSelBins];
    __shared__ unsigned long long wtot[NT / 64];
    __shared__ float qs[kDim];
    __shared__ double sA[kSelCap], sB[kSelCap];
    __shared__ int idA[kSelCap], idB[kSelCap];
    __shared__ int64_t cum[kSelCap];
    // from step 4 on, hist holds the sizes of the rescored centroids
    int* const szA = reinterpret_cast<int*>(hist);
    int* const szB = szA + kSelCap;
    static_assert(2 * kSelCap * sizeof(int) <= sizeof(hist), "sizes must fit the histogram's LDS");
    __shared__ int s_nA, s_nB, s_cross;
    __shared__ unsigned long long s_band_above;

    const int t = blockIdx.x;
    const int tid = threadIdx.x;
    const int n_c = a.n_c, P = a.nprobe;
    const unsigned long long tp = (unsigned long long)a.t_prime;
    for (int i = tid; i < kSelBins; i += NT) hist[i] = 0;
    if (tid < kDim) qs[tid] = a.queries[(int64_t)t * kDim + tid];
    if (tid == 0) {
        s_nA = 0;
        s_nB = 0;
        s_cross = kSelCap;
    }
    __syncthreads();

    // 1. histogram: one packed (count, size) word per bin
    const uint16_t* bins = a.filter_bins + (int64_t)t * n_c;
    const int32_t* sizes = a.sizes;
    // split: the token's histogram, and its two band lists read whole beside their counts (entries
    // past a count are unused), all in flight together
    if (SPLIT) {
        const unsigned long long* g = a.sel_hist + (int64_t)t * kSelBins;
        for (int i = tid; i < kSelBins; i += NT) hist[i] = g[i];
        const int32_t* cnt = a.sel_cnt + 2 * (int64_t)t;
        const int32_t* listA = a.sel_lists + 2 * (int64_t)t * kSelCap;
        for (int p = tid; p < kSelCap; p += NT) {
            idA[p] = listA[p];
            idB[p] = listA[kSelCap + p];
        }
        if (tid == 0) {  // after its zeroing above
            s_nA = cnt[0];
            s_nB = cnt[1];
        }
    } else {
        for_each_bin(bins, n_c, [&](int c, int b) {
            atomicAdd(&hist[b], kCntOne | (unsigned long long)sizes[c]);
        });
    }
    __syncthreads();

    // 2. the bins of the n_probe-th centroid and of the t' crossing
    const SelBounds bd = hist_bounds(hist, wtot, (uint32_t)P, tp);

    // 3. collect the centroids near the boundaries
    const SelBand band = sel_band(bd.bP, bd.bt, bd.blo);
    const bool clamp = band.clamp;
    const int bt_hi = band.hi;
    if (!SPLIT) {
        for_each_bin(bins, n_c, [&](int c, int b) {
            if (b >= band.bA) {
                const int p = atomicAdd(&s_nA, 1);
                if (p < kSelCap) idA[p] = c;
            }
            if (b >= band.lo && b <= band.hi) {
                const int p = atomicAdd(&s_nB, 1);
                if (p < kSelCap) idB[p] = c;
            }
        });
    }
    if (tid == 0 && !clamp) {  // size of every bin above the band (the histogram is reused below)
        unsigned long long band_above = bd.wabove;
        for (int b = bd.bt + 1; b <= bt_hi; ++b) band_above -= hist[b] & kSizeMask;
        s_band_above = band_above;
    }
    __syncthreads();
    const int nA = s_nA, nB = s_nB;
    int32_t* sel = a.sel + (int64_t)t * P;
    int32_t* base = a.base + (int64_t)t * P;
    int64_t* seg_pref = a.seg_pref + (int64_t)t * (P + 1);
    if (nA > kSelCap || nB > kSelCap || nA < P || nB < 1) {
        // degenerate score distribution: leave a token that probes and scans nothing
        for (int j = tid; j < P; j += NT) {
            sel[j] = -1;
            base[j] = 0;
        }
        for (int j = tid; j <= P; j += NT) seg_pref[j] = 0;
        if (tid == 0) {
            a.m_fixed[t] = 0;
            atomicOr(a.err, kErrSelOverflow);
        }
        return;
    }

    // 4. fp64 rescoring of both lists, four lanes per centroid; the sizes come in beside
    for (int p = tid >> 2; p < nA + nB; p += NT / 4) {  // uniform over each four lanes
        const int c = p < nA ? idA[p] : idB[p - nA];
        int sz;
        const double v = score64_quad<SPLIT>(a.centroids, sizes, c, qs, tid & 3, sz);
        if ((tid & 3) == 0) {
            if (p < nA) {
                sA[p] = v;
                szA[p] = sz;
            } else {
                sB[p - nA] = v;
                szB[p - nA] = sz;
            }
        }
    }
    __syncthreads();

    // 5. the n_probe best in exact order (an entry's position is its rank among the rescored
    //    entries), their fixed-point scores and the prefix of their sizes; each selected
    //    cluster counts the token among its probing tokens (the work plan's bucket sizes)
    rank_all(sA, idA, nA, [&](int p, int r) {
        if (r < P) {
            const int c = idA[p];
            sel[r] = c;
            atomicAdd(&a.ccount[c], 1);
            base[r] = (int32_t)to_fixed(sA[p]);
            cum[r] = szA[p];
            if (a.dbg_sel) a.dbg_sel[(int64_t)t * P + r] = c;
        }
    });
    __syncthreads();
    block_inclusive_scan(cum, P, wtot);
    for (int j = tid; j <= P; j += NT) seg_pref[j] = j == 0 ? 0 : cum[j - 1];
    __syncthreads();

    // 6. m_i: the band in exact order (its scores placed by rank into sA, free now), and the
    //    first entry whose cumulative size (from the size of everything above the band)
    //    exceeds t'
    rank_all(sB, idB, nB, [&](int p, int r) {
        sA[r] = sB[p];
        cum[r] = szB[p];
    });
    __syncthreads();
    block_inclusive_scan(cum, nB, wtot);
    if (!clamp) {
        const unsigned long long band_above = s_band_above;
        for (int p = tid; p < nB; p += NT)
            if (band_above + (unsigned long long)cum[p] > tp) atomicMin(&s_cross, p);
    }
    __syncthreads();
    if (tid == 0) {
        double m = sA[nB - 1];  // clamp: the lowest score
        if (!clamp) {
            if (s_cross < nB) m = sA[s_cross];
            else atomicOr(a.err, kErrSelNoCrossing);
        }
        a.m_fixed[t] = to_fixed(m);
        if (a.dbg_m) a.dbg_m[t] = to_fixed(m);
    }
}

void launch_select(const WaveArgs& a, hipStream_t s) {
    const int n_tok = a.n_q * a.n_qtok;
    if (a.sel_slices > 1) {
        const dim3 grid((unsigned)a.sel_slices, (unsigned)n_tok);
        hipLaunchKernelGGL(k_select_hist, grid, dim3(kSelThreads), 0, s, a);
        hipLaunchKernelGGL(k_select_collect, grid, dim3(kSelThreads), 0, s, a);
        hipLaunchKernelGGL(k_select<true>, dim3(n_tok), dim3(kSelThreads), 0, s, a);
    } else {
        hipLaunchKernelGGL(k_select<false>, dim3(n_tok), dim3(kSelThreads), 0, s, a);
    }
}

}  // namespace warp
