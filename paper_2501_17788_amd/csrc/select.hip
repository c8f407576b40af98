// WARP_SELECT (Section 4.3): for every query token, the n_probe centroids with
// the highest scores, ordered by (score desc, id asc), and the missing-similarity
// estimate m_i = score of the first centroid in that order whose inclusive
// cumulative cluster size exceeds t' (the last centroid when none does).
//
// The exact order is defined on fp64 scores S64 = sum_d (double)c_d (double)q_d
// taken in dimension order. One workgroup per token:
//   1. a histogram of the fp32 matrix-core scores f over kSelBins equal bins of
//      [-kSelLim, kSelLim), counting centroids and summing their sizes;
//   2. from the top bin down: the bin b_P where the centroid count reaches
//      n_probe and the bin b_t where the size sum first exceeds t';
//   3. every centroid whose bin is within 2 of those boundaries, or above b_P,
//      is rescored in fp64 and sorted by (S64 desc, id asc).
// Since |f - S64| <= kFilterEps and a bin is wider than 2 kFilterEps, a centroid
// three or more bins above (below) the t' bin scores strictly above (below) m_i,
// and no centroid outside the collected set can be among the n_probe best. So
// the rescored set decides sel and m_i exactly, as the full fp64 sort would.
#include "engine.h"

namespace warp {

__device__ __forceinline__ int score_bin(float f) {
    const float scale = (float)kSelBins / (2.0f * kSelLim);
    int b = (int)floorf((f + kSelLim) * scale);
    return b < 0 ? 0 : (b >= kSelBins ? kSelBins - 1 : b);
}

__device__ __forceinline__ int64_t to_fixed(double x) {
    return (int64_t)__builtin_rint(x * (double)(1 << kFrac));
}

// x comes before y in (score desc, id asc) order
__device__ __forceinline__ bool before(double xs, int xi, double ys, int yi) {
    return xs > ys || (xs == ys && xi < yi);
}

// Bitonic sort of n (a power of two) LDS entries in (score desc, id asc) order.
__device__ void sort_desc(double* s, int* id, int n) {
    for (int k = 2; k <= n; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < n; i += blockDim.x) {
                const int ixj = i ^ j;
                if (ixj > i) {
                    const bool asc = (i & k) == 0;
                    const bool swap = asc ? before(s[ixj], id[ixj], s[i], id[i])
                                          : before(s[i], id[i], s[ixj], id[ixj]);
                    if (swap) {
                        const double ts = s[i];
                        s[i] = s[ixj];
                        s[ixj] = ts;
                        const int ti = id[i];
                        id[i] = id[ixj];
                        id[ixj] = ti;
                    }
                }
            }
            __syncthreads();
        }
    }
}

// fp64 centroid score, accumulated in dimension order (each product is exact).
__device__ __forceinline__ double score64(const float* __restrict__ cen, int c, const float* qs) {
    const float4* row = reinterpret_cast<const float4*>(cen + (int64_t)c * kDim);
    double s = 0.0;
#pragma unroll 4
    for (int k = 0; k < kDim / 4; ++k) {
        const float4 v = row[k];
        s = __builtin_fma((double)v.x, (double)qs[4 * k + 0], s);
        s = __builtin_fma((double)v.y, (double)qs[4 * k + 1], s);
        s = __builtin_fma((double)v.z, (double)qs[4 * k + 2], s);
        s = __builtin_fma((double)v.w, (double)qs[4 * k + 3], s);
    }
    return s;
}

__device__ __forceinline__ int pow2_at_least(int n) {
    int p = 2;
    while (p < n) p <<= 1;
    return p;
}

__global__ __launch_bounds__(256) void k_select(WaveArgs a) {
    constexpr int NT = 256;
    constexpr int PER = kSelBins / NT;
    __shared__ uint32_t hcnt[kSelBins];
    __shared__ unsigned long long hw[kSelBins];
    __shared__ uint32_t scnt[NT];
    __shared__ unsigned long long sw[NT];
    __shared__ float qs[kDim];
    __shared__ double sA[kSelCap], sB[kSelCap];
    __shared__ int idA[kSelCap], idB[kSelCap];
    __shared__ int s_bP, s_bt, s_blo, s_nA, s_nB;
    __shared__ unsigned long long s_wabove;

    const int t = blockIdx.x;
    const int tid = threadIdx.x;
    const int n_c = a.n_c, P = a.nprobe;
    const unsigned long long tp = (unsigned long long)a.t_prime;
    for (int i = tid; i < kSelBins; i += NT) {
        hcnt[i] = 0;
        hw[i] = 0;
    }
    if (tid < kDim) qs[tid] = a.queries[(int64_t)t * kDim + tid];
    if (tid == 0) {
        s_bP = -1;
        s_bt = -1;
        s_blo = kSelBins;
        s_nA = 0;
        s_nB = 0;
        s_wabove = 0;
    }
    __syncthreads();

    // 1. histogram of filter scores: counts and size sums
    const float* f = a.filter + (int64_t)t * n_c;
    for (int c = tid; c < n_c; c += NT) {
        const int b = score_bin(f[c]);
        atomicAdd(&hcnt[b], 1u);
        const int32_t sz = a.sizes[c];
        if (sz) atomicAdd(&hw[b], (unsigned long long)sz);
    }
    __syncthreads();

    // 2. suffix sums over bins; thread tid owns bins [PER * tid, PER * tid + PER)
    uint32_t own_c = 0;
    unsigned long long own_w = 0;
    for (int j = 0; j < PER; ++j) {
        own_c += hcnt[PER * tid + j];
        own_w += hw[PER * tid + j];
    }
    scnt[tid] = own_c;
    sw[tid] = own_w;
    __syncthreads();
    for (int off = 1; off < NT; off <<= 1) {  // inclusive suffix scan over threads
        const uint32_t vc = tid + off < NT ? scnt[tid + off] : 0;
        const unsigned long long vw = tid + off < NT ? sw[tid + off] : 0;
        __syncthreads();
        scnt[tid] += vc;
        sw[tid] += vw;
        __syncthreads();
    }
    const uint32_t above_c = scnt[tid] - own_c;
    const unsigned long long above_w = sw[tid] - own_w;
    if (above_c < (uint32_t)P && above_c + own_c >= (uint32_t)P) {
        uint32_t run = above_c;
        for (int j = PER - 1; j >= 0; --j) {
            run += hcnt[PER * tid + j];
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
            if (run + hw[b] > tp) {
                s_bt = b;
                s_wabove = run;  // size of every bin above b
                break;
            }
            run += hw[b];
        }
    }
    for (int j = 0; j < PER; ++j) {
        if (hcnt[PER * tid + j]) {
            atomicMin(&s_blo, PER * tid + j);
            break;
        }
    }
    __syncthreads();

    // 3. collect the centroids near the boundaries
    const int bA = s_bP - 2 < 0 ? 0 : s_bP - 2;
    const bool clamp = s_bt < 0;  // total size <= t': m is the lowest score
    const int bt_lo = clamp ? s_blo : (s_bt - 2 < 0 ? 0 : s_bt - 2);
    const int bt_hi = clamp ? (s_blo + 2 < kSelBins ? s_blo + 2 : kSelBins - 1)
                            : (s_bt + 2 < kSelBins ? s_bt + 2 : kSelBins - 1);
    for (int c = tid; c < n_c; c += NT) {
        const int b = score_bin(f[c]);
        if (b >= bA) {
            const int p = atomicAdd(&s_nA, 1);
            if (p < kSelCap) idA[p] = c;
        }
        if (b >= bt_lo && b <= bt_hi) {
            const int p = atomicAdd(&s_nB, 1);
            if (p < kSelCap) idB[p] = c;
        }
    }
    __syncthreads();
    const int nA = s_nA, nB = s_nB;
    int32_t* sel = a.sel + (int64_t)t * P;
    int32_t* base = a.base + (int64_t)t * P;
    int64_t* seg_start = a.seg_start + (int64_t)t * P;
    int64_t* seg_pref = a.seg_pref + (int64_t)t * (P + 1);
    if (nA > kSelCap || nB > kSelCap || nA < P || nB < 1) {
        // degenerate score distribution: leave a token that scans nothing
        for (int j = tid; j < P; j += NT) {
            sel[j] = -1;  // probes nothing
            base[j] = 0;
            seg_start[j] = 0;
        }
        for (int j = tid; j <= P; j += NT) seg_pref[j] = 0;
        if (tid == 0) {
            a.m_fixed[t] = 0;
            atomicOr(a.err, kErrSelOverflow);
        }
        return;
    }

    // 4. fp64 rescoring and exact order
    const int pA = pow2_at_least(nA), pB = pow2_at_least(nB);
    for (int p = tid; p < pA; p += NT) {
        if (p < nA) {
            sA[p] = score64(a.centroids, idA[p], qs);
        } else {
            sA[p] = -__builtin_inf();
            idA[p] = 0x7fffffff;
        }
    }
    for (int p = tid; p < pB; p += NT) {
        if (p < nB) {
            sB[p] = score64(a.centroids, idB[p], qs);
        } else {
            sB[p] = -__builtin_inf();
            idB[p] = 0x7fffffff;
        }
    }
    __syncthreads();
    sort_desc(sA, idA, pA);
    sort_desc(sB, idB, pB);

    for (int j = tid; j < P; j += NT) {
        const int c = idA[j];
        sel[j] = c;
        base[j] = (int32_t)to_fixed(sA[j]);
        seg_start[j] = a.offsets[c];
        if (a.dbg_sel) a.dbg_sel[(int64_t)t * P + j] = c;
    }
    if (tid == 0) {
        int64_t run = 0;
        seg_pref[0] = 0;
        for (int j = 0; j < P; ++j) {
            run += a.sizes[idA[j]];
            seg_pref[j + 1] = run;
        }
        // m_i: walk the boundary band in exact order from the size of everything above it
        double m = sB[nB - 1];
        if (!clamp) {
            unsigned long long cum = s_wabove;
            for (int b = s_bt + 1; b <= bt_hi; ++b) cum -= hw[b];
            bool found = false;
            for (int p = 0; p < nB; ++p) {
                cum += (unsigned long long)a.sizes[idB[p]];
                if (cum > tp) {
                    m = sB[p];
                    found = true;
                    break;
                }
            }
            if (!found) atomicOr(a.err, kErrSelNoCrossing);
        }
        a.m_fixed[t] = to_fixed(m);
        if (a.dbg_m) a.dbg_m[t] = to_fixed(m);
    }
}

void launch_select(const WaveArgs& a, hipStream_t s) {
    const int n_tok = a.n_q * a.n_qtok;
    hipLaunchKernelGGL(k_select, dim3(n_tok), dim3(256), 0, s, a);
}

}  // namespace warp
