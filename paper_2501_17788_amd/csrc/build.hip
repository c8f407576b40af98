// Index construction on the GPU (Section 4.1): k-means on a sample of the token
// embeddings, assignment of every token to its nearest centroid, quantile
// bucket cutoffs and weights of the residuals, and packed b-bit residual codes
// grouped by cluster. Every decision is exact, so the result equals the CPU
// definition bit for bit:
//   * assignment: argmax over centroids of the fp64 score S64 (dimension order),
//     lowest id among equal scores. The fp32 matrix-core filter scores f satisfy
//     |f - S64| <= kFilterEps for tokens and centroids of norm <= 1 + 1e-3, so the
//     argmax is among the centroids with f >= max f - 2 kFilterEps; those are
//     rescored in fp64;
//   * k-means update: the sum over assigned sample tokens of round(x * 2^30) per
//     dimension (exact int64), normalised in fp64 (dimension-order sum of
//     squares, IEEE sqrt and division) and rounded to fp32; a centroid without
//     tokens keeps its value;
//   * quantiles: the ceil(n p)-th smallest residual component (n components of
//     the first n_quant tokens), cutoffs at p = j / 2^b, weights at
//     p = (j + 1/2) / 2^b;
//   * codes: the number of cutoffs <= the fp32 residual component, packed with
//     the first dimension in the most significant bits; embeddings ordered by
//     cluster, then by input order (a stable sort).
#include <algorithm>
#include <cmath>
#include <string>

#include "engine.h"

namespace warp {

constexpr int kArgBlock = 256;
constexpr int kArgCap = 1024;  // candidates within the filter band of one token

__device__ __forceinline__ double dot64(const float* __restrict__ c, const float* __restrict__ x) {
    double s = 0.0;
    for (int d = 0; d < kDim; ++d) s += (double)c[d] * (double)x[d];
    return s;
}

// assign[t] for tokens [t0, t0 + n) from their fp32 filter scores [n][n_c]
__global__ __launch_bounds__(kArgBlock) void k_rows_argmax(const float* __restrict__ scores, int32_t n_c,
                                                           const float* __restrict__ x, const float* __restrict__ cen,
                                                           int32_t* __restrict__ assign, int32_t* err) {
    __shared__ float s_max[kArgBlock / 64];
    __shared__ int s_n;
    __shared__ int s_id[kArgCap];
    __shared__ double s_best[kArgBlock / 64];
    __shared__ int s_bid[kArgBlock / 64];
    const int64_t t = blockIdx.x;
    const int tid = threadIdx.x;
    const float* row = scores + t * n_c;
    float m = -INFINITY;
    for (int c = tid; c < n_c; c += kArgBlock) m = fmaxf(m, row[c]);
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
    if ((tid & 63) == 0) s_max[tid >> 6] = m;
    if (tid == 0) s_n = 0;
    __syncthreads();
    float mx = s_max[0];
    for (int w = 1; w < kArgBlock / 64; ++w) mx = fmaxf(mx, s_max[w]);
    const float thr = mx - 2.5f * kFilterEps;
    for (int c = tid; c < n_c; c += kArgBlock)
        if (row[c] >= thr) {
            const int p = atomicAdd(&s_n, 1);
            if (p < kArgCap) s_id[p] = c;
        }
    __syncthreads();
    const int n = s_n;
    if (n > kArgCap) {
        if (tid == 0) {
            atomicOr(err, kErrArgOverflow);
            assign[t] = 0;
        }
        return;
    }
    const float* xt = x + t * kDim;
    double best = -INFINITY;
    int bid = INT32_MAX;
    for (int p = tid; p < n; p += kArgBlock) {
        const int c = s_id[p];
        const double s = dot64(cen + (int64_t)c * kDim, xt);
        if (s > best || (s == best && c < bid)) {
            best = s;
            bid = c;
        }
    }
    for (int off = 32; off > 0; off >>= 1) {
        const double ob = __shfl_xor(best, off, 64);
        const int oi = __shfl_xor(bid, off, 64);
        if (ob > best || (ob == best && oi < bid)) {
            best = ob;
            bid = oi;
        }
    }
    if ((tid & 63) == 0) {
        s_best[tid >> 6] = best;
        s_bid[tid >> 6] = bid;
    }
    __syncthreads();
    if (tid == 0) {
        best = s_best[0];
        bid = s_bid[0];
        for (int w = 1; w < kArgBlock / 64; ++w)
            if (s_best[w] > best || (s_best[w] == best && s_bid[w] < bid)) {
                best = s_best[w];
                bid = s_bid[w];
            }
        assign[t] = bid;
    }
}

__global__ void k_gather_rows(const float* __restrict__ x, const int64_t* __restrict__ ids, int64_t n,
                              float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n * kDim) return;
    out[i] = x[ids[i / kDim] * kDim + i % kDim];
}

// per centroid: sum of round(x * 2^30) over its assigned sample tokens, and their count
__global__ void k_kmeans_accum(const float* __restrict__ xs, const int32_t* __restrict__ assign, int64_t n,
                               unsigned long long* __restrict__ sums, unsigned long long* __restrict__ counts) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n * kDim) return;
    const int64_t t = i / kDim;
    const int d = (int)(i % kDim);
    const int c = assign[t];
    const long long q = (long long)__builtin_rint((double)xs[i] * 1073741824.0);
    atomicAdd(&sums[(int64_t)c * kDim + d], (unsigned long long)q);  // two's complement sum
    if (d == 0) atomicAdd(&counts[c], 1ull);
}

__global__ void k_kmeans_normalize(const unsigned long long* __restrict__ sums,
                                   const unsigned long long* __restrict__ counts, int32_t n_c,
                                   float* __restrict__ cen) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= n_c || counts[c] == 0) return;
    const unsigned long long* s = sums + (int64_t)c * kDim;
    double ss = 0.0;
    for (int d = 0; d < kDim; ++d) {
        const double m = (double)(long long)s[d];
        ss += m * m;
    }
    if (!(ss > 0.0)) return;
    const double norm = __builtin_sqrt(ss);
    for (int d = 0; d < kDim; ++d) cen[(int64_t)c * kDim + d] = (float)((double)(long long)s[d] / norm);
}

// rows of 128 fp32 values scaled to unit norm: (float)(x_d / ||x||), the norm in fp64 (sum
// of squares in dimension order, IEEE sqrt); the rows were checked to be finite and nonzero
__global__ void k_normalize_rows(float* __restrict__ rows, int32_t n) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= n) return;
    float* r = rows + (int64_t)c * kDim;
    double ss = 0.0;
    for (int d = 0; d < kDim; ++d) ss += (double)r[d] * (double)r[d];
    const double norm = __builtin_sqrt(ss);
    for (int d = 0; d < kDim; ++d) r[d] = (float)((double)r[d] / norm);
}

// residual components of tokens [0, n): x - C[assign]
__global__ void k_residuals(const float* __restrict__ x, const int32_t* __restrict__ assign, int64_t n,
                            const float* __restrict__ cen, float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n * kDim) return;
    out[i] = x[i] - cen[(int64_t)assign[i / kDim] * kDim + i % kDim];
}

// cutoffs (j = 1 .. 2^b - 1) and weights (j = 0 .. 2^b - 1) from the sorted components
__global__ void k_pick_quantiles(const float* __restrict__ sorted, int64_t n, int32_t nbits,
                                 float* __restrict__ cutoffs, float* __restrict__ weights) {
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    const int nb = 1 << nbits;
    auto at = [&](int64_t num, int shift) {  // the ceil(n * num / 2^shift)-th smallest
        int64_t k = (n * num + ((1ll << shift) - 1)) >> shift;
        k = k < 1 ? 1 : (k > n ? n : k);
        return sorted[k - 1];
    };
    if (j >= 1 && j < nb) cutoffs[j - 1] = at(j, nbits);
    if (j < nb) weights[j] = at(2 * j + 1, nbits + 1);
}

// embeddings in cluster order: codes and document ids at position p of token perm[p]
template <int NBITS>
__global__ void k_encode(const float* __restrict__ x, const int32_t* __restrict__ token_docs,
                         const int32_t* __restrict__ assign, const int64_t* __restrict__ perm, int64_t n,
                         const float* __restrict__ cen, const float* __restrict__ cutoffs,
                         uint8_t* __restrict__ codes, int32_t* __restrict__ doc_ids) {
    constexpr int NB = 1 << NBITS;
    constexpr int PER = 8 / NBITS;  // dimensions per byte
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (position, byte)
    constexpr int BYTES = kDim * NBITS / 8;
    if (i >= n * BYTES) return;
    const int64_t p = i / BYTES;
    const int byte = (int)(i % BYTES);
    const int64_t t = perm[p];
    const int c = assign[t];
    unsigned v = 0;
    for (int u = 0; u < PER; ++u) {
        const int d = byte * PER + u;
        const float r = x[t * kDim + d] - cen[(int64_t)c * kDim + d];
        int code = 0;  // number of cutoffs <= r (cutoffs ascend)
        int lo = 0, hi = NB - 1;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (cutoffs[mid] <= r) lo = mid + 1;
            else hi = mid;
        }
        code = lo;
        v |= (unsigned)code << (8 - NBITS * (u + 1));
    }
    codes[p * BYTES + byte] = (uint8_t)v;
    if (byte == 0) doc_ids[p] = token_docs[t];
}

__global__ void k_count_clusters(const int32_t* __restrict__ assign, int64_t n, unsigned long long* counts) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) atomicAdd(&counts[assign[i]], 1ull);
}

__global__ void k_iota64(int64_t* out, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] = i;
}

// ---------------------------------------------------------------------------- launchers

static unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

void launch_rows_argmax(const float* scores, int64_t n, int32_t n_c, const float* x, const float* cen,
                        int32_t* assign, int32_t* err, hipStream_t s) {
    if (n > 0) hipLaunchKernelGGL(k_rows_argmax, dim3((unsigned)n), dim3(kArgBlock), 0, s, scores, n_c, x, cen, assign, err);
}

void launch_gather_rows(const float* x, const int64_t* ids, int64_t n, float* out, hipStream_t s) {
    if (n > 0) hipLaunchKernelGGL(k_gather_rows, dim3(blocks_for(n * kDim, 256)), dim3(256), 0, s, x, ids, n, out);
}

void launch_kmeans_accum(const float* xs, const int32_t* assign, int64_t n, unsigned long long* sums,
                         unsigned long long* counts, hipStream_t s) {
    if (n > 0)
        hipLaunchKernelGGL(k_kmeans_accum, dim3(blocks_for(n * kDim, 256)), dim3(256), 0, s, xs, assign, n, sums,
                           counts);
}

void launch_kmeans_normalize(const unsigned long long* sums, const unsigned long long* counts, int32_t n_c,
                             float* cen, hipStream_t s) {
    hipLaunchKernelGGL(k_kmeans_normalize, dim3(blocks_for(n_c, 64)), dim3(64), 0, s, sums, counts, n_c, cen);
}

void launch_normalize_rows(float* rows, int32_t n, hipStream_t s) {
    if (n > 0) hipLaunchKernelGGL(k_normalize_rows, dim3(blocks_for(n, 64)), dim3(64), 0, s, rows, n);
}

void launch_residuals(const float* x, const int32_t* assign, int64_t n, const float* cen, float* out,
                      hipStream_t s) {
    if (n > 0) hipLaunchKernelGGL(k_residuals, dim3(blocks_for(n * kDim, 256)), dim3(256), 0, s, x, assign, n, cen, out);
}

void launch_pick_quantiles(const float* sorted, int64_t n, int32_t nbits, float* cutoffs, float* weights,
                           hipStream_t s) {
    hipLaunchKernelGGL(k_pick_quantiles, dim3(1), dim3(256), 0, s, sorted, n, nbits, cutoffs, weights);
}

void launch_encode(int32_t nbits, const float* x, const int32_t* token_docs, const int32_t* assign,
                   const int64_t* perm, int64_t n, const float* cen, const float* cutoffs, uint8_t* codes,
                   int32_t* doc_ids, hipStream_t s) {
    const int64_t work = n * (kDim * nbits / 8);
    if (work <= 0) return;
    const dim3 grid(blocks_for(work, 256)), block(256);
    switch (nbits) {
        case 1: hipLaunchKernelGGL(k_encode<1>, grid, block, 0, s, x, token_docs, assign, perm, n, cen, cutoffs, codes, doc_ids); break;
        case 2: hipLaunchKernelGGL(k_encode<2>, grid, block, 0, s, x, token_docs, assign, perm, n, cen, cutoffs, codes, doc_ids); break;
        case 4: hipLaunchKernelGGL(k_encode<4>, grid, block, 0, s, x, token_docs, assign, perm, n, cen, cutoffs, codes, doc_ids); break;
        default: hipLaunchKernelGGL(k_encode<8>, grid, block, 0, s, x, token_docs, assign, perm, n, cen, cutoffs, codes, doc_ids); break;
    }
}

void launch_count_clusters(const int32_t* assign, int64_t n, unsigned long long* counts, hipStream_t s) {
    if (n > 0) hipLaunchKernelGGL(k_count_clusters, dim3(blocks_for(n, 256)), dim3(256), 0, s, assign, n, counts);
}

void launch_iota64(int64_t* out, int64_t n, hipStream_t s) {
    if (n > 0) hipLaunchKernelGGL(k_iota64, dim3(blocks_for(n, 256)), dim3(256), 0, s, out, n);
}

}  // namespace warp
