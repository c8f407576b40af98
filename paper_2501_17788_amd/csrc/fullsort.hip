// Exact paths for requests beyond what the selection and top-k kernels hold in LDS
// (n_probe above kMaxProbe, k above kMaxK, and a selection band of more than kSelCap
// centroids in the blocking search's retry): whole score lists are sorted with the device
// radix sort, which gives the definitions of Sections 4.3 and 4.5 directly.
//
// Selection (Section 4.3): every (token, centroid) score S64 in
// fp64 (dimension order, as everywhere), sorted per token into (score desc, id asc) order
// (a 64-bit key sort, then a stable sort by token); then, per token, the n_probe first
// centroids, their fixed-point scores and size prefix, and m_i = the score of the first
// entry whose inclusive cumulative size exceeds t' (the last entry when none does).
//
// Top-k (Section 4.5) for k > kMaxK: every document key of the query (the fold's, larger
// is better, 0 for a non-candidate) sorted in descending order; the first min(k, #candidates)
// are decoded.
#include <algorithm>

#include "engine.h"

namespace warp {

hipError_t sort_u64(void* temp, size_t* temp_bytes, const uint64_t* keys_in, uint64_t* keys_out,
                    const int64_t* vals_in, int64_t* vals_out, int64_t n, int end_bit, hipStream_t s);
hipError_t sort_u32(void* temp, size_t* temp_bytes, const uint32_t* keys_in, uint32_t* keys_out,
                    const int64_t* vals_in, int64_t* vals_out, int64_t n, int end_bit, hipStream_t s);
size_t sort_u64_temp_bytes(int64_t n, bool vals);
size_t sort_u32_temp_bytes(int64_t n, bool vals);

static size_t al256(size_t b) { return (b + 255) & ~(size_t)255; }

// ascending order of these keys is (score desc); S64 is never -0.0 (its sum starts at +0.0)
__device__ __forceinline__ uint64_t desc_key(double x) {
    uint64_t b = (uint64_t)__double_as_longlong(x);
    b = (b >> 63) ? ~b : (b | (1ull << 63));
    return ~b;
}
__device__ __forceinline__ double desc_key_value(uint64_t k) {
    const uint64_t b = ~k;
    return __longlong_as_double((long long)((b >> 63) ? (b & ~(1ull << 63)) : ~b));
}

// keys[t n_c + c] = desc_key(S64(token t, centroid c)), vals = t n_c + c
__global__ __launch_bounds__(256) void k_score_keys(const float* __restrict__ q, const float* __restrict__ cen,
                                                    int64_t n_tok, int32_t n_c, uint64_t* __restrict__ keys,
                                                    int64_t* __restrict__ vals) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n_tok * n_c) return;
    const int64_t t = i / n_c;
    const int32_t c = (int32_t)(i - t * n_c);
    const float* x = q + t * kDim;
    const float* y = cen + (int64_t)c * kDim;
    double s = 0.0;
    for (int d = 0; d < kDim; ++d) s = __builtin_fma((double)y[d], (double)x[d], s);  // products are exact
    keys[i] = desc_key(s);
    vals[i] = i;
}

// token of each sorted entry, the key of the second (stable) sort
__global__ void k_token_keys(const int64_t* __restrict__ vals, int64_t n, int32_t n_c, uint32_t* __restrict__ tk) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) tk[i] = (uint32_t)(vals[i] / n_c);
}

constexpr int kWalkThreads = 512;

// block-wide inclusive prefix of one int64 per thread, plus the block total
__device__ int64_t walk_scan(int64_t v, int64_t* s_w, int64_t& total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int64_t t = __shfl_up(v, off, 64);
        if (lane >= off) v += t;
    }
    if (lane == 63) s_w[w] = v;
    __syncthreads();
    int64_t before = 0;
    total = 0;
#pragma unroll
    for (int i = 0; i < kWalkThreads / 64; ++i) {
        before += i < w ? s_w[i] : 0;
        total += s_w[i];
    }
    __syncthreads();
    return before + v;
}

// One workgroup per wave token over its n_c entries in (score desc, id asc) order (vals: the
// entries' original positions t n_c + c, grouped by token; keys: the score keys at those
// original positions): the selection's outputs as k_select writes them.
__global__ __launch_bounds__(kWalkThreads) void k_select_walk(WaveArgs a, const uint64_t* __restrict__ keys,
                                                              const int64_t* __restrict__ vals) {
    __shared__ int64_t s_w[kWalkThreads / 64];
    __shared__ int s_cross;
    const int t = blockIdx.x, tid = threadIdx.x;
    const int n_c = a.n_c, P = a.nprobe;
    const int64_t* v = vals + (int64_t)t * n_c;
    int32_t* sel = a.sel + (int64_t)t * P;
    int32_t* base = a.base + (int64_t)t * P;
    int64_t* seg_pref = a.seg_pref + (int64_t)t * (P + 1);
    const int64_t tp = a.t_prime;
    if (tid == 0) {
        s_cross = -1;
        seg_pref[0] = 0;
    }
    __syncthreads();
    int64_t carry = 0;  // cumulative size before this tile
    bool crossed = false;
    for (int p0 = 0; p0 < n_c; p0 += kWalkThreads) {  // uniform
        const int p = p0 + tid;
        const bool in = p < n_c;
        const int c = in ? (int)(v[p] % n_c) : 0;
        const int64_t sz = in ? a.sizes[c] : 0;
        int64_t total;
        const int64_t incl = walk_scan(sz, s_w, total) + carry;
        if (in && p < P) {
            sel[p] = c;
            base[p] = (int32_t)__builtin_rint(desc_key_value(keys[v[p]]) * (double)(1 << kFrac));
            seg_pref[p + 1] = incl;
            atomicAdd(&a.ccount[c], 1);
            if (a.dbg_sel) a.dbg_sel[(int64_t)t * P + p] = c;
        }
        if (!crossed && in && incl > tp && incl - sz <= tp) s_cross = p;  // the first entry past t'
        __syncthreads();
        crossed = s_cross >= 0;
        carry += total;
        if (crossed && p0 + kWalkThreads >= P) break;  // uniform: selection done and m_i found
    }
    if (tid == 0) {
        const int pc = s_cross >= 0 ? s_cross : n_c - 1;  // none exceeds t': the lowest score
        const int64_t m = (int64_t)__builtin_rint(desc_key_value(keys[v[pc]]) * (double)(1 << kFrac));
        a.m_fixed[t] = m;
        if (a.dbg_m) a.dbg_m[t] = m;
    }
}

// Sort scratch of the exact selection of n_tok tokens: keys and values twice, the token
// keys twice, and the sorts' temporary storage, in 256-byte aligned pieces; returns the bytes.
size_t select_full_bytes(int64_t n_tok, int32_t n_c) {
    const int64_t n = n_tok * n_c;
    const size_t t = std::max(sort_u64_temp_bytes(n, true), sort_u32_temp_bytes(n, true));
    return 2 * al256((size_t)n * 8) + 2 * al256((size_t)n * 8) + 2 * al256((size_t)n * 4) + al256(t);
}

hipError_t launch_select_full(const WaveArgs& a, void* scratch, hipStream_t s) {
    const int64_t n_tok = (int64_t)a.n_q * a.n_qtok, n = n_tok * a.n_c;
    char* p = (char*)scratch;
    uint64_t* k0 = (uint64_t*)p; p += al256((size_t)n * 8);
    uint64_t* k1 = (uint64_t*)p; p += al256((size_t)n * 8);
    int64_t* v0 = (int64_t*)p; p += al256((size_t)n * 8);
    int64_t* v1 = (int64_t*)p; p += al256((size_t)n * 8);
    uint32_t* t0 = (uint32_t*)p; p += al256((size_t)n * 4);
    uint32_t* t1 = (uint32_t*)p; p += al256((size_t)n * 4);
    void* temp = p;
    const unsigned g = (unsigned)((n + 255) / 256);
    hipLaunchKernelGGL(k_score_keys, dim3(g), dim3(256), 0, s, a.queries, a.centroids, n_tok, a.n_c, k0, v0);
    size_t tb = 0;
    hipError_t e = sort_u64(temp, &tb, k0, k1, v0, v1, n, 64, s);  // (score desc), ties in (token, id) order
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_token_keys, dim3(g), dim3(256), 0, s, v1, n, a.n_c, t0);
    int bits = 1;
    while (bits < 32 && ((int64_t)1 << bits) < n_tok) ++bits;
    e = sort_u32(temp, &tb, t0, t1, v1, v0, n, bits, s);  // stable by token
    if (e != hipSuccess) return e;
    // the keys in the final order: the sorted values index the score keys of the first sort
    // (k0 still holds them in their original positions)
    hipLaunchKernelGGL(k_select_walk, dim3((unsigned)n_tok), dim3(kWalkThreads), 0, s, a, (const uint64_t*)k0,
                       (const int64_t*)v0);
    return hipGetLastError();
}

__global__ void k_neg_keys(const uint64_t* __restrict__ keys, int64_t n, uint64_t* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) out[i] = ~keys[i];
}

// outputs of wave query q from its keys in descending order (stored complemented, ascending)
__global__ void k_topk_sorted(WaveArgs a, const uint64_t* __restrict__ nk, int q) {
    const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (r >= a.k) return;
    const uint64_t key = r < a.n_docs ? ~nk[r] : 0ull;
    const int64_t o = (int64_t)q * a.k + r;
    if (key != 0) {
        const int64_t score = (int64_t)(key >> 24) - (1ll << 39);
        a.out_ids[o] = (int32_t)(kMaxDocs - 1 - (int32_t)(key & (kMaxDocs - 1)));
        a.out_scores[o] = (float)((double)score * (1.0 / (double)(1 << kFrac)));
        if (a.out_fixed) a.out_fixed[o] = score;
    } else {
        a.out_ids[o] = -1;
        a.out_scores[o] = -__builtin_inff();
        if (a.out_fixed) a.out_fixed[o] = INT64_MIN;
    }
    // the candidates form a prefix: the count is the position of the first non-candidate
    const uint64_t next = r + 1 < a.k && r + 1 < a.n_docs ? ~nk[r + 1] : 0ull;
    if (a.out_counts && ((r == 0 && key == 0) || (key != 0 && next == 0))) a.out_counts[q] = key ? (int32_t)(r + 1) : 0;
}

size_t topk_full_bytes(int32_t n_docs) {
    return 2 * al256((size_t)n_docs * 8) + al256(sort_u64_temp_bytes(n_docs, false));
}

hipError_t launch_topk_full(const WaveArgs& a, void* scratch, hipStream_t s) {
    const int64_t nd = a.n_docs;
    uint64_t* x = (uint64_t*)scratch;
    uint64_t* y = (uint64_t*)((char*)scratch + al256((size_t)nd * 8));
    void* temp = (char*)scratch + 2 * al256((size_t)nd * 8);
    const unsigned g = (unsigned)((nd + 255) / 256), gk = (unsigned)((a.k + 255) / 256);
    for (int q = 0; q < a.n_q; ++q) {
        hipLaunchKernelGGL(k_neg_keys, dim3(g), dim3(256), 0, s, a.keys + (int64_t)q * nd, nd, x);
        size_t tb = 0;
        const hipError_t e = sort_u64(temp, &tb, x, y, nullptr, nullptr, nd, 64, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_topk_sorted, dim3(gk), dim3(256), 0, s, a, (const uint64_t*)y, q);
    }
    return hipGetLastError();
}

}  // namespace warp
