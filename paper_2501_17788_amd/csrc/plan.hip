// Work plan of one wave of queries: the probed embeddings of query token t
// (the concatenation of its n_probe clusters) are cut into tiles of kScanTile
// embeddings; tile_start is the exclusive prefix sum of tiles over tokens, so
// the residual scan can split all tiles evenly over a persistent grid. Also
// counts the embeddings scored per query.
#include "engine.h"

namespace warp {

__global__ __launch_bounds__(1024) void k_plan(WaveArgs a) {
    constexpr int NT = 1024;
    __shared__ int64_t part[NT];
    const int n_tok = a.n_q * a.n_qtok;
    const int P = a.nprobe;
    const int tid = threadIdx.x;
    const int per = (n_tok + NT - 1) / NT;
    const int lo = tid * per < n_tok ? tid * per : n_tok;
    const int hi = lo + per < n_tok ? lo + per : n_tok;
    int64_t mine = 0;
    for (int t = lo; t < hi; ++t) {
        const int64_t n = a.seg_pref[(int64_t)t * (P + 1) + P];
        mine += (n + kScanTile - 1) / kScanTile;
    }
    part[tid] = mine;
    __syncthreads();
    for (int off = 1; off < NT; off <<= 1) {  // inclusive prefix over threads
        const int64_t v = tid >= off ? part[tid - off] : 0;
        __syncthreads();
        part[tid] += v;
        __syncthreads();
    }
    int64_t run = part[tid] - mine;
    for (int t = lo; t < hi; ++t) {
        a.tile_start[t] = run;
        const int64_t n = a.seg_pref[(int64_t)t * (P + 1) + P];
        run += (n + kScanTile - 1) / kScanTile;
    }
    if (tid == NT - 1) a.tile_start[n_tok] = part[NT - 1];
    if (a.dbg_scored) {
        for (int q = tid; q < a.n_q; q += NT) {
            int64_t s = 0;
            for (int i = 0; i < a.n_qtok; ++i)
                s += a.seg_pref[((int64_t)q * a.n_qtok + i) * (P + 1) + P];
            a.dbg_scored[q] = s;
        }
    }
}

void launch_plan(const WaveArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(k_plan, dim3(1), dim3(1024), 0, s, a);
}

__global__ void k_fill_i32(int32_t* p, int64_t n, int32_t v) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

void launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
    if (n <= 0) return;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
}

}  // namespace warp

namespace warp {

__global__ void k_check_docs(const int32_t* ids, int64_t n, int32_t n_docs, int32_t* err) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    bool bad = false;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int32_t d = ids[i];
        bad |= d < 0 || d >= n_docs;
    }
    if (bad) atomicOr(err, kErrDocRange);
}

void launch_check_docs(const int32_t* ids, int64_t n, int32_t n_docs, int32_t* err, hipStream_t s) {
    if (n <= 0) return;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(k_check_docs, dim3((unsigned)blocks), dim3(256), 0, s, ids, n, n_docs, err);
}

// One wave per query token: finite entries and norm <= 1 + 1e-3.
__global__ void k_check_queries(const float* q, int64_t n_tok, int32_t* err) {
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= n_tok) return;
    const float a = q[t * kDim + lane], b = q[t * kDim + 64 + lane];
    double s = (double)a * a + (double)b * b;
    bool bad = !(__builtin_isfinite(a) && __builtin_isfinite(b));
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    bad = __any(bad);
    if (lane == 0 && (bad || !(s <= (1.0 + 1e-3) * (1.0 + 1e-3)))) atomicOr(err, kErrQueryNorm);
}

void launch_check_queries(const float* q, int64_t n_tok, int32_t* err, hipStream_t s) {
    if (n_tok <= 0) return;
    hipLaunchKernelGGL(k_check_queries, dim3((unsigned)((n_tok + 3) / 4)), dim3(256), 0, s, q, n_tok, err);
}

}  // namespace warp
