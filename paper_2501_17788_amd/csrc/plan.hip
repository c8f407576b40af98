// Embeddings scored per query (a debug output): the sum over its tokens of the
// sizes of their probed clusters. Also the small fill and check kernels.
#include "engine.h"

namespace warp {

__global__ __launch_bounds__(256) void k_scored(WaveArgs a) {
    const int q = blockIdx.x * 256 + threadIdx.x;
    if (q >= a.n_q) return;
    const int P = a.nprobe;
    int64_t s = 0;
    for (int i = 0; i < a.n_qtok; ++i) s += a.seg_pref[((int64_t)q * a.n_qtok + i) * (P + 1) + P];
    a.dbg_scored[q] = s;
}

void launch_scored(const WaveArgs& a, hipStream_t s) {
    if (!a.dbg_scored) return;
    hipLaunchKernelGGL(k_scored, dim3((a.n_q + 255) / 256), dim3(256), 0, s, a);
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

// Zeroes `units` 16-byte units with non-temporal stores (no L2 allocation).
__global__ __launch_bounds__(256) void k_zero16(unsigned __attribute__((ext_vector_type(4)))* p, int64_t units) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 z = {0u, 0u, 0u, 0u};
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < units; i += stride)
        __builtin_nontemporal_store(z, p + i);
}

// Zeroes n 32-bit cells from p (4-byte aligned): the 16-byte units inside the range with
// k_zero16, the cells before and after them with k_fill_i32.
void launch_zero_cells(uint32_t* p, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    int64_t head = (int64_t)((16 - ((uintptr_t)p & 15)) & 15) / 4;
    if (head > n) head = n;
    launch_fill_i32(reinterpret_cast<int32_t*>(p), head, 0, s);
    const int64_t units = (n - head) / 4;
    if (units > 0) {
        int64_t blocks = (units + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        hipLaunchKernelGGL(k_zero16, dim3((unsigned)blocks), dim3(256), 0, s,
                           reinterpret_cast<unsigned __attribute__((ext_vector_type(4)))*>(p + head), units);
    }
    launch_fill_i32(reinterpret_cast<int32_t*>(p + head + 4 * units), n - head - 4 * units, 0, s);
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

__global__ void k_doc_len(const int32_t* ids, int64_t n, int32_t* doc_len) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) atomicAdd(&doc_len[ids[i]], 1);
}

// embeddings per document (doc ids were checked to lie in [0, n_docs) on load)
void launch_doc_len(const int32_t* doc_ids, int64_t n, int32_t* doc_len, int32_t n_docs, hipStream_t s) {
    launch_fill_i32(doc_len, n_docs, 0, s);
    if (n <= 0) return;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_doc_len, dim3((unsigned)blocks), dim3(256), 0, s, doc_ids, n, doc_len);
}

}  // namespace warp
