// Cluster-major work plan of one wave of queries: every (query token, probed
// cluster) pair is bucketed by cluster (a counting sort), and each probed
// cluster is cut into work items of (kMxChunk embeddings) x (kMxGroup tokens),
// so that the residual scan reads a cluster chunk once for all the tokens that
// probe it. Pair order inside a bucket follows atomic arrival and does not
// affect results: the token-level max is exact and commutative.
#include "engine.h"

namespace warp {

// pairs of tokens whose selection overflowed carry cluster -1 and are skipped
__global__ __launch_bounds__(256) void k_pair_count(WaveArgs a) {
    const int64_t n = (int64_t)a.n_q * a.n_qtok * a.nprobe;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int c = a.sel[i];
    if (c >= 0) atomicAdd(&a.ccount[c], 1);
}

__device__ __forceinline__ int64_t cluster_items(int32_t n_tok, int32_t size) {
    if (n_tok <= 0 || size <= 0) return 0;
    return (int64_t)((size + kMxChunk - 1) / kMxChunk) * ((n_tok + kMxGroup - 1) / kMxGroup);
}

// exclusive scans of items and pairs inside each block of kPlanBlock clusters
__global__ __launch_bounds__(kPlanBlock) void k_cplan_local(WaveArgs a) {
    __shared__ int64_t si[kPlanBlock];
    __shared__ int64_t sp[kPlanBlock];
    const int tid = threadIdx.x;
    const int64_t c = (int64_t)blockIdx.x * kPlanBlock + tid;
    const bool in = c < a.n_c;
    const int32_t nt = in ? a.ccount[c] : 0;
    const int64_t items = in ? cluster_items(nt, a.sizes[c]) : 0;
    si[tid] = items;
    sp[tid] = nt;
    __syncthreads();
    for (int off = 1; off < kPlanBlock; off <<= 1) {
        const int64_t vi = tid >= off ? si[tid - off] : 0;
        const int64_t vp = tid >= off ? sp[tid - off] : 0;
        __syncthreads();
        si[tid] += vi;
        sp[tid] += vp;
        __syncthreads();
    }
    if (in) {
        a.item_start[c] = si[tid] - items;
        a.pair_start[c] = (int32_t)(sp[tid] - nt);
        a.cursor[c] = 0;
    }
    if (tid == kPlanBlock - 1) {
        a.blk[2 * blockIdx.x] = si[tid];
        a.blk[2 * blockIdx.x + 1] = sp[tid];
    }
}

// add the sums of all earlier blocks; the last block also writes the totals
__global__ __launch_bounds__(kPlanBlock) void k_cplan_add(WaveArgs a) {
    __shared__ int64_t ri[kPlanBlock];
    __shared__ int64_t rp[kPlanBlock];
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    const int nblk = gridDim.x;
    int64_t vi = 0, vp = 0;
    for (int j = tid; j < b; j += kPlanBlock) {
        vi += a.blk[2 * j];
        vp += a.blk[2 * j + 1];
    }
    ri[tid] = vi;
    rp[tid] = vp;
    __syncthreads();
    for (int off = kPlanBlock / 2; off > 0; off >>= 1) {
        if (tid < off) {
            ri[tid] += ri[tid + off];
            rp[tid] += rp[tid + off];
        }
        __syncthreads();
    }
    const int64_t oi = ri[0], op = rp[0];
    const int64_t c = (int64_t)b * kPlanBlock + tid;
    if (c < a.n_c) {
        a.item_start[c] += oi;
        a.pair_start[c] += (int32_t)op;
    }
    if (b == nblk - 1 && tid == 0) {
        a.item_start[a.n_c] = oi + a.blk[2 * b];
        a.pair_start[a.n_c] = (int32_t)(op + a.blk[2 * b + 1]);
    }
}

__global__ __launch_bounds__(256) void k_pair_scatter(WaveArgs a) {
    const int64_t n = (int64_t)a.n_q * a.n_qtok * a.nprobe;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int c = a.sel[i];
    if (c < 0) return;
    const int slot = atomicAdd(&a.cursor[c], 1);
    const int64_t p = (int64_t)a.pair_start[c] + slot;
    const int32_t tok = (int32_t)(i / a.nprobe);
    uint32_t bias, vmin;
    cell_code(a, tok / a.n_qtok, bias, vmin);
    a.plist[2 * p] = tok;                                   // wave token
    a.plist[2 * p + 1] = (int32_t)((uint32_t)a.base[i] + bias);  // R(S64) of (token, cluster) + the cell bias
}

// Probed chunks and their items (token groups of their cluster) in the index's chunk order.
__device__ __forceinline__ void chunk_items(const WaveArgs& a, int64_t j, int64_t& flag, int64_t& items) {
    flag = items = 0;
    if (j < a.n_chunks) {
        const int32_t nt = a.ccount[a.chunk_c[j]];
        items = (nt + kMxGroup - 1) / kMxGroup;
        flag = items > 0;
    }
}

// Inclusive prefix sums of two values per thread over a block of kPlanBlock threads
// (wave shuffles, then the wave totals through LDS).
__device__ __forceinline__ void block_scan2(int64_t& f, int64_t& it, int64_t* wf, int64_t* wi) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int64_t tf = __shfl_up(f, off, 64), ti = __shfl_up(it, off, 64);
        if (lane >= off) {
            f += tf;
            it += ti;
        }
    }
    if (lane == 63) {
        wf[w] = f;
        wi[w] = it;
    }
    __syncthreads();
    int64_t bf = 0, bi = 0;
    for (int i = 0; i < w; ++i) {
        bf += wf[i];
        bi += wi[i];
    }
    f += bf;
    it += bi;
}

// per block of kPlanBlock chunks: the number of probed chunks and their items
__global__ __launch_bounds__(kPlanBlock) void k_chunk_count(WaveArgs a) {
    __shared__ int64_t wf[kPlanBlock / 64], wi[kPlanBlock / 64];
    int64_t f, it;
    chunk_items(a, (int64_t)blockIdx.x * kPlanBlock + threadIdx.x, f, it);
    block_scan2(f, it, wf, wi);
    if (threadIdx.x == kPlanBlock - 1) {
        a.cblk[2 * blockIdx.x] = f;
        a.cblk[2 * blockIdx.x + 1] = it;
    }
}

// the compacted list of probed chunks with the exclusive prefix of their items
__global__ __launch_bounds__(kPlanBlock) void k_chunk_list(WaveArgs a) {
    __shared__ int64_t wf[kPlanBlock / 64], wi[kPlanBlock / 64];
    __shared__ unsigned long long s_of, s_oi;
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    if (tid == 0) {
        s_of = 0;
        s_oi = 0;
    }
    __syncthreads();
    {  // offsets of this block: the sums of the blocks before it
        int64_t vf = 0, vi = 0;
        for (int j = tid; j < b; j += kPlanBlock) {
            vf += a.cblk[2 * j];
            vi += a.cblk[2 * j + 1];
        }
        if (vf) atomicAdd(&s_of, (unsigned long long)vf);
        if (vi) atomicAdd(&s_oi, (unsigned long long)vi);
    }
    const int64_t j = (int64_t)b * kPlanBlock + tid;
    int64_t f0, it0;
    chunk_items(a, j, f0, it0);
    int64_t f = f0, it = it0;
    block_scan2(f, it, wf, wi);  // its barrier also orders the offsets above
    const int64_t pos = (int64_t)s_of + f - f0, item = (int64_t)s_oi + it - it0;
    if (f0) {
        const int c = a.chunk_c[j];
        const int64_t e0 = a.offsets[c] + (int64_t)a.chunk_k[j] * kMxChunk;
        const int64_t e1 = a.offsets[c + 1];
        const int64_t len = e1 - e0 < kMxChunk ? e1 - e0 : kMxChunk;  // 1 .. kMxChunk
        const uint64_t ew = (uint64_t)e0 | ((uint64_t)len << kRecLenShift);
        a.list_rec[pos] = make_int4((int)(uint32_t)ew, (int)(uint32_t)(ew >> 32), a.pair_start[c], a.ccount[c]);
        a.list_item[pos] = item;
    }
    if (b == (int)gridDim.x - 1 && tid == kPlanBlock - 1) {
        *a.list_n = (int64_t)s_of + f;
        a.list_item[(int64_t)s_of + f] = (int64_t)s_oi + it;
    }
}

void launch_pairing(const WaveArgs& a, hipStream_t s) {
    const int64_t n = (int64_t)a.n_q * a.n_qtok * a.nprobe;
    const unsigned pb = (unsigned)((n + 255) / 256);
    const unsigned nblk = (unsigned)((a.n_c + kPlanBlock - 1) / kPlanBlock);
    // (the token counters were zeroed by the wave's preparation)
    hipLaunchKernelGGL(k_pair_count, dim3(pb), dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_cplan_local, dim3(nblk), dim3(kPlanBlock), 0, s, a);
    hipLaunchKernelGGL(k_cplan_add, dim3(nblk), dim3(kPlanBlock), 0, s, a);
    hipLaunchKernelGGL(k_pair_scatter, dim3(pb), dim3(256), 0, s, a);
    const unsigned cb = (unsigned)((a.n_chunks + kPlanBlock - 1) / kPlanBlock);
    if (cb == 0) {  // an index without embeddings: no chunk, no item
        launch_fill_i32(reinterpret_cast<int32_t*>(a.list_n), 2, 0, s);
        launch_fill_i32(reinterpret_cast<int32_t*>(a.list_item), 2, 0, s);
        return;
    }
    hipLaunchKernelGGL(k_chunk_count, dim3(cb), dim3(kPlanBlock), 0, s, a);
    hipLaunchKernelGGL(k_chunk_list, dim3(cb), dim3(kPlanBlock), 0, s, a);
}

}  // namespace warp
