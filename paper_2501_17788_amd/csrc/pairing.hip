// Cluster-major work plan of one wave of queries: every (query token, probed
// cluster) pair is bucketed by cluster (a counting sort whose counts the selection
// takes), and each probed cluster is cut into work items of (kMxChunk embeddings) x
// (kMxGroup tokens), so that the residual scan reads a cluster chunk once for all the
// tokens that probe it. Pair order inside a bucket follows atomic arrival and does not
// affect results: the token-level max is exact and commutative. Two launches: the
// counts' prefix sums, then the buckets and the list of probed chunks.
#include "engine.h"

namespace warp {

constexpr int kPairPer = 32;  // clusters per thread and pass of the pair offsets

// The exclusive prefix of the clusters' probing-token counts (each cluster's first pair in
// the bucketed list), by one workgroup of kPlanBlock threads: per pass, thread tid takes
// kPairPer consecutive clusters, and the pass's running total carries to the next.
__device__ void pair_offsets(const WaveArgs& a, int64_t* ws) {
    constexpr int NW = kPlanBlock / 64;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t n_c = a.n_c;
    int64_t carry = 0;
    for (int64_t c0 = 0; c0 < n_c; c0 += (int64_t)kPlanBlock * kPairPer) {  // uniform
        const int64_t cb = c0 + (int64_t)tid * kPairPer;
        int32_t v[kPairPer];
        const bool whole = cb + kPairPer <= n_c;  // 16-byte aligned: cb is a multiple of 32
        if (whole) {
            const int4* src = reinterpret_cast<const int4*>(a.ccount + cb);
#pragma unroll
            for (int j = 0; j < kPairPer / 4; ++j) {
                const int4 x = src[j];
                v[4 * j] = x.x;
                v[4 * j + 1] = x.y;
                v[4 * j + 2] = x.z;
                v[4 * j + 3] = x.w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < kPairPer; ++j) v[j] = cb + j < n_c ? a.ccount[cb + j] : 0;
        }
        int64_t sum = 0;
#pragma unroll
        for (int j = 0; j < kPairPer; ++j) sum += v[j];
        int64_t x = sum;  // inclusive scan of the threads' sums
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int64_t t = __shfl_up(x, off, 64);
            if (lane >= off) x += t;
        }
        if (lane == 63) ws[w] = x;
        __syncthreads();
        int64_t before = 0, total = 0;
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            before += i < w ? ws[i] : 0;
            total += ws[i];
        }
        __syncthreads();  // ws is free for the next pass
        int32_t run = (int32_t)(carry + before + x - sum);
        if (whole) {
            int4* dst = reinterpret_cast<int4*>(a.pair_start + cb);
#pragma unroll
            for (int j = 0; j < kPairPer / 4; ++j) {
                int4 o;
                o.x = run;
                o.y = o.x + v[4 * j];
                o.z = o.y + v[4 * j + 1];
                o.w = o.z + v[4 * j + 2];
                run = o.w + v[4 * j + 3];
                dst[j] = o;
            }
        } else {
#pragma unroll
            for (int j = 0; j < kPairPer; ++j) {
                if (cb + j < n_c) a.pair_start[cb + j] = run;
                run += v[j];
            }
        }
        carry += total;
    }
    if (tid == 0) a.pair_start[n_c] = (int32_t)carry;
}

// Probed chunks in the index's chunk order: a chunk probed by more than narrow_max tokens
// goes to the wide scan with its items (token groups of its cluster), one probed by
// 1..narrow_max tokens to the narrow scan.
__device__ __forceinline__ void chunk_items(const WaveArgs& a, int64_t j, int64_t& flag, int64_t& items,
                                            int64_t& narrow) {
    flag = items = narrow = 0;
    if (j < a.n_chunks) {
        const int32_t nt = a.ccount[a.chunk_c[j]];
        if (nt > a.narrow_max) {
            items = (nt + kMxGroup - 1) / kMxGroup;
            flag = 1;
        } else {
            narrow = nt > 0;
        }
    }
}

// Inclusive prefix sums of three values per thread over a block of kPlanBlock threads
// (wave shuffles, then the wave totals through LDS).
__device__ __forceinline__ void block_scan3(int64_t& f, int64_t& it, int64_t& nr, int64_t* wf, int64_t* wi,
                                            int64_t* wn) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int64_t tf = __shfl_up(f, off, 64), ti = __shfl_up(it, off, 64), tn = __shfl_up(nr, off, 64);
        if (lane >= off) {
            f += tf;
            it += ti;
            nr += tn;
        }
    }
    if (lane == 63) {
        wf[w] = f;
        wi[w] = it;
        wn[w] = nr;
    }
    __syncthreads();
    int64_t bf = 0, bi = 0, bn = 0;
    for (int i = 0; i < w; ++i) {
        bf += wf[i];
        bi += wi[i];
        bn += wn[i];
    }
    f += bf;
    it += bi;
    nr += bn;
}

// Block 0: the clusters' pair offsets. Blocks 1 ..: per block of kPlanBlock chunks, the
// number of probed chunks and their items.
__global__ __launch_bounds__(kPlanBlock) void k_plan_count(WaveArgs a) {
    __shared__ int64_t wf[kPlanBlock / 64], wi[kPlanBlock / 64], wn[kPlanBlock / 64];
    if (blockIdx.x == 0) {
        pair_offsets(a, wf);
        return;
    }
    const int64_t b = (int64_t)blockIdx.x - 1;
    int64_t f, it, nr;
    chunk_items(a, b * kPlanBlock + threadIdx.x, f, it, nr);
    block_scan3(f, it, nr, wf, wi, wn);
    if (threadIdx.x == kPlanBlock - 1) {
        a.cblk[3 * b] = f;
        a.cblk[3 * b + 1] = it;
        a.cblk[3 * b + 2] = nr;
    }
}

// Every (token, probed cluster) pair placed in its cluster's bucket: the wave token and the
// token's centroid term R(S64) plus its query's cell bias. Pairs of tokens whose selection
// overflowed carry cluster -1 and are skipped.
__device__ __forceinline__ void pair_scatter(const WaveArgs& a, int64_t i) {
    const int64_t n = (int64_t)a.n_q * a.n_qtok * a.nprobe;
    if (i >= n) return;
    const int c = a.sel[i];
    if (c < 0) return;
    const int slot = atomicAdd(&a.cursor[c], 1);
    const int64_t p = (int64_t)a.pair_start[c] + slot;
    const int32_t tok = (int32_t)(i / a.nprobe);
    uint32_t bias, vmin;
    cell_code(a, tok / a.n_qtok, bias, vmin);
    a.plist[2 * p] = tok;
    a.plist[2 * p + 1] = (int32_t)((uint32_t)a.base[i] + bias);
}

// Blocks [0, cb): the compacted lists of probed chunks (wide, with the exclusive prefix of
// their items, and narrow). Blocks [cb, ...): the pairs, kPlanBlock per block, scattered
// into their buckets.
__global__ __launch_bounds__(kPlanBlock) void k_plan_emit(WaveArgs a, int32_t cb) {
    __shared__ int64_t wf[kPlanBlock / 64], wi[kPlanBlock / 64], wn[kPlanBlock / 64];
    __shared__ unsigned long long s_of, s_oi, s_on;
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    if (b >= cb) {  // uniform over the block
        pair_scatter(a, (int64_t)(b - cb) * kPlanBlock + tid);
        return;
    }
    if (tid == 0) {
        s_of = 0;
        s_oi = 0;
        s_on = 0;
    }
    __syncthreads();
    {  // offsets of this block: the sums of the blocks before it
        int64_t vf = 0, vi = 0, vn = 0;
        for (int j = tid; j < b; j += kPlanBlock) {
            vf += a.cblk[3 * j];
            vi += a.cblk[3 * j + 1];
            vn += a.cblk[3 * j + 2];
        }
        if (vf) atomicAdd(&s_of, (unsigned long long)vf);
        if (vi) atomicAdd(&s_oi, (unsigned long long)vi);
        if (vn) atomicAdd(&s_on, (unsigned long long)vn);
    }
    const int64_t j = (int64_t)b * kPlanBlock + tid;
    int64_t f0, it0, n0;
    chunk_items(a, j, f0, it0, n0);
    int64_t f = f0, it = it0, nr = n0;
    block_scan3(f, it, nr, wf, wi, wn);  // its barrier also orders the offsets above
    if (f0 || n0) {
        const int c = a.chunk_c[j];
        const int64_t e0 = a.offsets[c] + (int64_t)a.chunk_k[j] * kMxChunk;
        const int64_t e1 = a.offsets[c + 1];
        const int64_t len = e1 - e0 < kMxChunk ? e1 - e0 : kMxChunk;  // 1 .. kMxChunk
        const uint64_t ew = (uint64_t)e0 | ((uint64_t)len << kRecLenShift);
        const int4 rec = make_int4((int)(uint32_t)ew, (int)(uint32_t)(ew >> 32), a.pair_start[c], a.ccount[c]);
        if (f0) {
            const int64_t pos = (int64_t)s_of + f - f0;
            a.list_rec[pos] = rec;
            a.list_item[pos] = (int64_t)s_oi + it - it0;
        } else {
            a.list_rec2[(int64_t)s_on + nr - n0] = rec;
        }
    }
    if (b == cb - 1 && tid == kPlanBlock - 1) {
        *a.list_n = (int64_t)s_of + f;
        a.list_item[(int64_t)s_of + f] = (int64_t)s_oi + it;
        *a.list_n2 = (int64_t)s_on + nr;
    }
}

void launch_pairing(const WaveArgs& a, hipStream_t s) {
    // (the wave's preparation zeroed the token counters and cursors; the selection counted)
    const unsigned cb = (unsigned)((a.n_chunks + kPlanBlock - 1) / kPlanBlock);
    if (cb == 0) {  // an index without embeddings: no chunk, no item, no pair is read
        launch_fill_i32(reinterpret_cast<int32_t*>(a.list_n), 2, 0, s);
        launch_fill_i32(reinterpret_cast<int32_t*>(a.list_n2), 2, 0, s);
        launch_fill_i32(reinterpret_cast<int32_t*>(a.list_item), 2, 0, s);
        return;
    }
    const int64_t n = (int64_t)a.n_q * a.n_qtok * a.nprobe;
    const unsigned pb = (unsigned)((n + kPlanBlock - 1) / kPlanBlock);
    hipLaunchKernelGGL(k_plan_count, dim3(1 + cb), dim3(kPlanBlock), 0, s, a);
    hipLaunchKernelGGL(k_plan_emit, dim3(cb + pb), dim3(kPlanBlock), 0, s, a, (int32_t)cb);
}

}  // namespace warp
