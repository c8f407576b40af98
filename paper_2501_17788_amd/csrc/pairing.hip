// Cluster-major work plan of one wave of queries: every (query token, probed
// cluster) pair is bucketed by cluster (a counting sort whose counts the selection
// takes), and each probed cluster is cut into work items of (kMxChunk embeddings) x
// (kMxGroup tokens), so that the residual scan reads a cluster chunk once for all the
// tokens that probe it. Pair order inside a bucket follows atomic arrival and does not
// affect results: the token-level max is exact and commutative. Three launches: block
// sums of the counts (with the pair offsets inside each block of clusters), their
// prefixes, then the buckets and the lists of probed chunks.
#include "engine.h"

namespace warp {

constexpr int kPairPer = kPairBlock / kPlanBlock;  // clusters per thread of the pair offsets
static_assert(kPairPer % 4 == 0 && kPairBlock == kPairPer * kPlanBlock, "pair offset blocks");

// Block b of kPairBlock clusters: the exclusive prefix of their probing-token counts inside
// the block (thread tid takes kPairPer consecutive clusters) and the block's total, coff[b].
__device__ void pair_offsets(const WaveArgs& a, int64_t b, int64_t* ws) {
    constexpr int NW = kPlanBlock / 64;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t n_c = a.n_c;
    const int64_t cb = b * kPairBlock + (int64_t)tid * kPairPer;
    int32_t v[kPairPer];
    const bool whole = cb + kPairPer <= n_c;  // 16-byte aligned: cb is a multiple of kPairPer
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
    int32_t run = (int32_t)(before + x - sum);
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
    if (tid == 0) a.coff[b] = total;
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

// Block totals of one value per thread turned into exclusive prefixes in place (n values at
// stride `stride`), in passes of kPlanBlock; returns the sum of all.
__device__ int64_t block_prefix_inplace(int64_t* v, int64_t n, int stride, int64_t* ws) {
    constexpr int NW = kPlanBlock / 64;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    int64_t carry = 0;
    for (int64_t i0 = 0; i0 < n; i0 += kPlanBlock) {  // uniform
        const int64_t i = i0 + tid;
        const int64_t x0 = i < n ? v[i * stride] : 0;
        int64_t x = x0;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int64_t t = __shfl_up(x, off, 64);
            if (lane >= off) x += t;
        }
        if (lane == 63) ws[w] = x;
        __syncthreads();
        int64_t before = 0, total = 0;
#pragma unroll
        for (int k = 0; k < NW; ++k) {
            before += k < w ? ws[k] : 0;
            total += ws[k];
        }
        if (i < n) v[i * stride] = carry + before + x - x0;
        carry += total;
        __syncthreads();  // ws is free for the next pass
    }
    return carry;
}

// Blocks [0, ncb): the pair offsets of a block of kPairBlock clusters. Blocks ncb ..: per block
// of kPlanBlock chunks, the number of probed chunks and their items.
__global__ __launch_bounds__(kPlanBlock) void k_plan_count(WaveArgs a, int32_t ncb) {
    __shared__ int64_t wf[kPlanBlock / 64], wi[kPlanBlock / 64], wn[kPlanBlock / 64];
    const int tid = threadIdx.x;
    if ((int)blockIdx.x < ncb) {
        pair_offsets(a, blockIdx.x, wf);
    } else {
        const int64_t b = (int64_t)blockIdx.x - ncb;
        int64_t f, it, nr;
        chunk_items(a, b * kPlanBlock + tid, f, it, nr);
        block_scan3(f, it, nr, wf, wi, wn);
        if (tid == kPlanBlock - 1) {
            a.cblk[3 * b] = f;
            a.cblk[3 * b + 1] = it;
            a.cblk[3 * b + 2] = nr;
        }
    }
}

// One workgroup: the block sums of the count kernel turned into exclusive prefixes (so that
// every block of the emit kernel reads its offsets directly) and the lists' lengths.
__global__ __launch_bounds__(kPlanBlock) void k_plan_prefix(WaveArgs a, int32_t ncb, int32_t cb) {
    constexpr int NW = kPlanBlock / 64;
    __shared__ int64_t wf[NW], wi[NW], wn[NW];
    const int tid = threadIdx.x;
    int64_t cf = 0, ci = 0, cn = 0;  // totals of the passes before
    for (int64_t b0 = 0; b0 < cb; b0 += kPlanBlock) {  // uniform
        const int64_t b = b0 + tid;
        const bool in = b < cb;
        const int64_t f0 = in ? a.cblk[3 * b] : 0, i0 = in ? a.cblk[3 * b + 1] : 0, n0 = in ? a.cblk[3 * b + 2] : 0;
        int64_t f = f0, it = i0, nr = n0;
        block_scan3(f, it, nr, wf, wi, wn);
        if (in) {
            a.cblk[3 * b] = cf + f - f0;
            a.cblk[3 * b + 1] = ci + it - i0;
            a.cblk[3 * b + 2] = cn + nr - n0;
        }
        int64_t tf = 0, ti = 0, tn = 0;
#pragma unroll
        for (int k = 0; k < NW; ++k) {
            tf += wf[k];
            ti += wi[k];
            tn += wn[k];
        }
        cf += tf;
        ci += ti;
        cn += tn;
        __syncthreads();  // the wave totals are free for the next pass
    }
    (void)block_prefix_inplace(a.coff, ncb, 1, wf);
    if (tid == 0) {
        *a.list_n = cf;
        a.list_item[cf] = ci;
        *a.list_n2 = cn;
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
    const int64_t p = a.coff[c / kPairBlock] + a.pair_start[c] + slot;
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
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    if (b >= cb) {  // uniform over the block
        pair_scatter(a, (int64_t)(b - cb) * kPlanBlock + tid);
        return;
    }
    // this block's offsets: the chunks and items of the blocks before it
    const int64_t of = a.cblk[3 * b], oi = a.cblk[3 * b + 1], on = a.cblk[3 * b + 2];
    const int64_t j = (int64_t)b * kPlanBlock + tid;
    int64_t f0, it0, n0;
    chunk_items(a, j, f0, it0, n0);
    int64_t f = f0, it = it0, nr = n0;
    block_scan3(f, it, nr, wf, wi, wn);
    if (f0 || n0) {
        const int c = a.chunk_c[j];
        const int64_t e0 = a.offsets[c] + (int64_t)a.chunk_k[j] * kMxChunk;
        const int64_t e1 = a.offsets[c + 1];
        const int64_t len = e1 - e0 < kMxChunk ? e1 - e0 : kMxChunk;  // 1 .. kMxChunk
        const uint64_t ew = (uint64_t)e0 | ((uint64_t)len << kRecLenShift);
        const int first = (int)(a.coff[c / kPairBlock] + a.pair_start[c]);
        const int4 rec = make_int4((int)(uint32_t)ew, (int)(uint32_t)(ew >> 32), first, a.ccount[c]);
        if (f0) {
            const int64_t pos = of + f - f0;
            a.list_rec[pos] = rec;
            a.list_item[pos] = oi + it - it0;
        } else {
            a.list_rec2[on + nr - n0] = rec;
        }
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
    const unsigned ncb = (unsigned)((a.n_c + kPairBlock - 1) / kPairBlock);
    hipLaunchKernelGGL(k_plan_count, dim3(ncb + cb), dim3(kPlanBlock), 0, s, a, (int32_t)ncb);
    hipLaunchKernelGGL(k_plan_prefix, dim3(1), dim3(kPlanBlock), 0, s, a, (int32_t)ncb, (int32_t)cb);
    hipLaunchKernelGGL(k_plan_emit, dim3(cb + pb), dim3(kPlanBlock), 0, s, a, (int32_t)cb);
}

}  // namespace warp
