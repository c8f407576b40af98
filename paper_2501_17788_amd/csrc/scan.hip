// Implicit decompression and token-level max (Sections 4.4 and 4.5).
//
// For query token i and every embedding e of its n_probe clusters c:
//     t = R(S64[i][c]) + sum_d R(q_{i,d} * omega[code_{e,d}])        (int32, exact)
// followed by r_tok: tokmax[i][doc(e)] = max over the probed embeddings of doc(e).
//
// The per-token table upsilon = q_hat x omega_hat (Section 4.4) is held in LDS as
// a byte-indexed table: entry [p][v] is the sum of the per-dimension entries of
// the 8 / b dimensions packed in code byte p when that byte has value v. An
// embedding then costs one table lookup per code byte (64 for b = 4, 32 for
// b = 2) and no multiplication; the integer sums are the same as per dimension.
//
// Work split: the probed embeddings of token i, clusters concatenated in
// selection order, are cut into tiles (plan kernel); a persistent grid takes
// equal contiguous ranges of the tile list, so a workgroup rebuilds its table
// only when its range crosses into the next token. One embedding per lane:
// consecutive lanes read consecutive code rows (16-byte loads) and document
// ids. Embeddings of a cluster are sorted by document, so equal documents sit
// in adjacent lanes: a wave-level segmented max leaves the run maximum in the
// run's last lane (the inner-cluster max), which alone issues atomicMax. Integer
// max is exact and commutative, so runs split across lanes, waves, tiles or
// clusters need no further ordering.
#include "engine.h"

namespace warp {

template <int NBITS>
__global__ __launch_bounds__(kScanBlock) void k_scan(WaveArgs a) {
    constexpr int NB = 1 << NBITS;
    constexpr int BYTES = kDim * NBITS / 8;  // code bytes per embedding
    constexpr int VEC = BYTES / 16;          // 16-byte loads per embedding
    __shared__ int lut[BYTES * 256];
    __shared__ int v1[kDim * NB];
    __shared__ int64_t s_pref[kMaxProbe + 1];
    __shared__ int64_t s_start[kMaxProbe];
    __shared__ int s_base[kMaxProbe];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int P = a.nprobe;
    const int n_tok = a.n_q * a.n_qtok;
    const int64_t* tile_start = a.tile_start;
    const int64_t total = tile_start[n_tok];
    const int64_t G = gridDim.x;
    int64_t tile = total * blockIdx.x / G;
    const int64_t last = total * (blockIdx.x + 1) / G;
    if (tile >= last) return;

    // token owning the first tile: tile_start[t] <= tile < tile_start[t + 1]
    int lo = 0, hi = n_tok;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (tile_start[mid] <= tile) lo = mid;
        else hi = mid;
    }
    int t = lo;
    int cur = -1;
    const uint8_t* __restrict__ codes = a.codes;
    const int32_t* __restrict__ doc_ids = a.doc_ids;

    while (tile < last) {
        while (tile_start[t + 1] <= tile) ++t;
        if (t != cur) {
            __syncthreads();  // previous token's table no longer read
            const float* q = a.queries + (int64_t)t * kDim;
            for (int x = tid; x < kDim * NB; x += kScanBlock) {
                const int d = x / NB, b = x % NB;
                v1[x] = (int)__builtin_rint((double)q[d] * (double)a.weights[b] * (double)(1 << kFrac));
            }
            if (tid < P) {
                s_base[tid] = a.base[(int64_t)t * P + tid];
                s_start[tid] = a.seg_start[(int64_t)t * P + tid];
            }
            if (tid <= P) s_pref[tid] = a.seg_pref[(int64_t)t * (P + 1) + tid];
            __syncthreads();
            for (int x = tid; x < BYTES * 256; x += kScanBlock) {
                const int p = x >> 8, v = x & 255;
                int s;
                if (NBITS == 4) {
                    s = v1[(2 * p) * 16 + (v >> 4)] + v1[(2 * p + 1) * 16 + (v & 15)];
                } else {
                    s = v1[(4 * p) * 4 + (v >> 6)] + v1[(4 * p + 1) * 4 + ((v >> 4) & 3)] +
                        v1[(4 * p + 2) * 4 + ((v >> 2) & 3)] + v1[(4 * p + 3) * 4 + (v & 3)];
                }
                lut[x] = s;
            }
            __syncthreads();
            cur = t;
        }
        const int64_t n_emb = s_pref[P];
        const int64_t t_first = tile_start[t];
        const int64_t stop = last < tile_start[t + 1] ? last : tile_start[t + 1];
        int32_t* tokrow = a.tokmax + (int64_t)t * a.n_docs;
        for (; tile < stop; ++tile) {
            const int64_t v0 = (tile - t_first) * kScanTile;
            for (int it = 0; it < kScanIters; ++it) {
                const int64_t v = v0 + it * kScanBlock + tid;
                const bool active = v < n_emb;
                int doc = -1 - lane;  // inactive lanes never match a neighbour
                int score = INT32_MIN;
                if (active) {
                    int jl = 0, jh = P;  // s_pref[jl] <= v < s_pref[jh]
                    while (jh - jl > 1) {
                        const int jm = (jl + jh) >> 1;
                        if (s_pref[jm] <= v) jl = jm;
                        else jh = jm;
                    }
                    const int64_t e = s_start[jl] + (v - s_pref[jl]);
                    const uint4* row = reinterpret_cast<const uint4*>(codes + e * BYTES);
                    uint4 r[VEC];
#pragma unroll
                    for (int i = 0; i < VEC; ++i) r[i] = row[i];
                    doc = doc_ids[e];
                    int acc = s_base[jl];
#pragma unroll
                    for (int i = 0; i < VEC; ++i) {
                        const unsigned w[4] = {r[i].x, r[i].y, r[i].z, r[i].w};
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            const int p = 16 * i + 4 * k;  // first code byte of this dword
                            acc += lut[(p + 0) * 256 + (w[k] & 255u)];
                            acc += lut[(p + 1) * 256 + ((w[k] >> 8) & 255u)];
                            acc += lut[(p + 2) * 256 + ((w[k] >> 16) & 255u)];
                            acc += lut[(p + 3) * 256 + (w[k] >> 24)];
                        }
                    }
                    score = acc;
                }
                // segmented max over runs of equal doc ids in adjacent lanes
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    const int d2 = __shfl_up(doc, off, 64);
                    const int s2 = __shfl_up(score, off, 64);
                    if (lane >= off && d2 == doc && s2 > score) score = s2;
                }
                const int dn = __shfl_down(doc, 1, 64);
                if (active && (lane == 63 || dn != doc)) atomicMax(&tokrow[doc], score);
            }
        }
    }
}

void launch_scan(const WaveArgs& a, hipStream_t s) {
    if (a.nbits == 4)
        hipLaunchKernelGGL(k_scan<4>, dim3(a.scan_grid), dim3(kScanBlock), 0, s, a);
    else
        hipLaunchKernelGGL(k_scan<2>, dim3(a.scan_grid), dim3(kScanBlock), 0, s, a);
}

int scan_blocks_per_cu(int nbits) {
    int n = 0;
    if (nbits == 4)
        (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_scan<4>, kScanBlock, 0);
    else
        (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_scan<2>, kScanBlock, 0);
    return n > 0 ? n : 1;
}

}  // namespace warp
