// Cluster-major implicit decompression and token-level max (Sections 4.4, 4.5).
//
// Same arithmetic as the token-major scan: for a probing token i of cluster c and
// every embedding e of c,
//     t = R(S64[i][c]) + sum_d R(q_{i,d} * omega[code_{e,d}])          (int32, exact)
// then tokmax[i][doc(e)] = max(...) through a wave segmented max and one
// atomicMax per run of equal documents.
//
// Order of work: a work item is (cluster, chunk of kCmBlock embeddings, group of
// kCmGroup probing tokens); items of one chunk are consecutive, so a persistent
// workgroup walking a contiguous item range loads a chunk's codes into registers
// once and scores them against every token of its items. The HBM traffic of the
// scan is then about one read of every probed cluster per wave of queries,
// instead of one read per probing token.
//
// Table: the per-token table upsilon = q_hat x omega_hat (Section 4.4) is held
// per code nibble: entry [n][v] is the sum of the per-dimension entries of the
// dimensions packed in nibble n when it holds v (one dimension for b = 4, two for
// b = 2), so the integer sums are those of the per-dimension table. One 16-byte
// entry holds four tokens; with PACK = 8 a second table of the next four tokens
// sits at a fixed offset, read with the same address register. All lanes of a
// wave read the same nibble row of 16 entries at a time, which the LDS serves
// without bank conflicts. The table is built in LDS directly from the fp32 query
// tokens: R(q_d * omega_v) in fp64, as in the definition.
#include "engine.h"

namespace warp {

// R(q * w) for a query value already scaled by 2^kFrac (exact: a power of two).
__device__ __forceinline__ int fixed_prod(double q_scaled, double w) {
    return (int)__builtin_rint(q_scaled * w);
}

// 16 x (high nibble of byte B of w): one SDWA AND, the byte offset of table entry
// v in its row of 16-byte entries. The low nibble of byte B is the same operation
// on w << 4.
template <int B>
__device__ __forceinline__ unsigned nib16(unsigned w, unsigned mask_f0) {
    unsigned r;
    if (B == 0) {
        r = w & 0xF0u;
    } else if (B == 1) {
        asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD"
            : "=v"(r) : "v"(w), "v"(mask_f0));
    } else if (B == 2) {
        asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 src1_sel:DWORD"
            : "=v"(r) : "v"(w), "v"(mask_f0));
    } else {
        asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3 src1_sel:DWORD"
            : "=v"(r) : "v"(w), "v"(mask_f0));
    }
    return r;
}

// Wave-level segmented max-scan over runs of equal document ids, the gfx9 DPP
// pattern of a wave64 inclusive scan: row_shr 1, 2, 4, 8 inside rows of 16 lanes,
// then row_bcast 15 (rows 1, 3) and row_bcast 31 (rows 2, 3). A step merges the
// source lane only when it holds the same document; merging values of one
// document is always correct, and every lane of a contiguous run is covered by
// the run's last lane as in the plain scan.
constexpr int kDppCtrl[6] = {0x111, 0x112, 0x114, 0x118, 0x142, 0x143};
constexpr int kDppRows[6] = {0xf, 0xf, 0xf, 0xf, 0xa, 0xc};

template <int K>
__device__ __forceinline__ int dpp_src(int v) {
    return __builtin_amdgcn_update_dpp(INT32_MIN, v, kDppCtrl[K], kDppRows[K], 0xf, false);
}

// Bit k: the step-k source lane holds the same document as this lane.
__device__ __forceinline__ unsigned same_doc_steps(int doc) {
    unsigned m = 0;
    m |= (dpp_src<0>(doc) == doc) ? 1u : 0u;
    m |= (dpp_src<1>(doc) == doc) ? 2u : 0u;
    m |= (dpp_src<2>(doc) == doc) ? 4u : 0u;
    m |= (dpp_src<3>(doc) == doc) ? 8u : 0u;
    m |= (dpp_src<4>(doc) == doc) ? 16u : 0u;
    m |= (dpp_src<5>(doc) == doc) ? 32u : 0u;
    return m;
}

__device__ __forceinline__ int seg_max(int v, unsigned same) {
    int s;
    s = dpp_src<0>(v); v = (same & 1u) && s > v ? s : v;
    s = dpp_src<1>(v); v = (same & 2u) && s > v ? s : v;
    s = dpp_src<2>(v); v = (same & 4u) && s > v ? s : v;
    s = dpp_src<3>(v); v = (same & 8u) && s > v ? s : v;
    s = dpp_src<4>(v); v = (same & 16u) && s > v ? s : v;
    s = dpp_src<5>(v); v = (same & 32u) && s > v ? s : v;
    return v;
}

template <int NBITS, int PACK>
__global__ __launch_bounds__(kCmBlock) void k_scan_cm(WaveArgs a) {
    constexpr int BYTES = kDim * NBITS / 8;  // code bytes per embedding
    constexpr int VEC = BYTES / 16;          // 16-byte loads per embedding
    constexpr int NN = 2 * BYTES;            // nibbles per embedding
    constexpr int ENT = NN * 16;             // table entries per token
    constexpr int PER = ENT / kCmBlock;      // entries built per thread
    constexpr int TABLES = PACK / 4;         // 16-byte tables of four tokens
    static_assert(PER * kCmBlock == ENT, "table must split evenly");
    static_assert((PACK * kDim) % kCmBlock == 0, "query staging");
    static_assert((TABLES - 1) * ENT * 16 + NN * 256 <= 65536, "second table within the LDS offset field");
    __shared__ int4 lut[TABLES * ENT];
    __shared__ double qd[PACK][kDim];
    __shared__ int s_pair[PACK][2];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int n_c = a.n_c;
    const int64_t* item_start = a.item_start;
    const int64_t total = item_start[n_c];
    const int64_t G = gridDim.x;
    int64_t item = total * blockIdx.x / G;
    const int64_t last = total * (blockIdx.x + 1) / G;
    if (item >= last) return;

    // cluster of the first item: item_start[c] <= item < item_start[c + 1]
    int lo = 0, hi = n_c;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (item_start[mid] <= item) lo = mid;
        else hi = mid;
    }
    int c = lo;

    // every table entry this thread builds has nibble value v = tid % 16
    const int v = tid & 15;
    const double w_a = (double)a.weights[NBITS == 4 ? v : (v >> 2)];
    const double w_b = (double)a.weights[NBITS == 4 ? 0 : (v & 3)];

    int cur_c = -1;
    int64_t cur_chunk = -1;
    uint4 code[VEC];
    int doc = 0;
    bool act = false, wave_act = false, run_end = false;
    unsigned same = 0;  // DPP steps that merge the same document
    const uint8_t* __restrict__ codes = a.codes;

    while (item < last) {
        while (item_start[c + 1] <= item) ++c;
        const int nt = a.ccount[c];
        const int groups = (nt + kCmGroup - 1) / kCmGroup;
        const int64_t l = item - item_start[c];
        const int64_t chunk = l / groups;
        const int grp = (int)(l - chunk * groups);
        if (c != cur_c || chunk != cur_chunk) {
            const int64_t e = a.offsets[c] + chunk * kCmBlock + tid;
            act = e < a.offsets[c + 1];
            doc = -1 - lane;  // inactive lanes never match a neighbour
            if (act) {
                const uint4* row = reinterpret_cast<const uint4*>(codes + e * BYTES);
#pragma unroll
                for (int i = 0; i < VEC; ++i) code[i] = row[i];
                doc = a.doc_ids[e];
            }
            wave_act = __any(act);
            same = same_doc_steps(doc);
            const int dn = __shfl_down(doc, 1, 64);
            run_end = act && (lane == 63 || dn != doc);
            cur_c = c;
            cur_chunk = chunk;
        }
        const int p_first = a.pair_start[c] + grp * kCmGroup;
        const int p_end = min(p_first + kCmGroup, a.pair_start[c] + nt);
        for (int p = p_first; p < p_end; p += PACK) {
            const int ng = min(PACK, p_end - p);
            __syncthreads();  // the previous table and query rows are no longer read
            if (tid < PACK) {
                s_pair[tid][0] = tid < ng ? a.plist[2 * (int64_t)(p + tid)] : -1;
                s_pair[tid][1] = tid < ng ? a.plist[2 * (int64_t)(p + tid) + 1] : 0;
            }
#pragma unroll
            for (int h = 0; h < (PACK * kDim) / kCmBlock; ++h) {
                const int x = tid + kCmBlock * h;
                const int g = x >> 7, d = x & 127;
                float qv = 0.f;
                if (g < ng) {
                    const int t = a.plist[2 * (int64_t)(p + g)];
                    qv = a.queries[(int64_t)t * kDim + d];
                }
                qd[g][d] = (double)qv * (double)(1 << kFrac);
            }
            __syncthreads();
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int x = tid + kCmBlock * i;
                const int n = x >> 4;                   // nibble n of dword n / 8, nibble n % 8
                const int m = n & 7;
                const int j = 4 * (n >> 3) + (m >> 1);  // code byte holding the nibble
#pragma unroll
                for (int tb = 0; tb < TABLES; ++tb) {
                    int val[4];
                    if (NBITS == 4) {
                        const int d = 2 * j + ((m & 1) ? 0 : 1);  // high nibble: dimension 2j
#pragma unroll
                        for (int g = 0; g < 4; ++g) val[g] = fixed_prod(qd[4 * tb + g][d], w_a);
                    } else {
                        const int d = (m & 1) ? 4 * j : 4 * j + 2;  // high nibble: dimensions 4j, 4j+1
#pragma unroll
                        for (int g = 0; g < 4; ++g)
                            val[g] = fixed_prod(qd[4 * tb + g][d], w_a) + fixed_prod(qd[4 * tb + g][d + 1], w_b);
                    }
                    lut[tb * ENT + x] = make_int4(val[0], val[1], val[2], val[3]);
                }
            }
            __syncthreads();
            if (!wave_act) continue;  // wave-uniform
            int tok[PACK], acc[PACK];
#pragma unroll
            for (int g = 0; g < PACK; ++g) {  // uniform across the workgroup: scalar registers
                tok[g] = __builtin_amdgcn_readfirstlane(s_pair[g][0]);
                acc[g] = __builtin_amdgcn_readfirstlane(s_pair[g][1]);
            }
            const char* lbase = reinterpret_cast<const char*>(lut);
            const unsigned mask_f0 = 0xF0u;
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                uint4 cw = code[i];
                // keep the nibble extraction inside the token loop: hoisting all
                // table addresses out of it costs more registers than it saves
                asm volatile("" : "+v"(cw.x), "+v"(cw.y), "+v"(cw.z), "+v"(cw.w));
                const unsigned wv[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    // entry offsets: nibble 2b of the dword is the low nibble of byte b
                    // (read from w << 4), nibble 2b + 1 its high nibble
                    const unsigned w = wv[k], w4 = w << 4;
                    const unsigned off_lo[4] = {nib16<0>(w4, mask_f0), nib16<1>(w4, mask_f0),
                                                nib16<2>(w4, mask_f0), nib16<3>(w4, mask_f0)};
                    const unsigned off_hi[4] = {nib16<0>(w, mask_f0), nib16<1>(w, mask_f0),
                                                nib16<2>(w, mask_f0), nib16<3>(w, mask_f0)};
                    const int row = (4 * i + k) * 8;  // first nibble row of the dword
#pragma unroll
                    for (int h = 0; h < 2; ++h) {  // four lookups per table in flight
                        int4 e[TABLES][4];
#pragma unroll
                        for (int b = 2 * h; b < 2 * h + 2; ++b) {
                            const char* pe = lbase + (row + 2 * b) * 256 + off_lo[b];
                            const char* po = lbase + (row + 2 * b + 1) * 256 + off_hi[b];
#pragma unroll
                            for (int tb = 0; tb < TABLES; ++tb) {
                                e[tb][2 * (b - 2 * h)] = *reinterpret_cast<const int4*>(pe + tb * ENT * 16);
                                e[tb][2 * (b - 2 * h) + 1] = *reinterpret_cast<const int4*>(po + tb * ENT * 16);
                            }
                        }
#pragma unroll
                        for (int tb = 0; tb < TABLES; ++tb) {
#pragma unroll
                            for (int b = 0; b < 4; b += 2) {
                                acc[4 * tb + 0] += e[tb][b].x + e[tb][b + 1].x;
                                acc[4 * tb + 1] += e[tb][b].y + e[tb][b + 1].y;
                                acc[4 * tb + 2] += e[tb][b].z + e[tb][b + 1].z;
                                acc[4 * tb + 3] += e[tb][b].w + e[tb][b + 1].w;
                            }
                        }
                    }
                }
            }
            // inner-cluster max: segmented max over runs of equal documents, then one
            // atomicMax per run and token
#pragma unroll
            for (int g = 0; g < PACK; ++g) acc[g] = seg_max(acc[g], same);
            if (run_end) {
#pragma unroll
                for (int g = 0; g < PACK; ++g)
                    if (g < ng) atomicMax(&a.tokmax[(int64_t)tok[g] * a.n_docs + doc], acc[g]);
            }
        }
        ++item;
    }
}

template <int NBITS, int PACK>
static void launch_cm(const WaveArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((k_scan_cm<NBITS, PACK>), dim3(a.scan_grid), dim3(kCmBlock), 0, s, a);
}

void launch_scan_cm(const WaveArgs& a, hipStream_t s) {
    if (a.nbits == 4) {
        if (a.cm_pack == 8) launch_cm<4, 8>(a, s);
        else launch_cm<4, 4>(a, s);
    } else {
        if (a.cm_pack == 8) launch_cm<2, 8>(a, s);
        else launch_cm<2, 4>(a, s);
    }
}

int scan_cm_blocks_per_cu(int nbits, int pack) {
    int n = 0;
    if (nbits == 4)
        (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, pack == 8 ? k_scan_cm<4, 8> : k_scan_cm<4, 4>, kCmBlock, 0);
    else
        (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, pack == 8 ? k_scan_cm<2, 8> : k_scan_cm<2, 4>, kCmBlock, 0);
    return n > 0 ? n : 1;
}

}  // namespace warp
