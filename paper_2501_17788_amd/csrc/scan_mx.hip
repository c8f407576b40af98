// Residual scan on the matrix cores: implicit decompression, selective sum and
// token-level max (Sections 4.4 and 4.5) for every (probing token, probed
// embedding) pair of a wave of queries.
//
// Arithmetic. With Q(x) = round-half-even(x * 2^22), the residual part of the
// score of query token i against embedding e is the exact integer
//     V = sum_d Q(q_{i,d}) * Q(omega[code_{e,d}])            (units of 2^-44)
// and the token score is t = R(S64[i][c]) + floor(V * 2^-18 + 1/2), an int32 in
// units of 2^-26. Both factors lie in [-8421504, 8355711] (|q_d| <= 1 + 1e-3
// and |omega| <= 1.99 are checked on entry), so each is three signed base-256
// digits x = x2 2^16 + x1 2^8 + x0 with x_j in [-128, 127], and
//     V = sum_s 2^(8 s) A_s,   A_s = sum_{i + j = s} sum_d qdig_i[d] * wdig_j[d]
// for s = 0..4. Every A_s is an int8 matrix product over d, computed by
// v_mfma_i32_16x16x64_i8 with embedding digits as rows and query digits as
// columns (|A_s| <= 3 * 128 * 2^14 < 2^23: no overflow). The class-0 accumulator
// starts from the rounding half, mx_fold turns the five class sums into the rounded
// residual term, and adding the token's centroid term plus its query's cell bias
// (added by the pairing) gives the biased token score (below 2^32) without loss. No
// result depends on the order of a summation, so the scan equals the CPU definition
// bit for bit.
//
// Work. A work item is (cluster, chunk of kMxChunk embeddings, group of up to
// kMxGroup probing tokens); a persistent workgroup of four waves walks a
// contiguous range of items and loads the next item's data while it scores the
// current one. Per item, the query digit planes of the group are staged in LDS in
// operand order and the runs of equal document ids along the chunk are numbered.
// Each wave takes 16-embedding tiles of the chunk, decodes their codes into
// weight digits in registers (v_perm_b32 lookups in 16-byte digit tables, or a
// 256-entry LDS table at b = 8) and runs the 18 MFMAs of every 16-token tile of
// the group with the weight digits as rows and the query digits as columns, so that
// each lane holds one token against four consecutive embeddings. Every score goes
// into an LDS table of (token, run) maxima by an LDS atomic max: the 16 lanes of a
// row write 16 different tokens, so lanes meet on one cell only where a run covers
// embeddings four apart. At the end of the item the table is flushed with one device
// atomicMax per (token, run) into the token-max table.
#include "engine.h"

namespace warp {

typedef int v4i __attribute__((ext_vector_type(4)));

// Q(x): x * 2^22 is exact in fp32 and v_rndne_f32 rounds half to even.
__device__ __forceinline__ int quant22(float x) { return (int)__builtin_rintf(x * 4194304.0f); }

// Balanced base-256 digits of x in [-8421504, 8355711].
__device__ __forceinline__ void digits3(int x, int& d0, int& d1, int& d2) {
    d0 = ((x + 128) & 255) - 128;
    x = (x - d0) >> 8;
    d1 = ((x + 128) & 255) - 128;
    d2 = (x - d1) >> 8;
}

// floor((a0 + 2^8 a1 + 2^16 a2 + 2^24 a3 + 2^32 a4) / 2^18) modulo 2^32. The last two terms
// divide exactly, to 2^6 a3 + 2^14 a4. For the rest, n = a0 + 2^8 a1 fits in int32 (|a0| <=
// 2^21 + 2^17, |a1| <= 2^22) and nested floor division gives
// floor((n + 2^16 a2) / 2^18) = floor((floor(n / 2^16) + a2) / 4), two arithmetic shifts. With
// a0 = A0 + 2^17 (the class-0 accumulator starts at the rounding half: round half up) this is
// the rounded residual term floor(V / 2^18 + 1/2) modulo 2^32; the scan adds the token's
// centroid term plus its cell bias, and the sum, the biased token score, lies below 2^32,
// hence is exact.
__device__ __forceinline__ unsigned mx_fold(int a0, int a1, int a2, int a3, int a4) {
    const int n = (int)((unsigned)a0 + ((unsigned)a1 << 8));
    const int u = (n >> 16) + a2;
    return ((((unsigned)a4 << 8) + (unsigned)a3) << 6) + (unsigned)(u >> 2);
}

// Operand slot of dimension d: lane group g = d / 32 of the 16 x 64 operands,
// K slice s (two MFMAs of 64 dimensions), byte j of the lane's 16 bytes. The
// order follows the code layout so that decoding needs no byte shuffles:
//   b = 4: code byte 16 g + 4 m + t holds dimensions 32 g + 8 m + 2 t (high
//          nibble) and + 1 (low nibble); slice s takes code words m = 2 s, 2 s + 1
//          as [high nibbles of 2 s, low of 2 s, high of 2 s + 1, low of 2 s + 1];
//   b = 2: code byte 8 g + 4 s + t holds dimensions 32 g + 16 s + 4 t + u, u = 0
//          in the top bits; slice s holds the four fields u = 0..3 in that order;
//   b = 1: code byte 4 g + t holds dimensions 32 g + 8 t + (7 - k) in bit k; word
//          u of slice s holds bit k = 4 s + u of the four bytes;
//   b = 8: code byte 32 g + 16 s + j is dimension 32 g + 16 s + j.
template <int NBITS>
__device__ __forceinline__ void slot_of_dim(int d, int& s, int& g, int& j) {
    g = d >> 5;
    const int r = d & 31;
    if (NBITS == 4) {
        const int m = r >> 3, t = (r & 7) >> 1, lo = r & 1;
        s = m >> 1;
        j = 4 * (2 * (m & 1) + lo) + t;
    } else if (NBITS == 2) {
        s = r >> 4;
        j = 4 * (r & 3) + ((r & 15) >> 2);
    } else if (NBITS == 1) {
        const int k = 7 - (r & 7);
        s = k >> 2;
        j = 4 * (k & 3) + (r >> 3);
    } else {
        s = r >> 4;
        j = r & 15;
    }
}

// Weight digit tables of a workgroup: for b <= 4, tab[p][k] holds digit p of Q(omega[v]) for
// v = 4 k .. 4 k + 3 (in registers); for b = 8, s_wd[v] holds the three digits of Q(omega[v]) in
// bytes 0..2 (LDS, written by threads 0..255: the caller orders it with a barrier).
template <int NBITS>
__device__ __forceinline__ void weight_tables(const float* weights, unsigned (&tab)[3][4], unsigned* s_wd, int tid) {
    if (NBITS <= 4) {
#pragma unroll
        for (int v = 0; v < (NBITS <= 4 ? 1 << NBITS : 0); ++v) {
            int d[3];
            digits3(quant22(weights[v]), d[0], d[1], d[2]);
#pragma unroll
            for (int p = 0; p < 3; ++p) tab[p][v >> 2] |= ((unsigned)d[p] & 255u) << (8 * (v & 3));
        }
    } else if (tid < 256) {
        int d[3];
        digits3(quant22(weights[tid]), d[0], d[1], d[2]);
        s_wd[tid] = ((unsigned)d[0] & 255u) | (((unsigned)d[1] & 255u) << 8) | (((unsigned)d[2] & 255u) << 16);
    }
}

// The three weight-digit planes of one lane's 32 dimensions of a 16-embedding tile, in
// operand order: W[p][s] is digit plane p of K slice s (slot_of_dim). `wj` holds the
// lane's code words of the tile: v_perm_b32 lookups in the register tables (3 per four
// nibbles and plane at b = 4; 1 per four fields at b = 2 and per four bits at b = 1), or at
// b = 8 one LDS table lookup per code byte followed by 3 v_perm per plane and four dimensions.
template <int NBITS>
__device__ __forceinline__ void decode_weight_digits(const unsigned (&wj)[NBITS], const unsigned (&tab)[3][4],
                                                     const unsigned* s_wd, v4i (&W)[3][2]) {
    constexpr int CW = NBITS;
    if (NBITS == 4) {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const unsigned x = h == 0 ? (wj[m % CW] >> 4) & 0x0F0F0F0Fu : wj[m % CW] & 0x0F0F0F0Fu;
                const unsigned x7 = x & 0x07070707u;
                const unsigned pick = ((x >> 1) & 0x04040404u) | 0x03020100u;
#pragma unroll
                for (int p = 0; p < 3; ++p) {
                    const unsigned lo8 = __builtin_amdgcn_perm(tab[p][1], tab[p][0], x7);
                    const unsigned hi8 = __builtin_amdgcn_perm(tab[p][3], tab[p][2], x7);
                    W[p][m >> 1][2 * (m & 1) + h] = (int)__builtin_amdgcn_perm(hi8, lo8, pick);
                }
            }
        }
    } else if (NBITS == 2) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const unsigned x = (wj[s % CW] >> (6 - 2 * u)) & 0x03030303u;
#pragma unroll
                for (int p = 0; p < 3; ++p) W[p][s][u] = (int)__builtin_amdgcn_perm(tab[p][0], tab[p][0], x);
            }
        }
    } else if (NBITS == 1) {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const unsigned x = (wj[0] >> k) & 0x01010101u;  // bit k of each byte: 0 or 1
#pragma unroll
            for (int p = 0; p < 3; ++p) W[p][k >> 2][k & 3] = (int)__builtin_amdgcn_perm(tab[p][0], tab[p][0], x);
        }
    } else {
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const unsigned wm = wj[m % CW];
            const unsigned e0 = s_wd[wm & 255u], e1 = s_wd[(wm >> 8) & 255u];
            const unsigned e2 = s_wd[(wm >> 16) & 255u], e3 = s_wd[wm >> 24];
#pragma unroll
            for (int p = 0; p < 3; ++p) {
                const unsigned sel = 0x0C0C0000u | ((unsigned)(4 + p) << 8) | (unsigned)p;
                const unsigned lo2 = __builtin_amdgcn_perm(e1, e0, sel);  // bytes 0, 1: digit p of e0, e1
                const unsigned hi2 = __builtin_amdgcn_perm(e3, e2, sel);
                W[p][m >> 2][m & 3] = (int)__builtin_amdgcn_perm(hi2, lo2, 0x05040100u);
            }
        }
    }
}

// One operand of decode_weight_digits, W[p][s], alone (p and s are compile-time after
// unrolling), so that a caller can decode each operand just before its MFMA.
template <int NBITS>
__device__ __forceinline__ v4i weight_operand(const unsigned (&wj)[NBITS], const unsigned (&tab)[3][4],
                                              const unsigned* s_wd, int p, int s) {
    v4i w;
    if (NBITS == 4) {
#pragma unroll
        for (int mm = 0; mm < 2; ++mm) {
            const int m = 2 * s + mm;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const unsigned x = h == 0 ? (wj[m % NBITS] >> 4) & 0x0F0F0F0Fu : wj[m % NBITS] & 0x0F0F0F0Fu;
                const unsigned x7 = x & 0x07070707u;
                const unsigned pick = ((x >> 1) & 0x04040404u) | 0x03020100u;
                const unsigned lo8 = __builtin_amdgcn_perm(tab[p][1], tab[p][0], x7);
                const unsigned hi8 = __builtin_amdgcn_perm(tab[p][3], tab[p][2], x7);
                w[2 * mm + h] = (int)__builtin_amdgcn_perm(hi8, lo8, pick);
            }
        }
    } else if (NBITS == 2) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const unsigned x = (wj[s % NBITS] >> (6 - 2 * u)) & 0x03030303u;
            w[u] = (int)__builtin_amdgcn_perm(tab[p][0], tab[p][0], x);
        }
    } else if (NBITS == 1) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const unsigned x = (wj[0] >> (4 * s + kk)) & 0x01010101u;
            w[kk] = (int)__builtin_amdgcn_perm(tab[p][0], tab[p][0], x);
        }
    } else {
#pragma unroll
        for (int mm = 0; mm < 4; ++mm) {
            const unsigned wm = wj[(4 * s + mm) % NBITS];
            const unsigned e0 = s_wd[wm & 255u], e1 = s_wd[(wm >> 8) & 255u];
            const unsigned e2 = s_wd[(wm >> 16) & 255u], e3 = s_wd[wm >> 24];
            const unsigned sel = 0x0C0C0000u | ((unsigned)(4 + p) << 8) | (unsigned)p;
            const unsigned lo2 = __builtin_amdgcn_perm(e1, e0, sel);
            const unsigned hi2 = __builtin_amdgcn_perm(e3, e2, sel);
            w[mm] = (int)__builtin_amdgcn_perm(hi2, lo2, 0x05040100u);
        }
    }
    return w;
}

// A lane's code words of embedding `row` (null: zeros) in the tile layout: 4 * NBITS bytes
// at lane group lg of the embedding's code row.
template <int NBITS>
__device__ __forceinline__ void load_code_words(const uint8_t* row, int lg, unsigned (&wj)[NBITS]) {
#pragma unroll
    for (int m = 0; m < NBITS; ++m) wj[m] = 0;
    if (!row) return;
    row += 4 * NBITS * lg;
    if (NBITS == 8) {
        const uint4 v0 = reinterpret_cast<const uint4*>(row)[0];
        const uint4 v1 = reinterpret_cast<const uint4*>(row)[1];
        wj[0] = v0.x; wj[1 % NBITS] = v0.y; wj[2 % NBITS] = v0.z; wj[3 % NBITS] = v0.w;
        wj[4 % NBITS] = v1.x; wj[5 % NBITS] = v1.y; wj[6 % NBITS] = v1.z; wj[7 % NBITS] = v1.w;
    } else if (NBITS == 4) {
        const uint4 v = *reinterpret_cast<const uint4*>(row);
        wj[0] = v.x; wj[1 % NBITS] = v.y; wj[2 % NBITS] = v.z; wj[3 % NBITS] = v.w;
    } else if (NBITS == 2) {
        const uint2 v = *reinterpret_cast<const uint2*>(row);
        wj[0] = v.x; wj[1 % NBITS] = v.y;
    } else {
        wj[0] = *reinterpret_cast<const unsigned*>(row);
    }
}

// The code words at `row` (already offset to the lane group's bytes), which must exist.
template <int NBITS>
__device__ __forceinline__ void load_code_words_from(const uint8_t* row, unsigned (&wj)[NBITS]) {
    if (NBITS == 8) {
        const uint4 v0 = reinterpret_cast<const uint4*>(row)[0];
        const uint4 v1 = reinterpret_cast<const uint4*>(row)[1];
        wj[0] = v0.x; wj[1 % NBITS] = v0.y; wj[2 % NBITS] = v0.z; wj[3 % NBITS] = v0.w;
        wj[4 % NBITS] = v1.x; wj[5 % NBITS] = v1.y; wj[6 % NBITS] = v1.z; wj[7 % NBITS] = v1.w;
    } else if (NBITS == 4) {
        const uint4 v = *reinterpret_cast<const uint4*>(row);
        wj[0] = v.x; wj[1 % NBITS] = v.y; wj[2 % NBITS] = v.z; wj[3 % NBITS] = v.w;
    } else if (NBITS == 2) {
        const uint2 v = *reinterpret_cast<const uint2*>(row);
        wj[0] = v.x; wj[1 % NBITS] = v.y;
    } else {
        wj[0] = *reinterpret_cast<const unsigned*>(row);
    }
}

// Per-wave preparation in one launch, ordered after the previous wave's scan and fold and
// before this wave's selection. Blocks [0, nb0): the clusters' token counters and scatter
// cursors zeroed, the query slots' next epochs (1 after the last one, else one more; ep may
// be null), the scan's batch counter set to the grid size, and for the split selection the
// tokens' histograms and band counts zeroed. The next nb1 blocks: the norm check of the wave's
// query tokens (one wave per token; a failure sets kErrQueryNorm). The rest: the query digit
// planes of every wave token, qdig[t][(p * 2 + s) * 4 + g][16] bytes.
template <int NBITS>
__global__ __launch_bounds__(256) void k_wave_prep(WaveArgs a, uint32_t* ep, uint32_t last, int32_t nb0,
                                                   int32_t nb1) {
    const int64_t n_tok = (int64_t)a.n_q * a.n_qtok;
    const int b = blockIdx.x;
    if (b < nb0) {
        const int64_t i = (int64_t)b * 256 + threadIdx.x;
        if (i < a.n_c) {
            a.ccount[i] = 0;
            a.cursor[i] = 0;
        }
        if (a.sel_slices > 1) {  // the split selection's histograms and band counts
            if (i < n_tok * kSelBins) a.sel_hist[i] = 0;
            if (i < 2 * n_tok) a.sel_cnt[i] = 0;
        }
        if (ep && i < a.n_q) ep[i] = ep[i] >= last ? 1u : ep[i] + 1u;
        if (i == 0) *a.scan_queue = (uint32_t)a.scan_grid;
        return;
    }
    if (b < nb0 + nb1) {
        const int64_t t = (int64_t)(b - nb0) * 4 + (threadIdx.x >> 6);
        const int lane = threadIdx.x & 63;
        if (t >= n_tok) return;  // wave-uniform
        const float x0 = a.queries[t * kDim + lane], x1 = a.queries[t * kDim + 64 + lane];
        double ss = (double)x0 * x0 + (double)x1 * x1;
        bool bad = !(__builtin_isfinite(x0) && __builtin_isfinite(x1));
        for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
        bad = __any(bad);
        if (lane == 0 && (bad || !(ss <= (1.0 + 1e-3) * (1.0 + 1e-3)))) atomicOr(a.err, kErrQueryNorm);
        return;
    }
    const int64_t x = (int64_t)(b - nb0 - nb1) * 256 + threadIdx.x;
    if (x >= n_tok * kDim) return;
    const int64_t t = x / kDim;
    const int d = (int)(x % kDim);
    int s, g, j, d0, d1, d2;
    slot_of_dim<NBITS>(d, s, g, j);
    digits3(quant22(a.queries[x]), d0, d1, d2);
    int8_t* row = a.qdig + t * kQdigBytes;
    row[((0 * 2 + s) * 4 + g) * 16 + j] = (int8_t)d0;
    row[((1 * 2 + s) * 4 + g) * 16 + j] = (int8_t)d1;
    row[((2 * 2 + s) * 4 + g) * 16 + j] = (int8_t)d2;
}

struct MxItem {
    int64_t e0;   // first embedding of the chunk
    int64_t e1;   // end of the chunk
    int p0, np;   // pairs [p0, p0 + np) of the token group
};

// A wave-uniform load of the work plan through the scalar cache. The plan is read-only
// here (earlier kernels wrote it), and scalar loads are waited for on their own counter,
// so reading it never waits for the vector loads and atomics in flight.
template <typename T>
__device__ __forceinline__ T plan_load(const T* p, int64_t i) {
    return ((const __attribute__((address_space(4))) T*)p)[i];
}

// item of the wave's probed-chunk list entry p, whose record is rec (its chunk's token
// group item - list_item[p])
__device__ __forceinline__ MxItem mx_decode(const v4i rec, int64_t item, int64_t item0) {
    MxItem it;
    const uint64_t ew = (uint64_t)(uint32_t)rec[0] | ((uint64_t)(uint32_t)rec[1] << 32);
    const int grp = (int)(item - item0);
    const int nt = rec[3];
    it.e0 = (int64_t)(ew & ((1ull << kRecLenShift) - 1));
    it.e1 = it.e0 + (int64_t)(ew >> kRecLenShift);
    it.p0 = rec[2] + grp * kMxGroup;
    it.np = nt - grp * kMxGroup < kMxGroup ? nt - grp * kMxGroup : kMxGroup;
    return it;
}

// Registers that carry an item's global data from its prefetch, one item ahead,
// to its staging in LDS.
template <int QPT>
struct MxStage {
    v4i q[QPT];     // query digit slots tid + kMxBlock i of the group
    int tok, base;  // thread tid < kMxGroup: wave token and R(S64) + cell bias of group token tid
    int doc, prev;  // documents of chunk embeddings tid and tid - 1 (-1 outside the chunk)
};

template <int NBITS>
__global__ __launch_bounds__(kMxBlock, 3) void k_scan_mx(WaveArgs a) {
    constexpr int BYTES = kDim * NBITS / 8;  // code bytes per embedding
    constexpr int CW = NBITS;                // code words per lane: 32 dimensions of b bits
    constexpr int NSLOT = 24;                // (plane, slice, lane group) slots of 16 bytes
    // row of the run table: the 16 token rows one atomic writes start 4 banks apart; column
    // kMxChunk takes the scores of embeddings past the chunk's end and is never read
    constexpr int TPAD = kMxChunk + 4;
    constexpr int NW = kMxBlock / 64;
    constexpr int QPT = NSLOT * kMxGroup / kMxBlock;  // query slots staged per thread
    constexpr int TPW = kMxChunk / (16 * NW);          // 16-embedding tiles per wave
    // the run pass gives each thread at most one embedding of the chunk, the query staging
    // splits evenly over the threads, and the waves split the tiles evenly
    static_assert(kMxChunk <= kMxBlock, "one thread per chunk embedding");
    static_assert(NSLOT * kMxGroup % kMxBlock == 0, "query staging");
    static_assert(kMxChunk % (16 * NW) == 0, "tiles per wave");
    // query digit planes of the item's tokens, one padded row per token: the staging writes
    // of consecutive threads are contiguous, and the 16 tokens of an operand read lie 400 bytes apart
    __shared__ v4i s_q[kMxGroup][NSLOT + 1];
    __shared__ unsigned s_cterm[kMxGroup];   // R(S64) + the cell bias of each token (0 past the group)
    __shared__ __attribute__((aligned(16))) int64_t s_row[2][kMxGroup];  // its token-max row offset
    __shared__ unsigned s_tab[kMxGroup * TPAD];  // max score of (token, document run of the chunk)
    __shared__ __attribute__((aligned(16))) int s_run[kMxChunk];  // run of each chunk embedding (kMxChunk past its end)
    __shared__ int s_rdoc[kMxChunk];         // document of each run
    __shared__ int s_rstart[kMxChunk];       // its first embedding in the chunk
    __shared__ int s_wruns[NW];              // runs starting in each wave's quarter of the chunk
    __shared__ unsigned s_claim;             // the batch thread 0 claimed
    __shared__ unsigned s_wd[NBITS == 8 ? 256 : 1];  // b = 8: the three digits of Q(omega[v]) in bytes 0..2

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int li = lane & 15;  // operand row / column inside a 16 x 16 tile
    const int lg = lane >> 4;  // operand lane group

    // weight digit tables (for b = 8 in LDS, ordered by the first barrier below)
    unsigned tab[3][4] = {};
    weight_tables<NBITS>(a.weights, tab, s_wd, tid);

    // Items of the wave's probed chunks, in the index's chunk order, in batches of R =
    // kScanBatch: workgroup b starts with batch b; every later batch is claimed from the
    // batch counter (which starts at G) when the workgroup takes the first item of the batch
    // before it. Thread 0 claims with a wrapping increment (which the compiler does not turn
    // into a wave-wide add that waits for its result); the claimed batch reaches every wave
    // through LDS after the next item's staging wait, so a claim adds no wait. Consecutive
    // claims of the grid lie in unrelated clusters, since the chunk order is shuffled.
    const int64_t n_list = plan_load(a.list_n, 0);
    const int64_t* list_item = a.list_item;
    const int64_t total = plan_load(list_item, n_list);
    int64_t gpos = (int64_t)blockIdx.x * kScanBatch;
    if (gpos >= total) return;
    int64_t gend = gpos + kScanBatch < total ? gpos + kScanBatch : total;
    int64_t nb = -1;       // first item of the next batch, once claimed and published
    bool claimed = false;  // a claim is in flight (wave-uniform)
    unsigned claim = 0;    // thread 0: the batch its claim returned
    auto request = [&]() {
        if (tid == 0) claim = atomicInc(a.scan_queue, 0xFFFFFFFFu);
        claimed = true;
    };
    // The next item of the workgroup, or -1. A claim is issued on entering a batch and
    // published before the next call, so the workgroup never runs out of known items
    // while a batch remains; the prologue's claim is still in flight when the first batch
    // ends only if that batch was cut short by the last item, and then nothing is left.
    auto next_item = [&]() -> int64_t {
        if (gpos < gend) return gpos++;
        if (nb < 0 || nb >= total) return -1;
        gpos = nb;
        gend = nb + kScanBatch < total ? nb + kScanBatch : total;
        nb = -1;
        request();
        return gpos++;
    };
    int64_t p = 0;  // list entry of the newest decoded item; items increase along the sequence
    const v4i* qdig = reinterpret_cast<const v4i*>(a.qdig);
    const int32_t* __restrict__ plist = a.plist;
    const uint8_t* __restrict__ codes = a.codes;
    const int32_t* __restrict__ doc_ids = a.doc_ids;
    unsigned* __restrict__ tokmax = a.tokmax;
    for (int i = tid; i < kMxGroup * TPAD; i += kMxBlock) s_tab[i] = kTokAbsent;

    // the software pipeline: while item i is scored, the query digits, bases and documents of
    // item i + 1 are in flight, its codes are loaded before item i's flush, and the wave
    // tokens of item i + 2 (which address item i + 2's query digits) are loaded
    auto load_tokens = [&](const MxItem& x, int (&ptok)[QPT]) {
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
            const int tk = (tid + kMxBlock * i) / NSLOT;
            ptok[i] = tk < x.np ? plist[2 * (int64_t)(x.p0 + tk)] : -1;
        }
    };
    // the documents are loaded only for a new chunk: items of one chunk follow each other
    auto load_stage = [&](const MxItem& x, const int (&ptok)[QPT], MxStage<QPT>& st, bool new_chunk) {
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
            const int slot = (tid + kMxBlock * i) % NSLOT;
            st.q[i] = ptok[i] >= 0 ? qdig[(unsigned)(ptok[i] * NSLOT + slot)] : (v4i){0, 0, 0, 0};
        }
        const bool in = tid < x.np;
        st.tok = in ? plist[2 * (int64_t)(x.p0 + tid)] : 0;
        st.base = in ? plist[2 * (int64_t)(x.p0 + tid) + 1] : 0;
        if (new_chunk) {
            const int64_t e = x.e0 + tid;
            st.doc = e < x.e1 ? doc_ids[e] : -1;
            st.prev = tid > 0 && e < x.e1 ? doc_ids[e - 1] : -1;
        }
    };
    auto load_codes = [&](const MxItem& x, unsigned (&w)[TPW][CW]) {
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            const int64_t er = x.e0 + 16 * (wave + NW * j) + li;
            load_code_words<NBITS>(er < x.e1 ? codes + er * BYTES : nullptr, lg, w[j]);
        }
    };
    // the list entry of item (at or after p): galloping from p, then bisection; the entry's
    // record and first item are read once per entry
    v4i rec = {0, 0, 0, 0};
    int64_t rec_p = -1, rec_item = 0;
    auto decode_item = [&](int64_t item) {
        if (plan_load(list_item, p + 1) <= item) {
            int64_t lo = p + 1, step = 1, hi = lo + 1;  // list_item[lo] <= item
            while (hi < n_list && plan_load(list_item, hi) <= item) {
                lo = hi;
                step <<= 1;
                hi = lo + step;
            }
            if (hi > n_list) hi = n_list;  // list_item[hi] > item
            while (hi - lo > 1) {
                const int64_t mid = (lo + hi) >> 1;
                if (plan_load(list_item, mid) <= item) lo = mid;
                else hi = mid;
            }
            p = lo;
        }
        if (p != rec_p) {
            rec_p = p;
            rec = plan_load(reinterpret_cast<const v4i*>(a.list_rec), p);
            rec_item = plan_load(list_item, p);
        }
        return mx_decode(rec, item, rec_item);
    };

    request();
    MxItem it = decode_item(next_item()), nx = it;
    int ptok[QPT];
    MxStage<QPT> st;
    unsigned w[TPW][CW];
    load_tokens(it, ptok);
    load_stage(it, ptok, st, true);
    load_codes(it, w);
    int64_t nxi = next_item();
    if (nxi >= 0) {
        nx = decode_item(nxi);
        load_tokens(nx, ptok);
    }
    // stage an item from registers: tokens past the group's end have zero digits and centroid
    // terms (score 0 = absent); the token-max row offsets alternate between two buffers, since
    // the previous item's flush still reads its own
    auto stage = [&](const MxItem& x, int par) {
        if (tid < kMxGroup) {
            s_cterm[tid] = tid < x.np ? (unsigned)st.base : 0u;  // R(S64) + the cell bias
            s_row[par][tid] = (int64_t)st.tok * a.n_docs;
        }
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
            const int k = tid + kMxBlock * i;
            s_q[k / NSLOT][k % NSLOT] = st.q[i];
        }
        if (tid == 0 && claimed) s_claim = claim;
    };
    stage(it, 0);

    // The runs of the chunk in LDS (s_run, s_rdoc, s_rstart, n_runs) and the codes in w stay
    // valid while consecutive items share a chunk (the token groups of one chunk).
    int64_t run_e0 = -1;  // first embedding of the chunk whose runs are in LDS
    int n_runs = 0;
    int par = 0;  // buffer of s_row staged for the current item
    for (;;) {
        // the item is staged, and the previous item's flush has read and reset the table and
        // read the runs
        __syncthreads();
        if (claimed) {
            nb = (int64_t)s_claim * kScanBatch;
            claimed = false;
        }
        // runs of equal documents along a new chunk (ids ascend inside a cluster)
        if (it.e0 != run_e0) {  // uniform over the workgroup
            run_e0 = it.e0;
            const bool e_in = st.doc >= 0;
            const int doc = st.doc;
            const bool start = e_in && (tid == 0 || st.prev != doc);
            const unsigned long long starts = __ballot(start);
            if (lane == 0) s_wruns[wave] = __popcll(starts);
            __syncthreads();
            int run = __popcll(starts & ((2ull << lane) - 1)) - 1;  // starts in this wave up to this lane, minus one
            n_runs = 0;
#pragma unroll
            for (int w8 = 0; w8 < NW; ++w8) {
                run += w8 < wave ? s_wruns[w8] : 0;
                n_runs += s_wruns[w8];
            }
            s_run[tid] = e_in ? run : kMxChunk;
            if (start) {
                s_rdoc[run] = doc;
                s_rstart[run] = tid;
            }
            __syncthreads();
        }
        // prefetch: the next item's query digits, bases and documents, then (with the claim
        // published above) the tokens of the item after it
        const bool has_next = nxi >= 0;
        if (has_next) load_stage(nx, ptok, st, nx.e0 != it.e0);
        MxItem nn = nx;
        const int64_t nni = has_next ? next_item() : -1;
        if (nni >= 0) {
            nn = decode_item(nni);
            load_tokens(nn, ptok);
        }

        // the next item's codes replace each tile's codes once they are decoded (the same
        // codes serve the next item of the same chunk)
        const bool next_codes = has_next && nx.e0 != it.e0;
        const int n_et = (int)((it.e1 - it.e0 + 15) >> 4);
        const int n_tt = (it.np + 15) >> 4;
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
            const int et = wave + NW * j;
            const bool tile_in = et < n_et;  // wave-uniform
            // weight digits of the tile (MFMA A operand: row li = embedding e0 + 16 et + li)
            v4i A[3][2];
            if (tile_in) decode_weight_digits<NBITS>(w[j], tab, s_wd, A);
            if (next_codes) {
                const int64_t er = nx.e0 + 16 * et + li;
                load_code_words<NBITS>(er < nx.e1 ? codes + er * BYTES : nullptr, lg, w[j]);
            }
            if (!tile_in) continue;

            for (int tt = 0; tt < n_tt; ++tt) {
                // class accumulators; class 0 starts at the rounding half
                v4i acc[5];
                acc[0] = (v4i){1 << 17, 1 << 17, 1 << 17, 1 << 17};
#pragma unroll
                for (int c = 1; c < 5; ++c) acc[c] = (v4i){0, 0, 0, 0};
#pragma unroll
                for (int s = 0; s < 2; ++s) {
                    // query digits of slice s (MFMA B operand: column li = token 16 tt + li)
                    v4i B[3];
#pragma unroll
                    for (int p = 0; p < 3; ++p) B[p] = s_q[16 * tt + li][(p * 2 + s) * 4 + lg];
#pragma unroll
                    for (int i = 0; i < 3; ++i)
#pragma unroll
                        for (int jj = 0; jj < 3; ++jj)
                            acc[i + jj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[jj][s], B[i], acc[i + jj], 0, 0, 0);
                }
                // acc[k][r] of lane (li, lg): token 16 tt + li against embedding e0 + 16 et + 4 lg + r;
                // merge into the (token, run) table. The runs of the four embeddings come in one
                // read; embeddings past the chunk's end have the padding column.
                const v4i my_run = *reinterpret_cast<const v4i*>(&s_run[16 * et + 4 * lg]);
                const unsigned cterm = s_cterm[16 * tt + li];
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    atomicMax(&s_tab[(16 * tt + li) * TPAD + my_run[r]],
                              mx_fold(acc[0][r], acc[1][r], acc[2][r], acc[3][r], acc[4][r]) + cterm);
            }
        }
        __syncthreads();  // the table is complete, and the item's digits and terms are no longer read
        // Every load of the next item (staged data, codes, the claim) has landed before the
        // flush's atomics are issued. Vector memory operations complete in issue order, so a
        // wait for a load issued after the atomics would also wait for them; none follows
        // before the next item's flush, by which time they are long done.
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        if (has_next) stage(nx, par ^ 1);
        // flush: one device atomic per (token, run). With R = 2^lr the power of two at or above
        // the run count, thread tid takes run tid mod R of tokens tid / R, tid / R + 256 / R, ...:
        // consecutive lanes take consecutive runs of one token (ascending documents of one
        // token-max row), and no thread divides
        const int lr = n_runs <= 1 ? 0 : 32 - __builtin_clz((unsigned)(n_runs - 1));
        const int rn = tid & ((1 << lr) - 1);
        // Each cell is read and reset by one LDS exchange; the loop is unrolled so that the LDS
        // reads of several tokens are in flight together.
        if (rn < n_runs) {
            const int rdoc = s_rdoc[rn];
            const int step = kMxBlock >> lr;
            if (!a.tokcnt) {
                int tk = tid >> lr;
                for (; tk + 3 * step < it.np; tk += 4 * step) {  // four tokens at a time
                    unsigned v[4];
                    int64_t o[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        v[u] = atomicExch(&s_tab[(tk + u * step) * TPAD + rn], kTokAbsent);
                        o[u] = s_row[par][tk + u * step] + rdoc;
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) atomicMax(&tokmax[o[u]], v[u]);
                }
                for (; tk < it.np; tk += step) {
                    const unsigned v = atomicExch(&s_tab[tk * TPAD + rn], kTokAbsent);
                    atomicMax(&tokmax[s_row[par][tk] + rdoc], v);
                }
            } else {
                // Eq.-1-literal scoring: embeddings of the run retrieved for each token
                const unsigned len =
                    (unsigned)((rn + 1 < n_runs ? s_rstart[rn + 1] : (int)(it.e1 - it.e0)) - s_rstart[rn]);
                for (int tk = tid >> lr; tk < it.np; tk += step) {
                    const unsigned v = atomicExch(&s_tab[tk * TPAD + rn], kTokAbsent);
                    const int64_t o = s_row[par][tk] + rdoc;
                    atomicMax(&tokmax[o], v);
                    atomicAdd(&a.tokcnt[o], len);
                }
            }
        }
        par ^= 1;
        if (!has_next) break;
        it = nx;
        nx = nn;
        nxi = nni;
    }
}

// Orders a wave's LDS writes before its later LDS reads by other lanes (one wave per table).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_wave_barrier();
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

// Narrow scan: the chunks probed by 1..narrow_max tokens of the wave (Sections 4.4 and 4.5,
// the same arithmetic as k_scan_mx). One wave takes one chunk at a time, with no workgroup
// barrier: it numbers the chunk's runs of equal documents, then scores the chunk's 16-embedding
// tiles against groups of up to kNrGroup = 3 tokens. In a group's matrix-core tile the
// columns are the tile's embeddings and the rows are (token t, digit class s): row 4 t + s for
// s = 0..3 and row 12 + t for s = 4; the K dimension runs over (weight-digit plane j,
// dimension d), and row (t, s) takes query-digit plane s - j of token t (zero outside 0..2), so
// six v_mfma_i32_16x16x64_i8 give all five class sums A_s of up to three tokens. Lane (e, g)
// then holds rows 4 g .. 4 g + 3 of embedding e: lane group g < 3 holds classes 0..3 of token
// g and folds it, taking class 4 from lane group 3.
// Scores go into the wave's LDS table of (token, run) maxima, flushed with one device
// atomicMax per (token, run) after each group.
//
// Vector memory operations complete in issue order, so after a flush's atomics any wait for a
// load also waits for them. The wave therefore waits once per group, just before its flush,
// for everything the next group needs, and then runs a whole chunk of work before its next
// wait: while chunk c is scored, the pair-list entries of chunk c + 2's first group, the
// query digit rows of chunk c + 1's first group and the documents of chunk c + 1 are in
// flight, and the code words stream through DEPTH buffers (below). The query rows go through
// LDS into the operand registers, which are free once a group's tiles are scored.
template <int NBITS>
__global__ __launch_bounds__(kMxBlock) void k_scan_narrow(WaveArgs a) {
    constexpr int BYTES = kDim * NBITS / 8;
    constexpr int NW = kMxBlock / 64;
    constexpr int NSLOT = 24;                   // 16-byte query digit slots of a token
    constexpr int QSLOTS = kNrGroup * NSLOT;    // slots of a group's query rows
    constexpr int DEPTH = NBITS <= 4 ? 4 : 2;  // code-word buffers of the tile stream
    constexpr int TPAD = kMxChunk + 4;
    static_assert(kMxChunk % 64 == 0 && kMxChunk <= 4 * 64, "four rounds of the run pass");
    static_assert(kNrGroup == 3, "rows of a group's tile: four classes of three tokens, then their fifth");
    static_assert(QSLOTS > 64 && QSLOTS <= 128, "two query-row slots per lane");
    __shared__ unsigned s_tab[NW][kNrGroup * TPAD];  // (token of the group, run) maxima
    __shared__ int s_run[NW][kMxChunk];              // run of each embedding of the chunk
    __shared__ int s_rdoc[NW][kMxChunk];             // document of each run
    __shared__ int s_rstart[NW][kMxChunk + 1];       // its first embedding; the chunk's length after the last
    __shared__ v4i s_qrow[NW][QSLOTS];               // query digit rows of the next group's tokens
    __shared__ unsigned s_wd[NBITS == 8 ? 256 : 1];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: the plan reads are scalar
    const int lane = tid & 63;
    const int li = lane & 15;  // embedding of a tile (column), or row of the query operand
    const int lg = lane >> 4;  // lane group: rows 4 lg .. 4 lg + 3 of the output; token lg of the group
    unsigned tab[3][4] = {};
    weight_tables<NBITS>(a.weights, tab, s_wd, tid);
    if (NBITS == 8) __syncthreads();  // the only workgroup barrier: s_wd is written

    unsigned* stab = s_tab[wave];
    int* runs = s_run[wave];
    int* rdoc = s_rdoc[wave];
    int* rstart = s_rstart[wave];
    v4i* qrow = s_qrow[wave];
    for (int i = lane; i < kNrGroup * TPAD; i += 64) stab[i] = kTokAbsent;
    const int64_t n_list = plan_load(a.list_n2, 0);
    const v4i* qdig = reinterpret_cast<const v4i*>(a.qdig);
    const int32_t* __restrict__ plist = a.plist;
    const uint8_t* __restrict__ codes = a.codes;
    const int32_t* __restrict__ doc_ids = a.doc_ids;
    unsigned* __restrict__ tokmax = a.tokmax;
    const int64_t stride = (int64_t)gridDim.x * NW;
    // row (token, class) of this lane in the query operand (row 15 is zero)
    const int rt = li < 12 ? li >> 2 : li - 12, rs = li < 12 ? li & 3 : 4;
    const int c4_lane = 48 + li;  // the lane holding class 4 of this lane's embedding

    struct NrChunk {
        int64_t e0;
        int len, p0, nt;  // embeddings (1 .. kMxChunk), first pair, probing tokens (1 .. narrow_max)
    };
    auto chunk_at = [&](int64_t q) {
        const v4i rec = plan_load(reinterpret_cast<const v4i*>(a.list_rec2), q);
        const uint64_t ew = (uint64_t)(uint32_t)rec[0] | ((uint64_t)(uint32_t)rec[1] << 32);
        NrChunk c;
        c.e0 = (int64_t)(ew & ((1ull << kRecLenShift) - 1));
        c.len = (int)(ew >> kRecLenShift);
        c.p0 = rec[2];
        c.nt = rec[3];
        return c;
    };
    auto load_docs = [&](const NrChunk& c, int (&dd)[kMxChunk / 64]) {
#pragma unroll
        for (int j = 0; j < kMxChunk / 64; ++j) dd[j] = 64 * j + lane < c.len ? doc_ids[c.e0 + 64 * j + lane] : -1;
    };
    // A group's pair-list entries, per lane: the wave tokens of the query-row slots lane and
    // 64 + lane (-1: none), and the wave token and centroid term of the token lane group lg folds.
    struct NrGroup {
        int wa, wb, tok;
        unsigned cterm;
    };
    auto load_group = [&](const NrChunk& c, int g0, NrGroup& g) {
        const int ng = c.nt - g0 < kNrGroup ? c.nt - g0 : kNrGroup;
        const int64_t p0 = (int64_t)c.p0 + g0;
        const int ta = lane / NSLOT, tb = (64 + lane) / NSLOT;
        g.wa = ta < ng ? plist[2 * (p0 + ta)] : -1;
        g.wb = 64 + lane < QSLOTS && tb < ng ? plist[2 * (p0 + tb)] : -1;
        const bool mine = lg < ng;
        g.cterm = mine ? (unsigned)plist[2 * (p0 + lg) + 1] : 0u;
        g.tok = mine ? plist[2 * (p0 + lg)] : 0;
    };
    // the group's query digit rows (slots of tokens past the group are zero)
    auto load_qrows = [&](const NrGroup& g, v4i& qa, v4i& qb) {
        const v4i z = {0, 0, 0, 0};
        qa = g.wa >= 0 ? qdig[(unsigned)(g.wa * NSLOT + lane % NSLOT)] : z;
        qb = g.wb >= 0 ? qdig[(unsigned)(g.wb * NSLOT + (64 + lane) % NSLOT)] : z;
    };
    // query operand from the rows in LDS: row (rt, rs) takes digit plane rs - j of token rt in
    // K segment j
    auto stage_q = [&](const v4i& qa, const v4i& qb, v4i (&Q)[3][2]) {
        qrow[lane] = qa;
        if (64 + lane < QSLOTS) qrow[64 + lane] = qb;
        wave_lds_sync();
#pragma unroll
        for (int j = 0; j < 3; ++j) {
#pragma unroll
            for (int sl = 0; sl < 2; ++sl) {
                const int pl = rs - j;
                Q[j][sl] = li < 15 && pl >= 0 && pl <= 2 ? qrow[rt * NSLOT + (pl * 2 + sl) * 4 + lg]
                                                                  : (v4i){0, 0, 0, 0};
            }
        }
    };

    int64_t p = (int64_t)blockIdx.x * NW + wave;
    if (p >= n_list) return;  // wave-uniform; no barrier follows
    // the prologue: chunk p's inputs and its first group's operand, chunk p + stride's
    // first-group pair-list entries
    NrChunk cur = chunk_at(p);
    int d[kMxChunk / 64];
    load_docs(cur, d);
    NrGroup g_cur, g_nx;
    load_group(cur, 0, g_cur);
    v4i Q[3][2];
    {
        v4i qa, qb;
        load_qrows(g_cur, qa, qb);
        stage_q(qa, qb, Q);
    }
    if (p + stride < n_list) load_group(chunk_at(p + stride), 0, g_nx);
    // The code words of a group's tiles stream through DEPTH buffers: tile u sits in buffer
    // u % DEPTH, and once it is decoded the buffer takes the tile DEPTH places further along
    // the wave's sequence of (chunk, group) tile runs, each run padded to a multiple of DEPTH
    // tiles (padding tiles are not scored). The next run is the chunk's next group, else the
    // next chunk's first group. Every buffer load is issued, so that the compiler can count the
    // loads in flight and wait for each buffer alone: a lane with no embedding in the tile
    // reads the first code row of the chunk instead, and the scores of its column are never
    // merged.
    unsigned cb[DEPTH][NBITS];
    const unsigned lane_off = 4 * NBITS * lg;
    auto tile_off = [&](int len, int t) -> unsigned {
        const int e = 16 * t + li;
        return e < len ? (unsigned)e * BYTES + lane_off : lane_off;
    };
    auto chunk_base = [&](const NrChunk& c) { return codes + c.e0 * BYTES; };
#pragma unroll
    for (int k = 0; k < DEPTH; ++k) load_code_words_from<NBITS>(chunk_base(cur) + tile_off(cur.len, k), cb[k]);
    // the prologue's loads, waited for here so that no wait inside the loop is for them
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    for (;;) {
        const int64_t pn = p + stride, pnn = pn + stride;
        const bool has_next = pn < n_list;  // wave-uniform
        NrChunk nx = cur;
        int dn[kMxChunk / 64] = {};
        NrGroup g_nn = g_nx;
        v4i qa = {0, 0, 0, 0}, qb = {0, 0, 0, 0};  // query rows of the next chunk's first group
        if (has_next) {
            nx = chunk_at(pn);
            load_docs(nx, dn);
            load_qrows(g_nx, qa, qb);
            if (pnn < n_list) load_group(chunk_at(pnn), 0, g_nn);
        }
        const int len = cur.len, nt = cur.nt;
        // runs of equal documents along the chunk (ids ascend inside a cluster); the chunk's
        // first embedding starts a run
        int n_runs = 0;
#pragma unroll
        for (int j = 0; j < kMxChunk / 64; ++j) {
            const int last = j > 0 ? __shfl(d[j > 0 ? j - 1 : 0], 63, 64) : -1;
            int prev = __shfl_up(d[j], 1, 64);
            if (lane == 0) prev = last;
            const int e = 64 * j + lane;
            const bool in = e < len;
            const bool start = in && (e == 0 || prev != d[j]);
            const unsigned long long m = __ballot(start);
            const int r = n_runs + __popcll(m & ((2ull << lane) - 1)) - 1;
            runs[e] = in ? r : kMxChunk;
            if (start) {
                rdoc[r] = d[j];
                rstart[r] = e;
            }
            n_runs += __popcll(m);
        }
        if (lane == 0) rstart[n_runs] = len;
        wave_lds_sync();
        const int n_tiles = (len + 15) >> 4;
        const int n_pad = (n_tiles + DEPTH - 1) / DEPTH * DEPTH;
        // every chunk has a group (nt >= 1): a loop that runs at least once lets the compiler see
        // that the wait before the flush covers every load of the chunk
        int g0 = 0;
        do {  // wave-uniform
            const int ng = nt - g0 < kNrGroup ? nt - g0 : kNrGroup;
            const bool mine = lg < ng;  // this lane group folds token g0 + lg
            const unsigned cterm = g_cur.cterm;
            const int mytok = g_cur.tok;  // its wave token (the flush's row)
            // the run after this one: the next group of this chunk, else the next chunk (if any)
            const bool more = g0 + kNrGroup < nt;
            const uint8_t* const cur_base = chunk_base(cur);
            const uint8_t* const next_base = more || !has_next ? cur_base : chunk_base(nx);
            const int next_len = more || !has_next ? len : nx.len;
            const int next_n = more || has_next ? 1 << 30 : 0;  // tiles of the next run (0: none)
            for (int t0 = 0; t0 < n_pad; t0 += DEPTH) {  // wave-uniform
#pragma unroll
                for (int k = 0; k < DEPTH; ++k) {
                    const int t = t0 + k;
                    // each weight operand decoded just before its MFMA; then the buffer is refilled
                    // (in place, since its words are no longer read)
                    v4i acc = {0, 0, 0, 0};
                    if (t < n_tiles) {  // wave-uniform
#pragma unroll
                        for (int sl = 0; sl < 2; ++sl)
#pragma unroll
                            for (int j = 0; j < 3; ++j)
                                acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                                    Q[j][sl], weight_operand<NBITS>(cb[k], tab, s_wd, j, sl), acc, 0, 0, 0);
                    }
                    const int u = t + DEPTH;  // stream position of the buffer's next tile
                    if (u < n_pad) load_code_words_from<NBITS>(cur_base + tile_off(len, u), cb[k]);
                    else load_code_words_from<NBITS>(next_base + tile_off(u - n_pad < next_n ? next_len : 0, u - n_pad), cb[k]);
                    if (t >= n_tiles) continue;  // wave-uniform
                    // token lg's classes 0..3 are this lane's acc[0..3]; class 4 is element lg of
                    // lane c4_lane (lane group 3)
                    int a4 = __shfl(acc[0], c4_lane, 64);
                    if (ng > 1) {  // wave-uniform
                        const int a4b = __shfl(acc[1], c4_lane, 64);
                        a4 = lg == 1 ? a4b : a4;
                        if (ng > 2) {
                            const int a4c = __shfl(acc[2], c4_lane, 64);
                            a4 = lg == 2 ? a4c : a4;
                        }
                    }
                    const unsigned v = mx_fold(acc[0] + (1 << 17), acc[1], acc[2], acc[3], a4) + cterm;
                    const int e = 16 * t + li;
                    if (mine && e < len) atomicMax(&stab[lg * TPAD + runs[e]], v);
                }
            }
            wave_lds_sync();
            // the next group's inputs, before the flush: its query operand and fold inputs (for
            // a later group of this chunk, loaded here; for the next chunk's first group, from
            // the prefetch), and every load in flight
            if (more) {  // (only with narrow_max above kNrGroup)
                load_group(cur, g0 + kNrGroup, g_cur);
                v4i ga, gb;
                load_qrows(g_cur, ga, gb);
                __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
                stage_q(ga, gb, Q);
            } else {
                g_cur = g_nx;
                __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
                if (has_next) stage_q(qa, qb, Q);
                // the next chunk's documents and the first-group entries of the chunk after it
                // move into place here, before the atomics, so that no later wait is for them
                g_nx = g_nn;
#pragma unroll
                for (int j = 0; j < kMxChunk / 64; ++j) d[j] = dn[j];
            }
            // flush: one device atomic per (token, run). Every cell of a token's row is read and
            // reset by one LDS exchange (the columns past the chunk's runs hold kTokAbsent), all
            // before the atomics, so that the LDS reads are in flight together.
            for (int tk = 0; tk < ng; ++tk) {  // wave-uniform
                const int64_t row = (int64_t)__builtin_amdgcn_readlane(mytok, 16 * tk) * a.n_docs;
                if (!a.tokcnt) {
                    unsigned v[kMxChunk / 64];
                    int dd[kMxChunk / 64];
#pragma unroll
                    for (int j = 0; j < kMxChunk / 64; ++j) {
                        v[j] = atomicExch(&stab[tk * TPAD + lane + 64 * j], kTokAbsent);
                        dd[j] = rdoc[lane + 64 * j];
                    }
#pragma unroll
                    for (int j = 0; j < kMxChunk / 64; ++j)
                        if (lane + 64 * j < n_runs) atomicMax(&tokmax[row + dd[j]], v[j]);
                } else {
                    // Eq.-1-literal scoring: embeddings of the run retrieved for each token
                    for (int r = lane; r < n_runs; r += 64) {
                        const unsigned v = atomicExch(&stab[tk * TPAD + r], kTokAbsent);
                        const int64_t o = row + rdoc[r];
                        atomicMax(&tokmax[o], v);
                        atomicAdd(&a.tokcnt[o], (unsigned)(rstart[r + 1] - rstart[r]));
                    }
                }
            }
            wave_lds_sync();
            g0 += kNrGroup;
        } while (g0 < nt);
        if (!has_next) break;
        p = pn;
        cur = nx;
    }
}

void launch_wave_prep(const WaveArgs& a, uint32_t* ep, uint32_t last, hipStream_t s) {
    const int64_t n_tok = (int64_t)a.n_q * a.n_qtok;
    int64_t n0 = a.n_c > a.n_q ? a.n_c : a.n_q;
    if (a.sel_slices > 1 && n_tok * kSelBins > n0) n0 = n_tok * kSelBins;
    const int32_t nb0 = (int32_t)((n0 + 255) / 256), nb1 = (int32_t)((n_tok + 3) / 4);
    const dim3 grid((unsigned)(nb0 + nb1 + (n_tok * kDim + 255) / 256));
    switch (a.nbits) {
        case 1: hipLaunchKernelGGL(k_wave_prep<1>, grid, dim3(256), 0, s, a, ep, last, nb0, nb1); break;
        case 2: hipLaunchKernelGGL(k_wave_prep<2>, grid, dim3(256), 0, s, a, ep, last, nb0, nb1); break;
        case 4: hipLaunchKernelGGL(k_wave_prep<4>, grid, dim3(256), 0, s, a, ep, last, nb0, nb1); break;
        default: hipLaunchKernelGGL(k_wave_prep<8>, grid, dim3(256), 0, s, a, ep, last, nb0, nb1); break;
    }
}

void launch_scan_mx(const WaveArgs& a, hipStream_t s) {
    const dim3 grid(a.scan_grid), block(kMxBlock);
    // the first batch of every workgroup is fixed; the counter (set to the grid size by the
    // wave's preparation) hands out the rest
    switch (a.nbits) {
        case 1: hipLaunchKernelGGL(k_scan_mx<1>, grid, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL(k_scan_mx<2>, grid, block, 0, s, a); break;
        case 4: hipLaunchKernelGGL(k_scan_mx<4>, grid, block, 0, s, a); break;
        default: hipLaunchKernelGGL(k_scan_mx<8>, grid, block, 0, s, a); break;
    }
}

void launch_scan_narrow(const WaveArgs& a, int32_t grid, hipStream_t s) {
    if (grid <= 0) return;
    const dim3 g((unsigned)grid), block(kMxBlock);
    switch (a.nbits) {
        case 1: hipLaunchKernelGGL(k_scan_narrow<1>, g, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL(k_scan_narrow<2>, g, block, 0, s, a); break;
        case 4: hipLaunchKernelGGL(k_scan_narrow<4>, g, block, 0, s, a); break;
        default: hipLaunchKernelGGL(k_scan_narrow<8>, g, block, 0, s, a); break;
    }
}

int scan_narrow_blocks_per_cu(int nbits) {
    int n = 0;
    const void* k = nbits == 1   ? (const void*)k_scan_narrow<1>
                    : nbits == 2 ? (const void*)k_scan_narrow<2>
                    : nbits == 4 ? (const void*)k_scan_narrow<4>
                                 : (const void*)k_scan_narrow<8>;
    (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, kMxBlock, 0);
    return n > 0 ? n : 1;
}

int scan_mx_blocks_per_cu(int nbits) {
    int n = 0;
    const void* k = nbits == 1   ? (const void*)k_scan_mx<1>
                    : nbits == 2 ? (const void*)k_scan_mx<2>
                    : nbits == 4 ? (const void*)k_scan_mx<4>
                                 : (const void*)k_scan_mx<8>;
    (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, kMxBlock, 0);
    return n > 0 ? n : 1;
}

}  // namespace warp
