// Query-token x centroid scores on the matrix cores (Section 4.3: S = C q^T,
// a matrix product since both sides are normalised).
//
// Every fp32 operand x is split into two fp16 parts, hi = fp16(x) and
// lo = fp16(x - hi), so that |x - hi - lo| <= 2^-22 |x| + 2^-25 for |x| <= 1.001
// (the second term from fp16 subnormals), and
//     out[t][c] = sum_d (q_hi c_hi + q_hi c_lo + q_lo c_hi)[t][c][d]
// is accumulated in fp32 by v_mfma_f32_16x16x32_f16 (every fp16 product is exact in
// fp32). The split and the dropped lo x lo term change a score by at most
// 3 * 2^-22 sum_d |q_d c_d| + 2^-24 sqrt(128), about 1.4e-6 for unit vectors, and the
// fp32 accumulation of the 384 products by at most gamma_384 sum_d |q_d c_d| (2.3e-5):
// within the 2^-13 that centroid selection and the index build assume. These scores
// only steer selection: every centroid that lands near a selection boundary is
// rescored in fp64, so no result depends on how they were accumulated.
//
// Tiling: a workgroup of 4 waves computes 128-token x 128-centroid tiles; K = 128 is
// staged through LDS in quarters of 32, each fp32 row split into hi and lo fp16 rows
// padded to 40 halves (80 bytes). Each wave computes a 64 x 64 block as 4 x 4 MFMA blocks
// of 16 x 16, with the centroids as the rows of each product and the tokens as its
// columns, so that a lane holds four consecutive centroids of one token and writes them
// with one store; lane group g = lane / 16 supplies the 8 consecutive k = 8 g .. 8 g + 7 of
// both operands to each 32-wide k step, so every k is summed once.
#include "engine.h"

namespace warp {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));

constexpr int kGT = 128;        // tile rows (tokens) and columns (centroids)
constexpr int kGK = 32;         // k staged per quarter
constexpr int kGPad = kGK + 8;  // padded LDS row (halves): 80 bytes

__device__ __forceinline__ void split4(const float4 v, half4& hi, half4& lo) {
    hi = (half4){(_Float16)v.x, (_Float16)v.y, (_Float16)v.z, (_Float16)v.w};
    lo = (half4){(_Float16)(v.x - (float)hi.x), (_Float16)(v.y - (float)hi.y), (_Float16)(v.z - (float)hi.z),
                 (_Float16)(v.w - (float)hi.w)};
}

// BINS: write the selection histogram bin of each score (u16); else the fp32 score.
// A persistent grid (as many workgroups as fit the GPU at once) walks the output tiles,
// token tile major; workgroup b takes tiles b, b + G, ... While one quarter of K is
// multiplied out of LDS, the fp32 rows of the next quarter (or of the next tile's first
// quarter, during the epilogue as well) are in flight into registers.
template <bool BINS>
__global__ __launch_bounds__(256, 2) void k_filter_gemm(const float* __restrict__ q, int32_t n_tok,
                                                     const float* __restrict__ cen, int32_t n_c,
                                                     void* __restrict__ out) {
    __shared__ __attribute__((aligned(16))) _Float16 Ah[kGT * kGPad];
    __shared__ __attribute__((aligned(16))) _Float16 Al[kGT * kGPad];
    __shared__ __attribute__((aligned(16))) _Float16 Bh[kGT * kGPad];
    __shared__ __attribute__((aligned(16))) _Float16 Bl[kGT * kGPad];
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int li = lane & 15;
    const int g = lane >> 4;
    const int wr = (wave >> 1) * 64;  // this wave's rows within the tile
    const int wc = (wave & 1) * 64;   // and columns
    const int64_t tiles_c = (n_c + kGT - 1) / kGT;
    const int64_t n_tiles = tiles_c * ((n_tok + kGT - 1) / kGT);
    const bool vec4 = (n_c & 3) == 0;  // rows of the output start 4-element aligned

    // 128 rows x 32 floats per operand = 1024 float4, 4 per thread
    auto load = [&](int64_t tile, int quarter, float4 (&va)[4], float4 (&vb)[4]) {
        const int64_t t_base = tile / tiles_c * kGT, c_base = tile % tiles_c * kGT;
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int f = tid + 256 * it;
            const int row = f >> 3, c4 = f & 7;
            const int64_t tr = t_base + row, cr = c_base + row;
            va[it] = make_float4(0.f, 0.f, 0.f, 0.f);
            vb[it] = va[it];
            if (tr < n_tok) va[it] = *reinterpret_cast<const float4*>(q + tr * kDim + quarter * kGK + 4 * c4);
            if (cr < n_c) vb[it] = *reinterpret_cast<const float4*>(cen + cr * kDim + quarter * kGK + 4 * c4);
        }
    };
    auto stage = [&](const float4 (&va)[4], const float4 (&vb)[4]) {
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int f = tid + 256 * it;
            const int row = f >> 3, c4 = f & 7;
            half4 hi, lo;
            split4(va[it], hi, lo);
            *reinterpret_cast<half4*>(&Ah[row * kGPad + 4 * c4]) = hi;
            *reinterpret_cast<half4*>(&Al[row * kGPad + 4 * c4]) = lo;
            split4(vb[it], hi, lo);
            *reinterpret_cast<half4*>(&Bh[row * kGPad + 4 * c4]) = hi;
            *reinterpret_cast<half4*>(&Bl[row * kGPad + 4 * c4]) = lo;
        }
    };
    floatx4 acc[4][4];
    auto multiply = [&]() {
#pragma unroll
        for (int ks = 0; ks < kGK; ks += 32) {
            half8 bh[4], bl[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int rb = (wc + 16 * j + li) * kGPad + ks + 8 * g;
                bh[j] = *reinterpret_cast<const half8*>(&Bh[rb]);
                bl[j] = *reinterpret_cast<const half8*>(&Bl[rb]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int ra = (wr + 16 * i + li) * kGPad + ks + 8 * g;
                const half8 ah = *reinterpret_cast<const half8*>(&Ah[ra]);
                const half8 al = *reinterpret_cast<const half8*>(&Al[ra]);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(bh[j], ah, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(bl[j], ah, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(bh[j], al, acc[i][j], 0, 0, 0);
                }
            }
        }
    };

    int64_t tile = blockIdx.x;
    if (tile >= n_tiles) return;
    float4 va[4], vb[4];
    load(tile, 0, va, vb);
    for (;;) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = (floatx4){0.f, 0.f, 0.f, 0.f};
        const int64_t next = tile + gridDim.x;
#pragma unroll 1
        for (int h = 0; h < 4; ++h) {
            stage(va, vb);
            __syncthreads();
            if (h < 3) load(tile, h + 1, va, vb);
            else if (next < n_tiles) load(next, 0, va, vb);
            multiply();
            if (h < 3) __syncthreads();
        }
        // D[r][col] of a 16 x 16 block sits in lane col + 16 * (r / 4), element r % 4: lane (li, g)
        // holds centroids 4 g .. 4 g + 3 of block j against token li of block i.
        const int64_t t_base = tile / tiles_c * kGT, c_base = tile % tiles_c * kGT;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t t = t_base + wr + 16 * i + li;
            if (t >= n_tok) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t c0 = c_base + wc + 16 * j + 4 * g;
                const int64_t o = t * n_c + c0;
                if (vec4 && c0 + 3 < n_c) {  // four consecutive outputs, aligned: one store
                    if (BINS) {
                        const uint32_t lo = (uint32_t)score_bin(acc[i][j][0]) | ((uint32_t)score_bin(acc[i][j][1]) << 16);
                        const uint32_t hi = (uint32_t)score_bin(acc[i][j][2]) | ((uint32_t)score_bin(acc[i][j][3]) << 16);
                        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(out) + o) = make_uint2(lo, hi);
                    } else {
                        *reinterpret_cast<float4*>(static_cast<float*>(out) + o) =
                            make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
                    }
                    continue;
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (c0 + r >= n_c) continue;
                    if (BINS) static_cast<uint16_t*>(out)[o + r] = (uint16_t)score_bin(acc[i][j][r]);
                    else static_cast<float*>(out)[o + r] = acc[i][j][r];
                }
            }
        }
        if (next >= n_tiles) break;
        tile = next;
        __syncthreads();  // every wave has read the LDS operands before they are replaced
    }
}

// Workgroups of the filter GEMM that fit the current device at once.
int filter_gemm_grid() {
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, k_filter_gemm<true>, 256, 0) != hipSuccess) {
        (void)hipGetLastError();
        return 512;
    }
    return cus * (per > 0 ? per : 1);
}

void launch_filter_gemm(const float* q, int32_t n_tok, const float* c, int32_t n_c, uint16_t* out_bins,
                        float* out_scores, hipStream_t s) {
    const int64_t tiles = (int64_t)((n_c + kGT - 1) / kGT) * ((n_tok + kGT - 1) / kGT);
    static thread_local int grid_cap = 0;
    if (grid_cap == 0) grid_cap = filter_gemm_grid();
    const dim3 grid((unsigned)(tiles < grid_cap ? tiles : grid_cap));
    if (tiles == 0) return;
    if (out_bins)
        hipLaunchKernelGGL(k_filter_gemm<true>, grid, dim3(256), 0, s, q, n_tok, c, n_c, (void*)out_bins);
    else
        hipLaunchKernelGGL(k_filter_gemm<false>, grid, dim3(256), 0, s, q, n_tok, c, n_c, (void*)out_scores);
}

}  // namespace warp
