// Query-token x centroid scores on the matrix cores (Section 4.3: S = C q^T,
// a matrix product since both sides are normalised).
//
// out[t][c] = sum_d q[t][d] * centroids[c][d] in fp32 with v_mfma_f32_16x16x4_f32.
// These scores only steer centroid selection: every centroid that lands near a
// selection boundary is rescored in fp64 by the selection kernel, so the result
// of the search does not depend on the accumulation order used here.
//
// Tiling: a workgroup of 4 waves owns a 128-token x 128-centroid tile; K = 128
// is staged through LDS in two halves of 64 with coalesced 16-byte loads, rows
// padded to 68 floats so that the 16 lanes of each ds_read_b128 pass hit 16
// distinct 4-bank groups. Each wave computes a 64 x 64 block as 4 x 4 MFMA
// blocks of 16 x 16. Lane group g = lane / 16 reads 4 consecutive k with one
// 16-byte LDS read and feeds them to 4 successive MFMA steps: step s of a
// 16-wide k slice uses k = 4 g + s on both operands, so every k is summed once.
#include "engine.h"

namespace warp {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kGT = 128;       // tile rows (tokens) and columns (centroids)
constexpr int kGK = 64;        // k staged per half
constexpr int kGPad = kGK + 4;  // padded LDS row (floats)

// BINS: write the selection histogram bin of each score (u16); else the fp32 score.
template <bool BINS>
__global__ __launch_bounds__(256) void k_filter_gemm(const float* __restrict__ q, int32_t n_tok,
                                                     const float* __restrict__ cen, int32_t n_c,
                                                     void* __restrict__ out) {
    __shared__ float As[kGT * kGPad];
    __shared__ float Bs[kGT * kGPad];
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int li = lane & 15;
    const int g = lane >> 4;
    const int64_t t_base = (int64_t)blockIdx.y * kGT;
    const int64_t c_base = (int64_t)blockIdx.x * kGT;
    const int wr = (wave >> 1) * 64;  // this wave's rows within the tile
    const int wc = (wave & 1) * 64;   // and columns

    floatx4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = (floatx4){0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int half = 0; half < 2; ++half) {
        if (half) __syncthreads();
        // stage: 128 rows x 64 floats per operand = 2048 float4, 8 per thread
#pragma unroll
        for (int it = 0; it < 8; ++it) {
            const int f = tid + 256 * it;
            const int row = f >> 4, c4 = f & 15;
            const int64_t tr = t_base + row, cr = c_base + row;
            float4 va = make_float4(0.f, 0.f, 0.f, 0.f), vb = va;
            if (tr < n_tok) va = *reinterpret_cast<const float4*>(q + tr * kDim + half * kGK + 4 * c4);
            if (cr < n_c) vb = *reinterpret_cast<const float4*>(cen + cr * kDim + half * kGK + 4 * c4);
            *reinterpret_cast<float4*>(&As[row * kGPad + 4 * c4]) = va;
            *reinterpret_cast<float4*>(&Bs[row * kGPad + 4 * c4]) = vb;
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < kGK; ks += 16) {
            float4 a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                a[i] = *reinterpret_cast<const float4*>(&As[(wr + 16 * i + li) * kGPad + ks + 4 * g]);
                b[i] = *reinterpret_cast<const float4*>(&Bs[(wc + 16 * i + li) * kGPad + ks + 4 * g]);
            }
#pragma unroll
            for (int s = 0; s < 4; ++s) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float av = s == 0 ? a[i].x : s == 1 ? a[i].y : s == 2 ? a[i].z : a[i].w;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const float bv = s == 0 ? b[j].x : s == 1 ? b[j].y : s == 2 ? b[j].z : b[j].w;
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[i][j], 0, 0, 0);
                    }
                }
            }
        }
    }
    // D[r][cidx] of a 16 x 16 block sits in lane cidx + 16 * (r / 4), element r % 4.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t c = c_base + wc + 16 * j + li;
            if (c >= n_c) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t t = t_base + wr + 16 * i + 4 * g + r;
                if (t >= n_tok) continue;
                if (BINS) static_cast<uint16_t*>(out)[t * n_c + c] = (uint16_t)score_bin(acc[i][j][r]);
                else static_cast<float*>(out)[t * n_c + c] = acc[i][j][r];
            }
        }
    }
}

void launch_filter_gemm(const float* q, int32_t n_tok, const float* c, int32_t n_c, uint16_t* out_bins,
                        float* out_scores, hipStream_t s) {
    dim3 grid((n_c + kGT - 1) / kGT, (n_tok + kGT - 1) / kGT);
    if (out_bins)
        hipLaunchKernelGGL(k_filter_gemm<true>, grid, dim3(256), 0, s, q, n_tok, c, n_c, (void*)out_bins);
    else
        hipLaunchKernelGGL(k_filter_gemm<false>, grid, dim3(256), 0, s, q, n_tok, c, n_c, (void*)out_scores);
}

}  // namespace warp
