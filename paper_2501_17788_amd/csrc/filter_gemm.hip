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
// Tiling: a workgroup of 4 waves owns a 128-token x 128-centroid tile; K = 128 is
// staged through LDS in two halves of 64, each fp32 row split into hi and lo fp16 rows
// padded to 72 halves (144 bytes: the 16 rows of a 16-lane ds_read_b128 start in 16
// distinct 4-bank groups). Each wave computes a 64 x 64 block as 4 x 4 MFMA blocks of
// 16 x 16; lane group g = lane / 16 supplies the 8 consecutive k = ks + 8 g .. ks + 8 g + 7
// of both operands to each 32-wide k step ks, so every k is summed once.
#include "engine.h"

namespace warp {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));

constexpr int kGT = 128;        // tile rows (tokens) and columns (centroids)
constexpr int kGK = 64;         // k staged per half
constexpr int kGPad = kGK + 8;  // padded LDS row (halves)

__device__ __forceinline__ void split4(const float4 v, half4& hi, half4& lo) {
    hi = (half4){(_Float16)v.x, (_Float16)v.y, (_Float16)v.z, (_Float16)v.w};
    lo = (half4){(_Float16)(v.x - (float)hi.x), (_Float16)(v.y - (float)hi.y), (_Float16)(v.z - (float)hi.z),
                 (_Float16)(v.w - (float)hi.w)};
}

// BINS: write the selection histogram bin of each score (u16); else the fp32 score.
template <bool BINS>
__global__ __launch_bounds__(256) void k_filter_gemm(const float* __restrict__ q, int32_t n_tok,
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
        // stage: 128 rows x 64 floats per operand = 2048 float4, 8 per thread, split on the way
#pragma unroll
        for (int it = 0; it < 8; ++it) {
            const int f = tid + 256 * it;
            const int row = f >> 4, c4 = f & 15;
            const int64_t tr = t_base + row, cr = c_base + row;
            float4 va = make_float4(0.f, 0.f, 0.f, 0.f), vb = va;
            if (tr < n_tok) va = *reinterpret_cast<const float4*>(q + tr * kDim + half * kGK + 4 * c4);
            if (cr < n_c) vb = *reinterpret_cast<const float4*>(cen + cr * kDim + half * kGK + 4 * c4);
            half4 hi, lo;
            split4(va, hi, lo);
            *reinterpret_cast<half4*>(&Ah[row * kGPad + 4 * c4]) = hi;
            *reinterpret_cast<half4*>(&Al[row * kGPad + 4 * c4]) = lo;
            split4(vb, hi, lo);
            *reinterpret_cast<half4*>(&Bh[row * kGPad + 4 * c4]) = hi;
            *reinterpret_cast<half4*>(&Bl[row * kGPad + 4 * c4]) = lo;
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < kGK; ks += 32) {
            half8 ah[4], al[4], bh[4], bl[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int ra = (wr + 16 * i + li) * kGPad + ks + 8 * g;
                const int rb = (wc + 16 * i + li) * kGPad + ks + 8 * g;
                ah[i] = *reinterpret_cast<const half8*>(&Ah[ra]);
                al[i] = *reinterpret_cast<const half8*>(&Al[ra]);
                bh[i] = *reinterpret_cast<const half8*>(&Bh[rb]);
                bl[i] = *reinterpret_cast<const half8*>(&Bl[rb]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[i], bh[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[i], bl[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[i], bh[j], acc[i][j], 0, 0, 0);
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
