// Query-token x centroid scores on the matrix cores (Section 4.3: S = C q^T,
// a matrix product since both sides are normalised).
//
// out[t][c] = sum_d q[t][d] * centroids[c][d] in fp32 with v_mfma_f32_16x16x4_f32.
// These scores only steer centroid selection: every centroid that lands near a
// selection boundary is rescored in fp64 by the selection kernel, so the result
// of the search does not depend on the accumulation order used here.
//
// Work split: a workgroup of 4 waves owns a 64-token x 64-centroid tile, each
// wave a 32 x 32 block (2 x 2 MFMA blocks). Lane group g = lane / 16 supplies the
// K index k = 32 g + s of MFMA step s, so every lane streams one contiguous
// 128-byte half-row of its token and of its centroid with 16-byte loads; the
// sum over all 128 dimensions is the same whatever K order the steps take.
#include "engine.h"

namespace warp {

typedef float floatx4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void k_filter_gemm(const float* __restrict__ q, int32_t n_tok,
                                                     const float* __restrict__ cen, int32_t n_c,
                                                     float* __restrict__ out) {
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int li = lane & 15;
    const int g = lane >> 4;
    const int64_t t0 = (int64_t)blockIdx.y * 64 + (wave >> 1) * 32;
    const int64_t c0 = (int64_t)blockIdx.x * 64 + (wave & 1) * 32;

    const int64_t ta = t0 + li, tb = t0 + 16 + li;
    const int64_t ca = c0 + li, cb = c0 + 16 + li;
    const bool va = ta < n_tok, vb = tb < n_tok, vc = ca < n_c, vd = cb < n_c;
    const float4* pa = reinterpret_cast<const float4*>(q + (va ? ta : 0) * kDim + 32 * g);
    const float4* pb = reinterpret_cast<const float4*>(q + (vb ? tb : 0) * kDim + 32 * g);
    const float4* pc = reinterpret_cast<const float4*>(cen + (vc ? ca : 0) * kDim + 32 * g);
    const float4* pd = reinterpret_cast<const float4*>(cen + (vd ? cb : 0) * kDim + 32 * g);

    floatx4 acc00 = {0.f, 0.f, 0.f, 0.f}, acc01 = acc00, acc10 = acc00, acc11 = acc00;
    const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) {
        const float4 a0 = va ? pa[kc] : zero;
        const float4 a1 = vb ? pb[kc] : zero;
        const float4 b0 = vc ? pc[kc] : zero;
        const float4 b1 = vd ? pd[kc] : zero;
        const float av0[4] = {a0.x, a0.y, a0.z, a0.w};
        const float av1[4] = {a1.x, a1.y, a1.z, a1.w};
        const float bv0[4] = {b0.x, b0.y, b0.z, b0.w};
        const float bv1[4] = {b1.x, b1.y, b1.z, b1.w};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            acc00 = __builtin_amdgcn_mfma_f32_16x16x4f32(av0[s], bv0[s], acc00, 0, 0, 0);
            acc01 = __builtin_amdgcn_mfma_f32_16x16x4f32(av0[s], bv1[s], acc01, 0, 0, 0);
            acc10 = __builtin_amdgcn_mfma_f32_16x16x4f32(av1[s], bv0[s], acc10, 0, 0, 0);
            acc11 = __builtin_amdgcn_mfma_f32_16x16x4f32(av1[s], bv1[s], acc11, 0, 0, 0);
        }
    }
    // D[i][j] of a 16 x 16 block sits in lane j + 16 * (i / 4), element i % 4.
    const floatx4 accs[2][2] = {{acc00, acc01}, {acc10, acc11}};
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) {
            const int64_t c = c0 + 16 * bj + li;
            if (c >= n_c) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t t = t0 + 16 * bi + 4 * g + r;
                if (t < n_tok) out[t * n_c + c] = accs[bi][bj][r];
            }
        }
    }
}

void launch_filter_gemm(const float* q, int32_t n_tok, const float* c, int32_t n_c, float* out,
                        hipStream_t s) {
    dim3 grid((n_c + 63) / 64, (n_tok + 63) / 64);
    hipLaunchKernelGGL(k_filter_gemm, grid, dim3(256), 0, s, q, n_tok, c, n_c, out);
}

}  // namespace warp
