// long_rows.hip -- first level of the row DFT for rows longer than kMaxFastM points
// (fp16 grids).
//
// Algorithm 1's row DFT of a long row is itself split four-step: with m = m1 m2,
// j = m2 j1 + j2 and v = k1 + m1 k2,
//   Z(k1 + m1 k2) = sum_j2 w_m2^(j2 k2) [ w_m^(j2 k1) sum_j1 w_m1^(j1 k1) z(m2 j1 + j2) ].
// This kernel does the bracket: for every grid row u it writes sub-row k1 (m2 points,
// j2 in order) to row k1 N1 + u of the document's sub-row region.  The matrix-core row
// kernels then treat that region as a document of N1 m1 rows of m2 points: the
// frequency -f of (row u, v) is (N1 - u, m - 1 - v) for u > 0 and (0, m - v) for u = 0,
// which is sub-row N1 m1 - r, column m2 - 1 - k2 (r > 0) or column m2 - k2 (r = 0):
// the partner rule those kernels already follow.  The inverse undoes the bracket with
// conjugate roots, from the region back into the grid rows.  The forward carries
// 1 / sqrt(m1), so with the row tables' 1 / sqrt(m2) each spectrum carries 1 / sqrt(m)
// as before; the inverse is unscaled.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "fft_core.hpp"
#include "kernels.hpp"

namespace rubiconv {

namespace {

// Workgroup = grid row u of one item and one pair block; thread = (pair p, j2 lane).
template <int M1, bool INV>
__global__ __launch_bounds__(256) void lr_step_kernel(__half2* __restrict__ grid, int64_t grid_pb_stride,
                                                      LrItem it, const float2* __restrict__ tw, int n1) {
    const int u = blockIdx.x, pb = blockIdx.y;
    const int p = threadIdx.x & 15, jl = threadIdx.x >> 4;
    __half2* base = grid + pb * grid_pb_stride + p;
    const int m = it.m, m2 = it.m2;
    const float2* w = tw + it.tw_off;  // w_m^h = exp(-2 pi i h / m)
    const int64_t row = it.real_off + static_cast<int64_t>(u) * m;
    for (int j2 = jl; j2 < m2; j2 += 16) {
        float2 v[M1];
        if constexpr (!INV) {
#pragma unroll
            for (int j1 = 0; j1 < M1; ++j1) v[j1] = __half22float2(base[(row + m2 * j1 + j2) * 16]);
            Dft<M1, -1>::run(v);
            const float sc = 1.0f / sqrtf(static_cast<float>(M1));
#pragma unroll
            for (int k1 = 0; k1 < M1; ++k1) {
                const float2 z = cscale(cmul(v[k1], w[j2 * k1]), sc);
                base[(it.virt_off + (static_cast<int64_t>(k1) * n1 + u) * m2 + j2) * 16] = __float22half2_rn(z);
            }
        } else {
#pragma unroll
            for (int k1 = 0; k1 < M1; ++k1) {
                const float2 z = __half22float2(base[(it.virt_off + (static_cast<int64_t>(k1) * n1 + u) * m2 + j2) * 16]);
                v[k1] = cmul(z, cconj(w[j2 * k1]));
            }
            Dft<M1, 1>::run(v);
#pragma unroll
            for (int j1 = 0; j1 < M1; ++j1) base[(row + m2 * j1 + j2) * 16] = __float22half2_rn(v[j1]);
        }
    }
}

}  // namespace

hipError_t launch_lr_step(bool inverse, void* grid, int64_t grid_pb_stride, const LrItem& it,
                          const float2* tw, int n1, int npb, hipStream_t stream) {
    const dim3 g(n1, npb), b(256);
    __half2* gp = static_cast<__half2*>(grid);
#define RUBICONV_LR(M)                                                                                  \
    case M:                                                                                             \
        if (inverse)                                                                                    \
            hipLaunchKernelGGL((lr_step_kernel<M, true>), g, b, 0, stream, gp, grid_pb_stride, it, tw, n1); \
        else                                                                                            \
            hipLaunchKernelGGL((lr_step_kernel<M, false>), g, b, 0, stream, gp, grid_pb_stride, it, tw, n1); \
        break;
    switch (it.m1) {
        RUBICONV_LR(2) RUBICONV_LR(3) RUBICONV_LR(4) RUBICONV_LR(5) RUBICONV_LR(6) RUBICONV_LR(8)
        RUBICONV_LR(9) RUBICONV_LR(10) RUBICONV_LR(12) RUBICONV_LR(15) RUBICONV_LR(16) RUBICONV_LR(20)
        RUBICONV_LR(24) RUBICONV_LR(25) RUBICONV_LR(30) RUBICONV_LR(32)
        default: return hipErrorInvalidValue;
    }
#undef RUBICONV_LR
    return hipGetLastError();
}

}  // namespace rubiconv
