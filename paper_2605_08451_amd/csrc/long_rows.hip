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

__device__ __forceinline__ __amdgpu_buffer_rsrc_t lr_buffer(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000);
}

// Workgroup = 16 columns j2 of grid row u of one item and one pair block; thread =
// (pair p, column j2).
// Both the grid row and the row's slice of the sub-row region are addressed through
// buffer resources with workgroup-uniform bases, so each access costs one 32-bit
// offset instead of a 64-bit address.
template <int M1, bool INV>
__global__ __launch_bounds__(256) void lr_step_kernel(__half2* __restrict__ grid, int64_t grid_pb_stride,
                                                      LrItem it, const float2* __restrict__ tw, int n1) {
    const int m = it.m, m2 = it.m2;
    const int nj = (m2 + 15) >> 4;
    const int u = blockIdx.x / nj, pb = blockIdx.y;
    const int p = threadIdx.x & 15, j2 = (blockIdx.x - u * nj) * 16 + (threadIdx.x >> 4);
    if (j2 >= m2) return;
    __half2* gb = grid + pb * grid_pb_stride;
    const auto row = lr_buffer(gb + (it.real_off + static_cast<int64_t>(u) * m) * 16,
                               static_cast<uint32_t>(m) * 64u);
    // sub-row k1 of row u starts at (k1 n1 + u) m2 points into the region
    const uint32_t sub_stride = static_cast<uint32_t>(n1) * static_cast<uint32_t>(m2) * 64u;
    const auto sub = lr_buffer(gb + (it.virt_off + static_cast<int64_t>(u) * m2) * 16,
                               (M1 - 1) * sub_stride + static_cast<uint32_t>(m2) * 64u);
    const auto tws = lr_buffer(tw + it.tw_off, static_cast<uint32_t>(m) * 8u);  // w_m^h = exp(-2 pi i h / m)
    const uint32_t row_stride = static_cast<uint32_t>(m2) * 64u;
    {
        const uint32_t lane_off = static_cast<uint32_t>(j2 * 16 + p) * 4u;
        float2 v[M1];
        if constexpr (!INV) {
#pragma unroll
            for (int j1 = 0; j1 < M1; ++j1)
                v[j1] = __half22float2(__builtin_bit_cast(
                    __half2, __builtin_amdgcn_raw_buffer_load_b32(row, static_cast<int>(lane_off + j1 * row_stride), 0, 0)));
            // w_m^(j2 k1) as powers of w_m^j2: one table load, and no load waits
            // between the stores (a buffer load may not move past a buffer store)
            const float2 w1 = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(tws, j2 * 8, 0, 0));
            Dft<M1, -1>::run(v);
            const float sc = 1.0f / sqrtf(static_cast<float>(M1));
            float2 w = make_float2(sc, 0.0f);
#pragma unroll
            for (int k1 = 0; k1 < M1; ++k1) {
                const float2 z = cmul(v[k1], w);
                w = cmul(w, w1);
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, __float22half2_rn(z)), sub,
                                                      static_cast<int>(lane_off + k1 * sub_stride), 0, 0);
            }
        } else {
            const float2 w1 = cconj(__builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(tws, j2 * 8, 0, 0)));
            float2 w = make_float2(1.0f, 0.0f);
#pragma unroll
            for (int k1 = 0; k1 < M1; ++k1) {
                const float2 z = __half22float2(__builtin_bit_cast(
                    __half2, __builtin_amdgcn_raw_buffer_load_b32(sub, static_cast<int>(lane_off + k1 * sub_stride), 0, 0)));
                v[k1] = cmul(z, w);
                w = cmul(w, w1);
            }
            Dft<M1, 1>::run(v);
#pragma unroll
            for (int j1 = 0; j1 < M1; ++j1)
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, __float22half2_rn(v[j1])), row,
                                                      static_cast<int>(lane_off + j1 * row_stride), 0, 0);
        }
    }
}

}  // namespace

hipError_t launch_lr_step(bool inverse, void* grid, int64_t grid_pb_stride, const LrItem& it,
                          const float2* tw, int n1, int npb, hipStream_t stream) {
    const dim3 g(n1 * ((it.m2 + 15) / 16), npb), b(256);
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
