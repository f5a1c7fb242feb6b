// row_fast.hip -- register-resident row pass for row sizes m = M1 * M2 <= 256.
//
// One workgroup handles grid row u (0 <= u <= N1/2) of one document and its
// conjugate partner row (N1 - u) mod N1, for the 16 channel pairs of one pair
// block: 32 "lines" (row r in {0, 1} x pair p), each an m-point row.  Thread
// (p, r, q) = (tid % 16, tid / 16 % 2, tid / 32).  The m-point DFT is split
// j = M2 j1 + j2, v = k1 + M1 k2:
//   stage 1 (thread q = j2): M1-point DFT over j1 -> k1, times w_m^(j2 k1);
//   exchange through LDS ([element][32 lines], conflict free);
//   stage 2 (thread q = k1): M2-point DFT over j2 -> k2.
// The same rows of the document's filter class (the filter pair after its
// column stage) go through the same row DFT first; the conjugate-symmetry
// separation gives the filter spectra, which multiply the data rows' spectrum
// in registers (Algorithm 3's pointwise product on the 2-D grid).  The inverse
// row DFT then writes the rows back in place.  The frequency -f partner of
// f = u + N1 v sits at row (N1 - u) mod N1, column (-v - [u > 0]) mod m.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "fft_core.hpp"
#include "kernels.hpp"
#include "row_sizes.hpp"

namespace rubiconv {

namespace {

__device__ __forceinline__ float2 gload(const float2* p) { return *p; }
__device__ __forceinline__ float2 gload(const __half2* p) { return __half22float2(*p); }
__device__ __forceinline__ void gstore(float2* p, float2 v) { *p = v; }
__device__ __forceinline__ void gstore(__half2* p, float2 v) { *p = __float22half2_rn(v); }

__device__ __forceinline__ int partner_v(int u, int v, int m) {
    return u == 0 ? (v == 0 ? 0 : m - v) : m - 1 - v;
}

// Forward m-point DFT of the rows held in v (stage-1 layout) through `lds`;
// leaves w[k2] = Z(row r, v = q + M1 k2) in registers and Z in natural order in
// LDS for the partner lookups.  Every thread of the workgroup must call it.
template <int M1, int M2>
__device__ __forceinline__ void row_forward(float2 (&v)[M1], float2 (&w)[M2], float2* lds,
                                            const float2* roots, bool act, int q, int line) {
    if (act && q < M2) {
        Dft<M1, -1>::run(v);
#pragma unroll
        for (int k1 = 1; k1 < M1; ++k1) v[k1] = cmul(v[k1], roots[q * k1]);
#pragma unroll
        for (int k1 = 0; k1 < M1; ++k1) lds[(k1 * M2 + q) * 32 + line] = v[k1];
    }
    __syncthreads();
    if (act) {
#pragma unroll
        for (int j2 = 0; j2 < M2; ++j2) w[j2] = lds[(q * M2 + j2) * 32 + line];
        Dft<M2, -1>::run(w);
    }
    __syncthreads();
    if (act) {
#pragma unroll
        for (int k2 = 0; k2 < M2; ++k2) lds[(q + M1 * k2) * 32 + line] = w[k2];
    }
    __syncthreads();
}

template <int M1, int M2, class G>
__global__ __launch_bounds__(32 * M1) void row_fast_kernel(G* __restrict__ grid,
                                                           int64_t grid_pb_stride,
                                                           const G* __restrict__ fgrid,
                                                           int64_t fgrid_pb_stride,
                                                           const Seg* __restrict__ segs,
                                                           const int32_t* __restrict__ list,
                                                           const float2* __restrict__ tw, int n1,
                                                           int corr) {
    constexpr int M = M1 * M2;
    __shared__ float2 lds[M * 32];
    __shared__ float2 roots[M];  // w_m^h, h < m

    const int nu = n1 / 2 + 1;
    const Seg* sg = segs + list[blockIdx.x / nu];
    const int u = blockIdx.x % nu;
    const int ub = (n1 - u) & (n1 - 1);
    const int nrows = (ub == u) ? 1 : 2;
    const int pb = blockIdx.y;
    const int tid = threadIdx.x;
    const int p = tid & 15, r = (tid >> 4) & 1, q = tid >> 5;
    const int line = tid & 31;
    const bool act = r < nrows;
    // the partner of line (r, p) is line (1 - r, p) for two rows, itself for one
    const int pline = nrows == 2 ? (line ^ 16) : line;
    const int urow = r ? ub : u;

    const float2* twm = tw + sg->tw_off;
    for (int h = tid; h < M; h += 32 * M1) roots[h] = twm[h];

    // both row sets are read up front: the filter class rows and the document rows
    G* row = grid + pb * grid_pb_stride +
             (sg->grid_off + static_cast<int64_t>(urow) * M) * kPairsPerBlock + p;
    const G* frow = fgrid + pb * fgrid_pb_stride +
                    (static_cast<int64_t>(sg->spec_off) + static_cast<int64_t>(urow) * M) *
                        kPairsPerBlock + p;
    float2 vh[M1], vx[M1];
    if (act && q < M2) {
#pragma unroll
        for (int j1 = 0; j1 < M1; ++j1) vh[j1] = gload(frow + (M2 * j1 + q) * kPairsPerBlock);
#pragma unroll
        for (int j1 = 0; j1 < M1; ++j1) vx[j1] = gload(row + (M2 * j1 + q) * kPairsPerBlock);
    }
    __syncthreads();  // roots ready

    // filter spectra S, Df at this thread's elements (for r = 1 they belong to -f)
    float2 w[M2], s[M2], df[M2];
    row_forward<M1, M2>(vh, w, lds, roots, act, q, line);
    // the stored grids are DFT / sqrt(N1): S and Df carry sqrt(N1) / (2 m)
    const float c = 0.5f * sqrtf(static_cast<float>(n1)) / static_cast<float>(M);
    if (act) {
#pragma unroll
        for (int k2 = 0; k2 < M2; ++k2) {
            const int vv = q + M1 * k2;
            const float2 par = lds[partner_v(u, vv, M) * 32 + pline];
            // correlation: the filter spectrum read at -f (its conjugate for real taps)
            const bool own_first = (r == 0) != (corr != 0);
            filter_sdf(own_first ? w[k2] : par, own_first ? par : w[k2], c, s[k2], df[k2]);
        }
    }
    __syncthreads();  // partner reads done before the data reuses LDS

    row_forward<M1, M2>(vx, w, lds, roots, act, q, line);
    if (act) {
#pragma unroll
        for (int k2 = 0; k2 < M2; ++k2) {
            const int vv = q + M1 * k2;
            const float2 par = lds[partner_v(u, vv, M) * 32 + pline];
            w[k2] = r == 0 ? product_f(w[k2], par, s[k2], df[k2])
                           : product_neg_f(par, w[k2], s[k2], df[k2]);
        }
    }
    __syncthreads();  // every partner read is done before LDS is reused

    // inverse row DFT: thread q = k1 holds W[k1 + M1 k2]
    if (act) {
        Dft<M2, 1>::run(w);  // over k2 -> j2
#pragma unroll
        for (int j2 = 1; j2 < M2; ++j2) w[j2] = cmul(w[j2], cconj(roots[j2 * q]));
#pragma unroll
        for (int j2 = 0; j2 < M2; ++j2) lds[(j2 * M1 + q) * 32 + line] = w[j2];
    }
    __syncthreads();
    if (act && q < M2) {
#pragma unroll
        for (int k1 = 0; k1 < M1; ++k1) vx[k1] = lds[(q * M1 + k1) * 32 + line];
        Dft<M1, 1>::run(vx);  // over k1 -> j1, thread q = j2
#pragma unroll
        for (int j1 = 0; j1 < M1; ++j1) gstore(row + (M2 * j1 + q) * kPairsPerBlock, vx[j1]);
    }
}

template <int M1, int M2, class G>
hipError_t launch_mg(void* grid, int64_t gs, const void* fgrid, int64_t fs, const Seg* segs,
                     const int32_t* list, int nlist, const float2* tw, int n1, int npb,
                     int corr, hipStream_t stream) {
    const dim3 g(nlist * (n1 / 2 + 1), npb), b(32 * M1);
    hipLaunchKernelGGL((row_fast_kernel<M1, M2, G>), g, b, 0, stream, static_cast<G*>(grid), gs,
                       static_cast<const G*>(fgrid), fs, segs, list, tw, n1, corr);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_row_fast(int m, bool half, void* grid, int64_t grid_pb_stride, const void* fgrid,
                           int64_t fgrid_pb_stride, const Seg* segs, const int32_t* list,
                           int nlist, const float2* tw, int n1, int npb, int corr,
                           hipStream_t stream) {
    if (nlist == 0) return hipSuccess;
    switch (m) {
#define RUBICONV_CASE(mm, a, b)                                                                  \
    case mm:                                                                                     \
        return half ? launch_mg<a, b, __half2>(grid, grid_pb_stride, fgrid, fgrid_pb_stride, segs, \
                                               list, nlist, tw, n1, npb, corr, stream)            \
                    : launch_mg<a, b, float2>(grid, grid_pb_stride, fgrid, fgrid_pb_stride, segs,  \
                                              list, nlist, tw, n1, npb, corr, stream);
        RUBICONV_ROW_SIZES(RUBICONV_CASE)
#undef RUBICONV_CASE
        default:
            return hipErrorInvalidValue;
    }
}

}  // namespace rubiconv
