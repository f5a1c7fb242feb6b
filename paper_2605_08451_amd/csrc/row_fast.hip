// row_fast.hip -- register-resident row pass for row sizes m = M1 * M2 <= 256.
//
// One workgroup handles grid row u (0 <= u <= N1/2) of one segment and its
// conjugate partner row (N1 - u) mod N1, for the 16 channel pairs of one pair
// block: 32 "lines" (row r in {0, 1} x pair p), each an m-point row.  Thread
// (p, r, q) = (tid % 16, tid / 16 % 2, tid / 32).  The m-point DFT is split
// j = M2 j1 + j2, v = k1 + M1 k2:
//   stage 1 (thread q = j2): M1-point DFT over j1 -> k1, times w_m^(j2 k1);
//   exchange through LDS ([element][32 lines], conflict free);
//   stage 2 (thread q = k1): M2-point DFT over j2 -> k2.
// The row's frequency -f partner of f = u + N1 v sits at row (N1 - u) mod N1,
// column (-v - [u > 0]) mod m, which the threads read back from LDS.
#include <hip/hip_runtime.h>

#include "fft_core.hpp"
#include "kernels.hpp"
#include "row_sizes.hpp"

namespace rubiconv {

namespace {

__device__ __forceinline__ int partner_v(int u, int v, int m) {
    return u == 0 ? (v == 0 ? 0 : m - v) : m - 1 - v;
}

// SPEC = false: convolution (forward row DFT, product with the class spectrum,
// inverse row DFT, written back in place).  SPEC = true: filter side (forward
// row DFT of the filter pair, separation into S and Df, written to the spectrum).
template <int M1, int M2, bool SPEC>
__global__ __launch_bounds__(32 * M1) void row_fast_kernel(float2* __restrict__ grid,
                                                           int64_t grid_pb_stride,
                                                           float2* __restrict__ spec,
                                                           int64_t spec_pb_stride,
                                                           const Seg* __restrict__ segs,
                                                           const int32_t* __restrict__ list,
                                                           const float2* __restrict__ tw, int n1) {
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

    const float2* twm = tw + sg->tw_off + n1;
    for (int h = tid; h < M; h += 32 * M1) roots[h] = twm[h];

    float2* row = grid + pb * grid_pb_stride + (sg->grid_off + static_cast<int64_t>(r ? ub : u) * M) *
                                                   kPairsPerBlock + p;
    float2 v[M1];
    if (act && q < M2) {
#pragma unroll
        for (int j1 = 0; j1 < M1; ++j1) v[j1] = row[(M2 * j1 + q) * kPairsPerBlock];
    }
    __syncthreads();  // roots ready
    if (act && q < M2) {
        Dft<M1, -1>::run(v);
#pragma unroll
        for (int k1 = 1; k1 < M1; ++k1) v[k1] = cmul(v[k1], roots[q * k1]);
#pragma unroll
        for (int k1 = 0; k1 < M1; ++k1) lds[(k1 * M2 + q) * 32 + line] = v[k1];
    }
    __syncthreads();
    float2 w[M2];
    if (act) {
#pragma unroll
        for (int j2 = 0; j2 < M2; ++j2) w[j2] = lds[(q * M2 + j2) * 32 + line];
        Dft<M2, -1>::run(w);  // w[k2] = Z(row r, v = q + M1 k2)
    }
    __syncthreads();
    if (act) {
#pragma unroll
        for (int k2 = 0; k2 < M2; ++k2) lds[(q + M1 * k2) * 32 + line] = w[k2];
    }
    __syncthreads();

    float2* sp = spec + pb * spec_pb_stride +
                 (static_cast<int64_t>(sg->spec_off) + static_cast<int64_t>(u) * M) *
                     (2 * kPairsPerBlock) +
                 2 * p;
    if constexpr (SPEC) {
        // H_d = (Z(f) + conj Z(-f)) / 2, H_{d+1} = (Z(f) - conj Z(-f)) / (2i);
        // S = (H_d + H_{d+1}) / (2P), Df = (H_d - H_{d+1}) / (2P); row u only.
        if (r == 0) {
            const float c = 0.5f / static_cast<float>(sg->P);
#pragma unroll
            for (int k2 = 0; k2 < M2; ++k2) {
                const int vv = q + M1 * k2;
                const float2 a = w[k2];
                const float2 b = lds[partner_v(u, vv, M) * 32 + pline];
                const float2 hd = make_float2(0.5f * (a.x + b.x), 0.5f * (a.y - b.y));
                const float2 hd1 = make_float2(0.5f * (a.y + b.y), 0.5f * (b.x - a.x));
                sp[vv * 2 * kPairsPerBlock] = cscale(cadd(hd, hd1), c);
                sp[vv * 2 * kPairsPerBlock + 1] = cscale(csub(hd, hd1), c);
            }
        }
    } else {
        // W(f) = Z(f) S(f) + conj Z(-f) Df(f) on row u; on the partner row the
        // stored entries of -f give W(-f) = Z(-f) conj S(f) + conj Z(f) conj Df(f).
        if (act) {
#pragma unroll
            for (int k2 = 0; k2 < M2; ++k2) {
                const int vv = q + M1 * k2;
                const int vb = partner_v(u, vv, M);
                const float2 b = cconj(lds[vb * 32 + pline]);
                const int vs = r == 0 ? vv : vb;
                float2 s = sp[vs * 2 * kPairsPerBlock];
                float2 df = sp[vs * 2 * kPairsPerBlock + 1];
                if (r) {
                    s = cconj(s);
                    df = cconj(df);
                }
                w[k2] = cadd(cmul(w[k2], s), cmul(b, df));
            }
        }
        __syncthreads();  // every partner read is done before LDS is reused
        if (act) {
            Dft<M2, 1>::run(w);  // over k2 -> j2, thread q = k1
#pragma unroll
            for (int j2 = 1; j2 < M2; ++j2) w[j2] = cmul(w[j2], cconj(roots[j2 * q]));
#pragma unroll
            for (int j2 = 0; j2 < M2; ++j2) lds[(j2 * M1 + q) * 32 + line] = w[j2];
        }
        __syncthreads();
        if (act && q < M2) {
#pragma unroll
            for (int k1 = 0; k1 < M1; ++k1) v[k1] = lds[(q * M1 + k1) * 32 + line];
            Dft<M1, 1>::run(v);  // over k1 -> j1, thread q = j2
#pragma unroll
            for (int j1 = 0; j1 < M1; ++j1) row[(M2 * j1 + q) * kPairsPerBlock] = v[j1];
        }
    }
}

template <int M1, int M2>
hipError_t launch_m(bool spec_mode, float2* grid, int64_t gs, float2* spec, int64_t ss,
                    const Seg* segs, const int32_t* list, int nlist, const float2* tw, int n1,
                    int npb, hipStream_t stream) {
    dim3 g(nlist * (n1 / 2 + 1), npb), b(32 * M1);
    if (spec_mode)
        hipLaunchKernelGGL((row_fast_kernel<M1, M2, true>), g, b, 0, stream, grid, gs, spec, ss,
                           segs, list, tw, n1);
    else
        hipLaunchKernelGGL((row_fast_kernel<M1, M2, false>), g, b, 0, stream, grid, gs, spec, ss,
                           segs, list, tw, n1);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_row_fast(int m, bool spec_mode, float2* grid, int64_t grid_pb_stride,
                           float2* spec, int64_t spec_pb_stride, const Seg* segs,
                           const int32_t* list, int nlist, const float2* tw, int n1, int npb,
                           hipStream_t stream) {
    if (nlist == 0) return hipSuccess;
    switch (m) {
#define RUBICONV_CASE(mm, a, b)                                                                 \
    case mm:                                                                                    \
        return launch_m<a, b>(spec_mode, grid, grid_pb_stride, spec, spec_pb_stride, segs, list, \
                              nlist, tw, n1, npb, stream);
        RUBICONV_ROW_SIZES(RUBICONV_CASE)
#undef RUBICONV_CASE
        default:
            return hipErrorInvalidValue;
    }
}

}  // namespace rubiconv
