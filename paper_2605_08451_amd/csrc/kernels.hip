// kernels.hip -- gfx950 kernels of the packed four-step convolution.
//
// Notation (Algorithm 1 and its proof): a segment of P = N1 * m points is laid
// out as an N1 x m grid in row-major order, time t = m * a + j (row a < N1,
// column j < m).  Its DFT is
//     Z[u + N1 v] = sum_j w_m^(j v) * w_P^(u j) * sum_a w_N1^(a u) X[a][j],
// i.e. N1-point column DFTs, the per-segment twiddle w_P^(u j), then m-point row
// DFTs (one block of the block-diagonal right DFT).  The inverse applies the
// same steps backwards with conjugate roots.  Two real channels 2p, 2p+1 travel
// as one complex value (Appendix, dual real FFTs).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "fft_core.hpp"
#include "kernels.hpp"

namespace rubiconv {

// ---------------------------------------------------------------- element I/O
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;  // NaN stays a (quiet) NaN
    u += 0x7fffu + ((u >> 16) & 1u);                                 // round to nearest, ties to even
    return u >> 16;
}

// Channels ch (real part) and ch + 1 (imaginary part) of one token; idx is the
// element index of channel ch.  `both` is false when ch + 1 == D (odd D).
template <class T>
__device__ __forceinline__ float2 load_pair(const void* base, int64_t idx, bool both, bool even_d);

template <>
__device__ __forceinline__ float2 load_pair<F32>(const void* base, int64_t idx, bool both, bool even_d) {
    const float* p = static_cast<const float*>(base) + idx;
    if (even_d) return *reinterpret_cast<const float2*>(p);
    return make_float2(p[0], both ? p[1] : 0.0f);
}

template <>
__device__ __forceinline__ float2 load_pair<BF16>(const void* base, int64_t idx, bool both, bool even_d) {
    const uint16_t* p = static_cast<const uint16_t*>(base) + idx;
    if (even_d) {
        uint32_t w = *reinterpret_cast<const uint32_t*>(p);
        return make_float2(bf16_to_f32(w & 0xffffu), bf16_to_f32(w >> 16));
    }
    return make_float2(bf16_to_f32(p[0]), both ? bf16_to_f32(p[1]) : 0.0f);
}

template <class T>
__device__ __forceinline__ void store_pair(void* base, int64_t idx, float2 v, bool both, bool even_d);

template <>
__device__ __forceinline__ void store_pair<F32>(void* base, int64_t idx, float2 v, bool both, bool even_d) {
    float* p = static_cast<float*>(base) + idx;
    if (even_d) {
        *reinterpret_cast<float2*>(p) = v;
        return;
    }
    p[0] = v.x;
    if (both) p[1] = v.y;
}

template <>
__device__ __forceinline__ void store_pair<BF16>(void* base, int64_t idx, float2 v, bool both, bool even_d) {
    uint16_t* p = static_cast<uint16_t*>(base) + idx;
    if (even_d) {
        *reinterpret_cast<uint32_t*>(p) = f32_to_bf16(v.x) | (f32_to_bf16(v.y) << 16);
        return;
    }
    p[0] = static_cast<uint16_t>(f32_to_bf16(v.x));
    if (both) p[1] = static_cast<uint16_t>(f32_to_bf16(v.y));
}

// w_P^r for 0 <= r < P from the class table: w_P^(N1 hi + lo) = w_m^hi * w_P^lo.
template <int N1>
__device__ __forceinline__ float2 seg_root(const float2* tw_cls, int r) {
    return cmul(tw_cls[N1 + r / N1], tw_cls[r % N1]);
}

// ---------------------------------------------------------------- column passes
// One workgroup = one grid column j of one segment x one block of 16 channel
// pairs; 16 * R threads, thread (p, q) = (tid % 16, tid / 16).  N1 = R * R is
// split as a = R n1 + n2, u = k1 + R k2:
//   stage 1 (thread q = n2): R-point DFT over n1 -> k1, times w_N1^(n2 k1);
//   exchange through LDS;
//   stage 2 (thread q = k1): R-point DFT over n2 -> k2.
// LDS holds [k1][n2][16 pairs] with a padded k1 stride so that both access
// patterns are free of bank conflicts.
template <int R, class TX>
__global__ __launch_bounds__(16 * R) void col_fwd_kernel(const void* __restrict__ src,
                                                         int64_t src_row_stride, int D,
                                                         float2* __restrict__ grid,
                                                         int64_t grid_pb_stride, LaunchTables t) {
    constexpr int N1 = R * R;
    constexpr int LD = R * 16 + 16;
    __shared__ float2 lds[R * LD];
    const int tid = threadIdx.x;
    const int p = tid & 15, q = tid >> 4;
    const int col = blockIdx.x, pb = blockIdx.y;
    const Seg* sg = t.segs + t.col_seg[col];
    const int j = col - sg->col0, m = sg->m, len = sg->len;
    const int ch = 2 * (pb * kPairsPerBlock + p);
    const bool even_d = (D & 1) == 0;
    const bool live = ch < D;

    float2 v[R];
    const int64_t base = static_cast<int64_t>(sg->row) * src_row_stride +
                         static_cast<int64_t>(sg->start) * D + ch;
#pragma unroll
    for (int n1 = 0; n1 < R; ++n1) {
        const int tt = m * (R * n1 + q) + j;
        v[n1] = (live && tt < len) ? load_pair<TX>(src, base + static_cast<int64_t>(tt) * D,
                                                   ch + 1 < D, even_d)
                                   : make_float2(0.0f, 0.0f);
    }
    Dft<R, -1>::run(v);
#pragma unroll
    for (int k1 = 1; k1 < R; ++k1) v[k1] = cmul(v[k1], t.tw_n1[q * k1]);
#pragma unroll
    for (int k1 = 0; k1 < R; ++k1) lds[k1 * LD + q * 16 + p] = v[k1];
    __syncthreads();
#pragma unroll
    for (int n2 = 0; n2 < R; ++n2) v[n2] = lds[q * LD + n2 * 16 + p];
    Dft<R, -1>::run(v);

    const float2* twc = t.tw + sg->tw_off;
    float2* out = grid + pb * grid_pb_stride + (sg->grid_off + j) * kPairsPerBlock + p;
#pragma unroll
    for (int k2 = 0; k2 < R; ++k2) {
        const int u = q + R * k2;
        out[static_cast<int64_t>(u) * m * kPairsPerBlock] = cmul(v[k2], seg_root<N1>(twc, u * j));
    }
}

template <int R, class TY>
__global__ __launch_bounds__(16 * R) void col_inv_kernel(const float2* __restrict__ grid,
                                                         int64_t grid_pb_stride,
                                                         void* __restrict__ dst,
                                                         int64_t dst_row_stride, int D,
                                                         LaunchTables t) {
    constexpr int N1 = R * R;
    constexpr int LD = R * 16 + 16;
    __shared__ float2 lds[R * LD];
    const int tid = threadIdx.x;
    const int p = tid & 15, q = tid >> 4;
    const int col = blockIdx.x, pb = blockIdx.y;
    const Seg* sg = t.segs + t.col_seg[col];
    const int j = col - sg->col0, m = sg->m, len = sg->len;
    const int ch = 2 * (pb * kPairsPerBlock + p);
    const bool even_d = (D & 1) == 0;

    const float2* twc = t.tw + sg->tw_off;
    const float2* in = grid + pb * grid_pb_stride + (sg->grid_off + j) * kPairsPerBlock + p;
    float2 v[R];
#pragma unroll
    for (int k2 = 0; k2 < R; ++k2) {
        const int u = q + R * k2;  // thread q holds k1 = q
        v[k2] = cmul(in[static_cast<int64_t>(u) * m * kPairsPerBlock],
                     cconj(seg_root<N1>(twc, u * j)));
    }
    Dft<R, 1>::run(v);  // over k2 -> n2
#pragma unroll
    for (int n2 = 1; n2 < R; ++n2) v[n2] = cmul(v[n2], cconj(t.tw_n1[q * n2]));
#pragma unroll
    for (int n2 = 0; n2 < R; ++n2) lds[q * LD + n2 * 16 + p] = v[n2];
    __syncthreads();
#pragma unroll
    for (int k1 = 0; k1 < R; ++k1) v[k1] = lds[k1 * LD + q * 16 + p];  // thread q holds n2 = q
    Dft<R, 1>::run(v);  // over k1 -> n1

    if (ch >= D) return;
    const int64_t base = static_cast<int64_t>(sg->row) * dst_row_stride +
                         static_cast<int64_t>(sg->start) * D + ch;
#pragma unroll
    for (int n1 = 0; n1 < R; ++n1) {
        const int tt = m * (R * n1 + q) + j;
        if (tt < len)
            store_pair<TY>(dst, base + static_cast<int64_t>(tt) * D, v[n1], ch + 1 < D, even_d);
    }
}

// ---------------------------------------------------------------- row pass
// Stockham autosort stage of radix R on `lines` independent m-point rows held
// in LDS as [row][j][spb pairs]; Ns = product of the radices already applied.
template <int R, int S>
__device__ __forceinline__ void stockham_butterfly(const float2* in, float2* out, int i, int mr,
                                                   int spb, int Ns, int m, const float2* twm) {
    const int k = i % Ns;
    const int step = (m / (Ns * R)) * k;
    float2 v[R];
#pragma unroll
    for (int qq = 0; qq < R; ++qq) v[qq] = in[(i + qq * mr) * spb];
#pragma unroll
    for (int qq = 1; qq < R; ++qq) {
        const float2 w = twm[qq * step];
        v[qq] = cmul(v[qq], S < 0 ? w : cconj(w));
    }
    Dft<R, S>::run(v);
    const int d = (i / Ns) * Ns * R + k;
#pragma unroll
    for (int qq = 0; qq < R; ++qq) out[(d + qq * Ns) * spb] = v[qq];
}

// m-point DFT (sign S) of nrows * spb lines; ping-pongs between a and b and
// returns the buffer holding the natural-order result.
template <int S>
__device__ float2* row_dft(float2* a, float2* b, int nrows, int m, int spb, int spb_log2,
                           const Seg* sg, const float2* twm) {
    int Ns = 1;
    const int nfac = sg->nfac;
    for (int f = 0; f < nfac; ++f) {
        const int R = sg->fac[f];
        const int mr = m / R;
        const int nbf = nrows * spb * mr;
        for (int e = threadIdx.x; e < nbf; e += blockDim.x) {
            const int pp = e & (spb - 1);
            const int rest = e >> spb_log2;
            const int i = rest % mr;
            const int row = rest / mr;
            const float2* in = a + row * m * spb + pp;
            float2* out = b + row * m * spb + pp;
            switch (R) {
                case 2: stockham_butterfly<2, S>(in, out, i, mr, spb, Ns, m, twm); break;
                case 3: stockham_butterfly<3, S>(in, out, i, mr, spb, Ns, m, twm); break;
                case 4: stockham_butterfly<4, S>(in, out, i, mr, spb, Ns, m, twm); break;
                default: stockham_butterfly<5, S>(in, out, i, mr, spb, Ns, m, twm); break;
            }
        }
        __syncthreads();
        float2* tmp = a;
        a = b;
        b = tmp;
        Ns *= R;
    }
    return a;
}

__device__ __forceinline__ int ilog2(int v) { return 31 - __clz(v); }

// One workgroup = grid row u (0 <= u <= N1/2) and its conjugate partner row
// (N1 - u) mod N1 of one segment, for spb channel pairs of one pair block.
// The frequency -f of f = u + N1 v lies at ((N1 - u) mod N1, (-v - [u > 0]) mod m).
struct RowTask {
    const Seg* sg;
    int m, spb, spb_log2, u, ub, nrows, s;
};

__device__ __forceinline__ RowTask row_task(const LaunchTables& t, int n1) {
    RowTask r;
    const int task = blockIdx.x;
    r.sg = t.segs + t.task_seg[task];
    r.m = r.sg->m;
    r.spb = r.sg->spb;
    r.spb_log2 = ilog2(r.spb);
    const int nsub = kPairsPerBlock / r.spb;
    const int rem = task - r.sg->task0;
    r.u = rem / nsub;
    r.s = rem - r.u * nsub;
    r.ub = (n1 - r.u) & (n1 - 1);
    r.nrows = (r.ub == r.u) ? 1 : 2;
    return r;
}

__device__ __forceinline__ int partner_col(int u, int v, int m) {
    return u == 0 ? (v == 0 ? 0 : m - v) : m - 1 - v;
}

__device__ __forceinline__ void load_rows(float2* lds, const float2* g, const RowTask& r) {
    const int rowlen = r.m * r.spb;
    for (int e = threadIdx.x; e < r.nrows * rowlen; e += blockDim.x) {
        const int pp = e & (r.spb - 1);
        const int jj = (e >> r.spb_log2) % r.m;
        const int uu = e < rowlen ? r.u : r.ub;
        lds[e] = g[(static_cast<int64_t>(uu) * r.m + jj) * kPairsPerBlock + pp];
    }
}

__global__ __launch_bounds__(256) void row_conv_kernel(float2* __restrict__ grid,
                                                       int64_t grid_pb_stride,
                                                       const float2* __restrict__ spec,
                                                       int64_t spec_pb_stride, LaunchTables t,
                                                       int n1) {
    extern __shared__ float2 sm[];
    const RowTask r = row_task(t, n1);
    const int pb = blockIdx.y;
    const int rowlen = r.m * r.spb;
    float2* bufa = sm;
    float2* bufb = sm + 2 * rowlen;
    float2* g = grid + pb * grid_pb_stride + r.sg->grid_off * kPairsPerBlock + r.s * r.spb;
    load_rows(bufa, g, r);
    __syncthreads();

    const float2* twm = t.tw + r.sg->tw_off + n1;
    float2* z = row_dft<-1>(bufa, bufb, r.nrows, r.m, r.spb, r.spb_log2, r.sg, twm);
    float2* w = (z == bufa) ? bufb : bufa;

    // W(f) = Z(f) S(f) + conj(Z(-f)) Df(f) and W(-f) = conj(conj(Z(-f)) S(f) + Z(f) Df(f)):
    // the spectrum of y_d + i y_{d+1} (Algorithm 3, separation and product fused).
    const float2* sp = spec + pb * spec_pb_stride +
                       (static_cast<int64_t>(r.sg->spec_off) + static_cast<int64_t>(r.u) * r.m) *
                           (2 * kPairsPerBlock) +
                       2 * r.s * r.spb;
    for (int e = threadIdx.x; e < rowlen; e += blockDim.x) {
        const int pp = e & (r.spb - 1);
        const int v = e >> r.spb_log2;
        const int vb = partner_col(r.u, v, r.m);
        const float2 a = z[e];
        const float2 b = z[((r.nrows - 1) * r.m + vb) * r.spb + pp];
        const float2 s = sp[(v * kPairsPerBlock + pp) * 2];
        const float2 df = sp[(v * kPairsPerBlock + pp) * 2 + 1];
        w[e] = cadd(cmul(a, s), cmul(cconj(b), df));
        if (r.nrows == 2) w[(r.m + vb) * r.spb + pp] = cconj(cadd(cmul(cconj(b), s), cmul(a, df)));
    }
    __syncthreads();

    float2* y = row_dft<1>(w, z, r.nrows, r.m, r.spb, r.spb_log2, r.sg, twm);
    for (int e = threadIdx.x; e < r.nrows * rowlen; e += blockDim.x) {
        const int pp = e & (r.spb - 1);
        const int jj = (e >> r.spb_log2) % r.m;
        const int uu = e < rowlen ? r.u : r.ub;
        g[(static_cast<int64_t>(uu) * r.m + jj) * kPairsPerBlock + pp] = y[e];
    }
}

// Filter side: forward row DFT of the filter pair h_d + i h_{d+1}, then
// H_d = (Z(f) + conj Z(-f)) / 2, H_{d+1} = (Z(f) - conj Z(-f)) / (2i) and the
// stored combinations S = (H_d + H_{d+1}) / (2P), Df = (H_d - H_{d+1}) / (2P).
__global__ __launch_bounds__(256) void row_spec_kernel(const float2* __restrict__ grid,
                                                       int64_t grid_pb_stride,
                                                       float2* __restrict__ spec,
                                                       int64_t spec_pb_stride, LaunchTables t,
                                                       int n1) {
    extern __shared__ float2 sm[];
    const RowTask r = row_task(t, n1);
    const int pb = blockIdx.y;
    const int rowlen = r.m * r.spb;
    float2* bufa = sm;
    float2* bufb = sm + 2 * rowlen;
    const float2* g = grid + pb * grid_pb_stride + r.sg->grid_off * kPairsPerBlock + r.s * r.spb;
    load_rows(bufa, g, r);
    __syncthreads();

    const float2* twm = t.tw + r.sg->tw_off + n1;
    const float2* z = row_dft<-1>(bufa, bufb, r.nrows, r.m, r.spb, r.spb_log2, r.sg, twm);

    const float c = 0.5f / static_cast<float>(r.sg->P);
    float2* sp = spec + pb * spec_pb_stride +
                 (static_cast<int64_t>(r.sg->spec_off) + static_cast<int64_t>(r.u) * r.m) *
                     (2 * kPairsPerBlock) +
                 2 * r.s * r.spb;
    for (int e = threadIdx.x; e < rowlen; e += blockDim.x) {
        const int pp = e & (r.spb - 1);
        const int v = e >> r.spb_log2;
        const int vb = partner_col(r.u, v, r.m);
        const float2 a = z[e];
        const float2 b = z[((r.nrows - 1) * r.m + vb) * r.spb + pp];
        const float2 hd = make_float2(0.5f * (a.x + b.x), 0.5f * (a.y - b.y));
        const float2 hd1 = make_float2(0.5f * (a.y + b.y), 0.5f * (b.x - a.x));
        sp[(v * kPairsPerBlock + pp) * 2] = cscale(cadd(hd, hd1), c);
        sp[(v * kPairsPerBlock + pp) * 2 + 1] = cscale(csub(hd, hd1), c);
    }
}

// ---------------------------------------------------------------- transpose
// out[c][r] = in[r][c] for r < rows, c < cols (32 x 32 tiles through LDS).
__global__ __launch_bounds__(256) void transpose_kernel(const float* __restrict__ in, int rows,
                                                        int cols, int in_ld,
                                                        float* __restrict__ out, int out_ld) {
    __shared__ float tile[32][33];
    const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int k = ty; k < 32; k += 8) {
        const int rr = r0 + k, cc = c0 + tx;
        if (rr < rows && cc < cols) tile[k][tx] = in[static_cast<int64_t>(rr) * in_ld + cc];
    }
    __syncthreads();
    for (int k = ty; k < 32; k += 8) {
        const int cc = c0 + k, rr = r0 + tx;
        if (rr < rows && cc < cols) out[static_cast<int64_t>(cc) * out_ld + rr] = tile[tx][k];
    }
}

// ---------------------------------------------------------------- launchers
template <int R>
static hipError_t col_fwd_r(int x_dtype, const void* src, int64_t rs, int D, float2* grid,
                            int64_t gs, const LaunchTables& t, int n_cols, int npb,
                            hipStream_t stream) {
    dim3 g(n_cols, npb), b(16 * R);
    if (x_dtype == 0)
        hipLaunchKernelGGL((col_fwd_kernel<R, F32>), g, b, 0, stream, src, rs, D, grid, gs, t);
    else
        hipLaunchKernelGGL((col_fwd_kernel<R, BF16>), g, b, 0, stream, src, rs, D, grid, gs, t);
    return hipGetLastError();
}

hipError_t launch_col_fwd(int r, int x_dtype, const void* src, int64_t src_row_stride, int D,
                          float2* grid, int64_t grid_pb_stride, const LaunchTables& t,
                          int n_cols, int npb, hipStream_t stream) {
    if (n_cols == 0) return hipSuccess;
    if (r == 16)
        return col_fwd_r<16>(x_dtype, src, src_row_stride, D, grid, grid_pb_stride, t, n_cols, npb,
                             stream);
    return col_fwd_r<8>(x_dtype, src, src_row_stride, D, grid, grid_pb_stride, t, n_cols, npb,
                        stream);
}

template <int R>
static hipError_t col_inv_r(int y_dtype, const float2* grid, int64_t gs, void* dst, int64_t rs,
                            int D, const LaunchTables& t, int n_cols, int npb,
                            hipStream_t stream) {
    dim3 g(n_cols, npb), b(16 * R);
    if (y_dtype == 0)
        hipLaunchKernelGGL((col_inv_kernel<R, F32>), g, b, 0, stream, grid, gs, dst, rs, D, t);
    else
        hipLaunchKernelGGL((col_inv_kernel<R, BF16>), g, b, 0, stream, grid, gs, dst, rs, D, t);
    return hipGetLastError();
}

hipError_t launch_col_inv(int r, int y_dtype, const float2* grid, int64_t grid_pb_stride,
                          void* dst, int64_t dst_row_stride, int D, const LaunchTables& t,
                          int n_cols, int npb, hipStream_t stream) {
    if (n_cols == 0) return hipSuccess;
    if (r == 16)
        return col_inv_r<16>(y_dtype, grid, grid_pb_stride, dst, dst_row_stride, D, t, n_cols, npb,
                             stream);
    return col_inv_r<8>(y_dtype, grid, grid_pb_stride, dst, dst_row_stride, D, t, n_cols, npb,
                        stream);
}

hipError_t launch_row_conv(int n1, float2* grid, int64_t grid_pb_stride, const float2* spec,
                           int64_t spec_pb_stride, const LaunchTables& t, int n_tasks, int npb,
                           int lds_bytes, hipStream_t stream) {
    if (n_tasks == 0) return hipSuccess;
    hipLaunchKernelGGL(row_conv_kernel, dim3(n_tasks, npb), dim3(256), lds_bytes, stream, grid,
                       grid_pb_stride, spec, spec_pb_stride, t, n1);
    return hipGetLastError();
}

hipError_t launch_row_spec(int n1, const float2* grid, int64_t grid_pb_stride, float2* spec,
                           int64_t spec_pb_stride, const LaunchTables& t, int n_tasks, int npb,
                           int lds_bytes, hipStream_t stream) {
    if (n_tasks == 0) return hipSuccess;
    hipLaunchKernelGGL(row_spec_kernel, dim3(n_tasks, npb), dim3(256), lds_bytes, stream, grid,
                       grid_pb_stride, spec, spec_pb_stride, t, n1);
    return hipGetLastError();
}

hipError_t launch_transpose(const float* in, int rows, int cols, int in_ld, float* out,
                            int out_ld, hipStream_t stream) {
    if (rows == 0 || cols == 0) return hipSuccess;
    dim3 g((cols + 31) / 32, (rows + 31) / 32);
    hipLaunchKernelGGL(transpose_kernel, g, dim3(256), 0, stream, in, rows, cols, in_ld, out,
                       out_ld);
    return hipGetLastError();
}

}  // namespace rubiconv
