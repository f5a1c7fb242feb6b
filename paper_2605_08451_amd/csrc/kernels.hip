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

#include <hip/hip_bf16.h>
#include <hip/hip_fp16.h>

#include <cstdint>
#include <type_traits>

#include "fft_core.hpp"
#include "kernels.hpp"
#include "pk_half.hpp"

namespace rubiconv {

// ---------------------------------------------------------------- element I/O
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// Two floats rounded to bf16 (nearest, ties to even; one v_cvt_pk_bf16_f32 on gfx950),
// low half = v.x.
__device__ __forceinline__ uint32_t pack_bf16x2(float2 v) { return bf2_bits(v.x, v.y); }

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
    const uint32_t w = pack_bf16x2(v);
    if (even_d) {
        *reinterpret_cast<uint32_t*>(p) = w;
        return;
    }
    p[0] = static_cast<uint16_t>(w & 0xffffu);
    if (both) p[1] = static_cast<uint16_t>(w >> 16);
}

// Grid and spectrum elements: complex fp32 (float2) or complex fp16 (__half2),
// always computed in fp32.
__device__ __forceinline__ float2 gload(const float2* p) { return *p; }
__device__ __forceinline__ float2 gload(const __half2* p) { return __half22float2(*p); }
__device__ __forceinline__ void gstore(float2* p, float2 v) { *p = v; }
__device__ __forceinline__ void gstore(__half2* p, float2 v) { *p = __float22half2_rn(v); }

// Buffer resource over one document's tokens: accesses at byte offsets outside
// [0, bytes) read as zero and are dropped on store, which implements the zero
// padding beyond the document (and its cut-off) without branches.
constexpr int kBufferWord3 = 0x00020000;  // gfx9 raw buffer: 32-bit data format

__device__ __forceinline__ __amdgpu_buffer_rsrc_t doc_buffer(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes),
                                             kBufferWord3);
}

// Column-pass modes: channel count D a multiple of 32 (every lane live), D even,
// or D odd (the last pair has a single channel).
enum ColMode { kFull = 0, kEven = 1, kOdd = 2 };

template <class T, int MODE>
__device__ __forceinline__ float2 col_load(__amdgpu_buffer_rsrc_t rs, const void* doc, uint32_t off,
                                           int64_t idx, bool live, bool in_doc, bool both) {
    if constexpr (MODE == kOdd) {
        if (!(live && in_doc)) return make_float2(0.0f, 0.0f);
        return load_pair<T>(doc, idx, both, false);
    } else {
        float2 v;
        if constexpr (sizeof(T) == sizeof(F32) && std::is_same<T, F32>::value) {
            const auto w = __builtin_amdgcn_raw_buffer_load_b64(rs, static_cast<int>(off), 0, 0);
            v = make_float2(__uint_as_float(w[0]), __uint_as_float(w[1]));
        } else {
            const uint32_t w = __builtin_amdgcn_raw_buffer_load_b32(rs, static_cast<int>(off), 0, 0);
            v = make_float2(bf16_to_f32(w & 0xffffu), bf16_to_f32(w >> 16));
        }
        if constexpr (MODE == kEven) {
            if (!live) v = make_float2(0.0f, 0.0f);
        }
        return v;
    }
}

template <class T, int MODE>
__device__ __forceinline__ void col_store(__amdgpu_buffer_rsrc_t rs, void* doc, uint32_t off,
                                          int64_t idx, float2 v, bool in_doc, bool both) {
    if constexpr (MODE == kOdd) {
        if (in_doc) store_pair<T>(doc, idx, v, both, false);
    } else if constexpr (std::is_same<T, F32>::value) {
        __builtin_amdgcn_raw_buffer_store_b64(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(rs, 0, 0, 0)), v), rs,
            static_cast<int>(off), 0, 0);
    } else {
        __builtin_amdgcn_raw_buffer_store_b32(pack_bf16x2(v), rs, static_cast<int>(off), 0, 0);
    }
}

template <class T>
constexpr int elem_bytes() { return std::is_same<T, F32>::value ? 4 : 2; }

// ---------------------------------------------------------------- column passes
// One workgroup = one grid column j of one segment x one block of 16 channel
// pairs (1-D grid, pair block fastest, so that neighbouring workgroups touch the
// two halves of each 128-byte line of x and y together); 16 * R threads,
// thread (p, q) = (tid % 16, tid / 16).  N1 = R * R is split as a = R n1 + n2,
// u = k1 + R k2:
//   stage 1 (thread q = n2): R-point DFT over n1 -> k1, times w_N1^(n2 k1);
//   exchange through LDS;
//   stage 2 (thread q = k1): R-point DFT over n2 -> k2.
// LDS holds [k1][n2][16 pairs] with a padded k1 stride so that both access
// patterns are free of bank conflicts.  The per-document twiddle w_P^(u j)
// (scaled by 1/sqrt(N1)) comes from the class's full root table.
template <int R, class TX, class G, int MODE>
__global__ __launch_bounds__(16 * R) void col_fwd_kernel(const void* __restrict__ src,
                                                         int64_t src_row_stride, int D,
                                                         G* __restrict__ grid,
                                                         int64_t grid_pb_stride, LaunchTables t,
                                                         GridScale sc, int npb) {
    constexpr int LD = R * 16 + 16;
    constexpr int ES = elem_bytes<TX>();
    __shared__ float2 lds[R * LD];
    const int tid = threadIdx.x;
    const int p = tid & 15, q = tid >> 4;
    const int col = blockIdx.x / npb, pb = blockIdx.x - col * npb;
    const Seg* sg = t.segs + t.col_seg[col];
    const int j = col - sg->col0, m = sg->m, len = sg->len;
    const int ch = 2 * (pb * kPairsPerBlock + p);
    const bool live = MODE == kFull || ch < D;

    const char* doc = static_cast<const char*>(src) +
                      (static_cast<int64_t>(sg->row) * src_row_stride +
                       static_cast<int64_t>(sg->start) * D) * ES;
    const __amdgpu_buffer_rsrc_t rs = doc_buffer(doc, static_cast<uint32_t>(len) * D * ES);
    float2 v[R];
#pragma unroll
    for (int n1 = 0; n1 < R; ++n1) {
        const int tt = m * (R * n1 + q) + j;
        v[n1] = col_load<TX, MODE>(rs, doc, (static_cast<uint32_t>(tt) * D + ch) * ES,
                                   static_cast<int64_t>(tt) * D + ch, live, tt < len, ch + 1 < D);
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

    const float2* twf = t.tw + sg->twf_off;
    G* out = grid + pb * grid_pb_stride + (sg->grid_off + j) * kPairsPerBlock + p;
    const float mul = sc.pair[pb * kPairsPerBlock + p].x * sc.glob->x;
#pragma unroll
    for (int k2 = 0; k2 < R; ++k2) {
        const int u = q + R * k2;
        gstore(out + static_cast<int64_t>(u) * m * kPairsPerBlock, cscale(cmul(v[k2], twf[u * j]), mul));
    }
}

template <int R, class TY, class G, int MODE>
__global__ __launch_bounds__(16 * R) void col_inv_kernel(const G* __restrict__ grid,
                                                         int64_t grid_pb_stride,
                                                         void* __restrict__ dst,
                                                         int64_t dst_row_stride, int D,
                                                         LaunchTables t, GridScale sc, int npb) {
    constexpr int LD = R * 16 + 16;
    constexpr int ES = elem_bytes<TY>();
    __shared__ float2 lds[R * LD];
    const int tid = threadIdx.x;
    const int p = tid & 15, q = tid >> 4;
    const int col = blockIdx.x / npb, pb = blockIdx.x - col * npb;
    const Seg* sg = t.segs + t.col_seg[col];
    const int j = col - sg->col0, m = sg->m, len = sg->len;
    const int ch = 2 * (pb * kPairsPerBlock + p);

    const float2* twf = t.tw + sg->twf_off;
    const G* in = grid + pb * grid_pb_stride + (sg->grid_off + j) * kPairsPerBlock + p;
    float2 v[R];
#pragma unroll
    for (int k2 = 0; k2 < R; ++k2) {
        const int u = q + R * k2;  // thread q holds k1 = q
        v[k2] = cmul(gload(in + static_cast<int64_t>(u) * m * kPairsPerBlock), cconj(twf[u * j]));
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
    const float mul = sc.pair[pb * kPairsPerBlock + p].y * sc.glob->y;
#pragma unroll
    for (int n1 = 0; n1 < R; ++n1) v[n1] = cscale(v[n1], mul);

    if (MODE != kFull && ch >= D) return;
    char* doc = static_cast<char*>(dst) + (static_cast<int64_t>(sg->row) * dst_row_stride +
                                           static_cast<int64_t>(sg->start) * D) * ES;
    const __amdgpu_buffer_rsrc_t rs = doc_buffer(doc, static_cast<uint32_t>(len) * D * ES);
#pragma unroll
    for (int n1 = 0; n1 < R; ++n1) {
        const int tt = m * (R * n1 + q) + j;
        col_store<TY, MODE>(rs, doc, (static_cast<uint32_t>(tt) * D + ch) * ES,
                            static_cast<int64_t>(tt) * D + ch, v[n1], tt < len, ch + 1 < D);
    }
}

// ---------------------------------------------------------------- row pass
// Stockham autosort stage of radix R on `lines` independent m-point rows held
// in LDS as [row][j][spb pairs]; Ns = product of the radices already applied.
// Quotient and remainder of x / d for 0 <= x < 2^24 and a divisor shared by the
// workgroup, through a float reciprocal and one correction step (the hardware has
// no integer division, and its emulation costs tens of instructions).
struct FastDiv {
    int d;
    float inv;
    __device__ explicit FastDiv(int dv) : d(dv), inv(1.0f / static_cast<float>(dv)) {}
    __device__ __forceinline__ int div(int x, int* rem) const {
        int q = static_cast<int>(static_cast<float>(x) * inv);
        int r = x - q * d;
        if (r < 0) { --q; r += d; }
        if (r >= d) { ++q; r -= d; }
        *rem = r;
        return q;
    }
};

template <int R, int S, class E>
__device__ __forceinline__ void stockham_butterfly(const E* in, E* out, int i, int mr,
                                                   int spb, int Ns, const FastDiv& fns, int mstep,
                                                   const float2* twm) {
    int k;
    const int iq = fns.div(i, &k);  // i / Ns, i % Ns
    const int step = mstep * k;
    float2 v[R];
#pragma unroll
    for (int qq = 0; qq < R; ++qq) v[qq] = gload(in + (i + qq * mr) * spb);
#pragma unroll
    for (int qq = 1; qq < R; ++qq) {
        const float2 w = twm[qq * step];
        v[qq] = cmul(v[qq], S < 0 ? w : cconj(w));
    }
    Dft<R, S>::run(v);
    const int d = iq * Ns * R + k;
#pragma unroll
    for (int qq = 0; qq < R; ++qq) gstore(out + (d + qq * Ns) * spb, v[qq]);
}

// m-point DFT (sign S) of nrows * spb lines of LDS elements E (complex fp32, or
// complex fp16 for fp16 grids: every stage computes in fp32 and rounds its outputs);
// ping-pongs between a and b and returns the buffer holding the natural-order result.
template <int S, class E>
__device__ E* row_dft(E* a, E* b, int nrows, int m, int spb, int spb_log2,
                      const Seg* sg, const float2* twm) {
    int Ns = 1;
    const int nfac = sg->nfac;
    for (int f = 0; f < nfac; ++f) {
        const int R = sg->fac[f];
        const int mr = m / R;
        const int nbf = nrows * spb * mr;
        const FastDiv fmr(mr), fns(Ns);
        const int mstep = m / (Ns * R);
        for (int e = threadIdx.x; e < nbf; e += blockDim.x) {
            const int pp = e & (spb - 1);
            const int rest = e >> spb_log2;
            int i;
            const int row = fmr.div(rest, &i);  // rest / mr, rest % mr
            const E* in = a + row * m * spb + pp;
            E* out = b + row * m * spb + pp;
            switch (R) {
                case 2: stockham_butterfly<2, S>(in, out, i, mr, spb, Ns, fns, mstep, twm); break;
                case 3: stockham_butterfly<3, S>(in, out, i, mr, spb, Ns, fns, mstep, twm); break;
                case 4: stockham_butterfly<4, S>(in, out, i, mr, spb, Ns, fns, mstep, twm); break;
                default: stockham_butterfly<5, S>(in, out, i, mr, spb, Ns, fns, mstep, twm); break;
            }
        }
        __syncthreads();
        E* tmp = a;
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

// Workgroups go to the eight XCDs in turn (workgroup b to XCD b % 8).  Task
// numbers are dealt so that each XCD takes runs of kXcdRun consecutive tasks, i.e.
// the sub-blocks of channel pairs of a grid row together: their 4- to 16-byte
// pieces of each 64-byte grid point then meet in one XCD's L2 instead of being
// fetched by several.  The launch covers a multiple of 8 kXcdRun workgroups;
// numbers past the last task return at once.
constexpr int kXcdRun = 16;
__device__ __forceinline__ int xcd_task(int b) {
    const int xcd = b & 7, k = b >> 3;
    return (k % kXcdRun) + kXcdRun * (xcd + 8 * (k / kXcdRun));
}

__device__ __forceinline__ RowTask row_task(const LaunchTables& t, int n1, int task) {
    RowTask r;
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

// LDS holds the grid's own element type: rows are copied as they are
template <class G>
__device__ __forceinline__ void load_rows(G* lds, const G* g, const RowTask& r) {
    const int rowlen = r.m * r.spb;
    const FastDiv fm(r.m);
    for (int e = threadIdx.x; e < r.nrows * rowlen; e += blockDim.x) {
        const int pp = e & (r.spb - 1);
        int jj;
        (void)fm.div(e >> r.spb_log2, &jj);
        const int uu = e < rowlen ? r.u : r.ub;
        lds[e] = g[(static_cast<int64_t>(uu) * r.m + jj) * kPairsPerBlock + pp];
    }
}

// Generic row pass (long rows): the filter class rows go through the row DFT
// first; their conjugate-symmetry separation leaves S and Df for every row-u
// frequency in the third LDS buffer ([0][v] = S, [1][v] = Df).  Then the
// document rows go through the same DFT, the product, the inverse row DFT and
// back to the grid.  LDS: three buffers of two rows of m * spb values of the
// grid's element type.
template <class G>
__global__ __launch_bounds__(256) void row_conv_kernel(G* __restrict__ grid,
                                                       int64_t grid_pb_stride,
                                                       const G* __restrict__ fgrid,
                                                       int64_t fgrid_pb_stride, LaunchTables t,
                                                       int n1, int n_tasks, int corr) {
    extern __shared__ __align__(16) unsigned char row_smem[];
    G* const sm = reinterpret_cast<G*>(row_smem);
    const int task = xcd_task(static_cast<int>(blockIdx.x));
    if (task >= n_tasks) return;  // whole workgroup
    const RowTask r = row_task(t, n1, task);
    const int pb = blockIdx.y;
    const int rowlen = r.m * r.spb;
    G* b0 = sm;
    G* b1 = sm + 2 * rowlen;
    G* sdf = sm + 4 * rowlen;
    const float2* twm = t.tw + r.sg->tw_off;

    const G* fg = fgrid + pb * fgrid_pb_stride + static_cast<int64_t>(r.sg->spec_off) * kPairsPerBlock +
                  r.s * r.spb;
    load_rows(b0, fg, r);
    __syncthreads();
    const G* zh = row_dft<-1>(b0, b1, r.nrows, r.m, r.spb, r.spb_log2, r.sg, twm);
    const float c = 0.5f * sqrtf(static_cast<float>(n1)) / static_cast<float>(r.m);
    for (int e = threadIdx.x; e < rowlen; e += blockDim.x) {
        const int pp = e & (r.spb - 1);
        const int v = e >> r.spb_log2;
        const int vb = partner_col(r.u, v, r.m);
        float2 s, df;
        // correlation: the filter spectrum read at -f (its conjugate for real taps)
        const float2 fa = gload(zh + e), fb = gload(zh + ((r.nrows - 1) * r.m + vb) * r.spb + pp);
        filter_sdf(corr ? fb : fa, corr ? fa : fb, c, s, df);
        gstore(sdf + e, s);
        gstore(sdf + rowlen + e, df);
    }
    __syncthreads();

    G* g = grid + pb * grid_pb_stride + r.sg->grid_off * kPairsPerBlock + r.s * r.spb;
    load_rows(b0, g, r);
    __syncthreads();
    G* z = row_dft<-1>(b0, b1, r.nrows, r.m, r.spb, r.spb_log2, r.sg, twm);
    G* w = (z == b0) ? b1 : b0;
    for (int e = threadIdx.x; e < rowlen; e += blockDim.x) {
        const int pp = e & (r.spb - 1);
        const int v = e >> r.spb_log2;
        const int vb = partner_col(r.u, v, r.m);
        const float2 a = gload(z + e);
        const int eb = ((r.nrows - 1) * r.m + vb) * r.spb + pp;
        const float2 b = gload(z + eb);
        const float2 s = gload(sdf + e), df = gload(sdf + rowlen + e);
        gstore(w + e, product_f(a, b, s, df));
        if (r.nrows == 2) gstore(w + eb, product_neg_f(a, b, s, df));
    }
    __syncthreads();

    const G* y = row_dft<1>(w, z, r.nrows, r.m, r.spb, r.spb_log2, r.sg, twm);
    const FastDiv fm(r.m);
    for (int e = threadIdx.x; e < r.nrows * rowlen; e += blockDim.x) {
        const int pp = e & (r.spb - 1);
        int jj;
        (void)fm.div(e >> r.spb_log2, &jj);
        const int uu = e < rowlen ? r.u : r.ub;
        g[(static_cast<int64_t>(uu) * r.m + jj) * kPairsPerBlock + pp] = y[e];
    }
}

// ---------------------------------------------------------------- transpose
// out[c][r] = in[r][c] for r < rows, c < cols (32 x 32 tiles through LDS).
// Sum of |tile[row][0 .. 31]| for the rows of a tile in LDS, in a fixed order (the same
// result on every call): eight threads per row, four values each, then a butterfly over
// the eight.  Thread `tid` of 256 covers row tid / 8; the result is in every thread of
// the row's group.
template <int LDW>
__device__ __forceinline__ float tile_row_abs_sum32(const float (*tile)[LDW], int row_base, int tid) {
    const int r = row_base + (tid >> 3), part = tid & 7;
    float a = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) a += fabsf(tile[r][4 * part + i]);
    a += __shfl_xor(a, 1);
    a += __shfl_xor(a, 2);
    a += __shfl_xor(a, 4);
    return a;
}

__global__ __launch_bounds__(256) void transpose_kernel(const float* __restrict__ in, int rows,
                                                        int cols, int in_ld,
                                                        float* __restrict__ out, int out_ld,
                                                        float* __restrict__ partials) {
    __shared__ float tile[32][33];
    const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int k = ty; k < 32; k += 8) {
        const int rr = r0 + k, cc = c0 + tx;
        tile[k][tx] = (rr < rows && cc < cols) ? in[static_cast<int64_t>(rr) * in_ld + cc] : 0.0f;
    }
    __syncthreads();
    if (partials != nullptr) {  // per row (channel): sum of |k| over this tile's 32 columns (taps)
        const float a = tile_row_abs_sum32<33>(tile, 0, threadIdx.x);
        const int rr = r0 + (threadIdx.x >> 3);
        if ((threadIdx.x & 7) == 0 && rr < rows) partials[static_cast<int64_t>(blockIdx.x) * rows + rr] = a;
    }
    for (int k = ty; k < 32; k += 8) {
        const int cc = c0 + k, rr = r0 + tx;
        if (rr < rows && cc < cols) out[static_cast<int64_t>(cc) * out_ld + rr] = tile[tx][k];
    }
}

// Filter taps [D][in_ld] fp32 -> [taps][D / 2] complex fp16 channel pairs (2q, 2q + 1),
// the input of the matrix-core column pass (which computes in fp16).  Tiles of 64
// channels x 32 taps through LDS: coalesced reads along taps, writes along pairs.
__global__ __launch_bounds__(256) void transpose_pairs_kernel(const float* __restrict__ in, int D,
                                                              int taps, int in_ld,
                                                              uint32_t* __restrict__ out,
                                                              float* __restrict__ partials) {
    __shared__ float tile[64][33];
    const int t0 = blockIdx.x * 32, c0 = blockIdx.y * 64;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int k = ty; k < 64; k += 8) {
        const int c = c0 + k, t = t0 + tx;
        tile[k][tx] = (c < D && t < taps) ? in[static_cast<int64_t>(c) * in_ld + t] : 0.0f;
    }
    __syncthreads();
    if (partials != nullptr) {  // per channel: sum of |k| over this tile's 32 taps
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const float a = tile_row_abs_sum32<33>(tile, 32 * h, threadIdx.x);
            const int c = c0 + 32 * h + (threadIdx.x >> 3);
            if ((threadIdx.x & 7) == 0 && c < D) partials[static_cast<int64_t>(blockIdx.x) * D + c] = a;
        }
    }
    const int half_d = D / 2;
    for (int k = ty; k < 32; k += 8) {
        const int t = t0 + k, q = c0 / 2 + tx;
        if (t < taps && q < half_d) {
            const __half2 v = __float22half2_rn(make_float2(tile[2 * tx][k], tile[2 * tx + 1][k]));
            out[static_cast<int64_t>(t) * half_d + q] = __builtin_bit_cast(uint32_t, v);
        }
    }
}

// Short documents (at most kMaxDirect tokens) by their defining sums, one workgroup
// per document and 64 channels, lanes along channels (coalesced rows of x), four
// output positions in flight.  taps: the first T filter taps transposed, [T][D]
// fp32 (T >= every lag a direct document uses).  Modes:
//   kDirectConv:  out[t]   = sum_{tau <= min(t, L-1)} k[tau] a[t - tau]   (y from x)
//   kDirectCorr:  out[s]   = sum_{tau <= min(len-1-s, L-1)} k[tau] a[s + tau]   (dx from dy)
//   kDirectXcorr: out[tau] = sum_{t = tau}^{len-1} a[t] b[t - tau], tau < min(len, L)
//                 (the filter gradient's per-document correlation of dy with x, fp32)
// All sums run in fp32 in ascending lag (or token) order.

template <class T>
__device__ __forceinline__ float load_elem(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p, int64_t i) {
    return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}
__device__ __forceinline__ void store_elem(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store_elem(uint16_t* p, int64_t i, float v) {
    p[i] = static_cast<uint16_t>(bf16_rne_bits(v));
}

template <int MODE, int MAXLEN, class TA, class TB, class TO>
__global__ __launch_bounds__(256) void direct_kernel(const TA* __restrict__ a, const TB* __restrict__ b,
                                                     const float* __restrict__ taps,
                                                     const Seg* __restrict__ docs, int N, int D,
                                                     int L, TO* __restrict__ out) {
    // the document's 64 channels of a, and of the taps (conv, corr) or b (xcorr), in LDS
    __shared__ float sa[MAXLEN][65];
    __shared__ float sb[MAXLEN][65];
    const Seg sg = docs[blockIdx.x];
    const int len = sg.len;
    const int c = threadIdx.x & 63, tq = threadIdx.x >> 6;
    const int d = blockIdx.y * 64 + c;
    const bool live = d < D;
    const int64_t base = (static_cast<int64_t>(sg.row) * N + sg.start) * D + d;
    const int nb = MODE == kDirectXcorr ? len : (len < L ? len : L);  // rows of sb in use
    for (int t = tq; t < len; t += 4) sa[t][c] = live ? load_elem(a, base + static_cast<int64_t>(t) * D) : 0.0f;
    for (int t = tq; t < nb; t += 4) {
        if constexpr (MODE == kDirectXcorr)
            sb[t][c] = live ? load_elem(b, base + static_cast<int64_t>(t) * D) : 0.0f;
        else
            sb[t][c] = live ? taps[static_cast<int64_t>(t) * D + d] : 0.0f;
    }
    __syncthreads();  // the only barrier: every thread reaches it
    if (!live) return;
    // four consecutive outputs per thread share each operand load: a window of four
    // values of the sliding operand moves by one element per step of the sum.  Values
    // outside [0, len) and taps at or past L read as zero, which keeps every sum exact.
    auto at = [&](float (*m)[65], int i, int lim) { return (i >= 0 && i < lim) ? m[i][c] : 0.0f; };
    for (int t0 = 4 * tq; t0 < len; t0 += 16) {
        float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if constexpr (MODE == kDirectConv) {
            // out[t0 + i] = sum_tau k[tau] a[t0 + i - tau], tau <= t0 + i, tau < L
            const int kl = len < L ? len : L;
            float w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) w[i] = at(sa, t0 + i, len);  // a[t0 + i - tau], tau = 0
            const int last = t0 + 3 < kl - 1 ? t0 + 3 : kl - 1;
            for (int tau = 0; tau <= last; ++tau) {
                const float kv = sb[tau][c];
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[i] += kv * w[i];
                w[3] = w[2]; w[2] = w[1]; w[1] = w[0];
                w[0] = at(sa, t0 - tau - 1, len);
            }
        } else if constexpr (MODE == kDirectCorr) {
            // out[t0 + i] = sum_tau k[tau] a[t0 + i + tau], t0 + i + tau < len, tau < L
            const int kl = len < L ? len : L;
            float w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) w[i] = at(sa, t0 + i, len);
            const int last = len - 1 - t0 < kl - 1 ? len - 1 - t0 : kl - 1;
            for (int tau = 0; tau <= last; ++tau) {
                const float kv = sb[tau][c];
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[i] += kv * w[i];
                w[0] = w[1]; w[1] = w[2]; w[2] = w[3];
                w[3] = at(sa, t0 + tau + 4, len);
            }
        } else {
            // out[t0 + i] = sum_{s >= t0 + i} a[s] b[s - t0 - i], lags t0 + i < min(len, L)
            float w[4];  // b[s - t0 - i] for the current s
#pragma unroll
            for (int i = 0; i < 4; ++i) w[i] = at(sb, -i, len);  // s = t0
            for (int s = t0; s < len; ++s) {
                const float av = sa[s][c];
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[i] += av * w[i];
                w[3] = w[2]; w[2] = w[1]; w[1] = w[0];
                w[0] = at(sb, s + 1 - t0, len);
            }
        }
        const int lim = MODE == kDirectXcorr ? (len < L ? len : L) : len;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (t0 + i < lim) store_elem(out, base + static_cast<int64_t>(t0 + i) * D, acc[i]);
    }
}

// Filter gradient, last step: every document's cross-correlation r_i[tau] of dy
// with x (lags 0 <= tau < min(len_i, L), written by the inverse passes at the
// document's token positions s_i + tau of a [B][N][D] fp32 buffer; the direct path
// writes its documents' correlations there too) summed over the documents into
// dk[D][L].  A workgroup owns 8 lags x 64 VEC channels; its four waves split the
// documents (rounds of four documents, round k to wave k mod 4) and their partial
// sums are added in wave order through LDS, so the order of every sum is fixed.
// segs lists the documents longest first: a wave stops at the first round whose
// longest document ends before the workgroup's lags.  Lanes run along channels for
// the reads (VEC channels per lane) and along lags for the writes.
template <int VEC>
__global__ __launch_bounds__(256) void lag_sum_kernel(const float* __restrict__ r,
                                                      const Seg* __restrict__ segs, int n_docs,
                                                      int N, int D, int L, float* __restrict__ dk) {
    typedef float fv __attribute__((ext_vector_type(VEC)));
    constexpr int C = 64 * VEC;                 // channels per workgroup
    constexpr int T = 8;                        // lags per workgroup
    constexpr int U = 4;                        // documents per round of loads
    __shared__ float part[4][T][C + 1];
    // workgroup b runs on XCD b mod 8: the four lag tiles of one 128-byte row segment
    // of dk go to workgroups 8 apart on one XCD, whose L2 joins their 32-byte writes
    const int b = blockIdx.x;
    const int tile = 4 * (8 * (b >> 5) + (b & 7)) + ((b >> 3) & 3);
    const int tau0 = tile * T, d0 = blockIdx.y * C;
    if (tau0 >= L) return;  // grid padding; no barrier has been reached
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int d = d0 + VEC * lane;
    fv acc[T];
#pragma unroll
    for (int i = 0; i < T; ++i) acc[i] = fv(0.0f);
    if (d < D) {
        for (int k = U * w; k < n_docs; k += 4 * U) {
            if ((segs[k].len < L ? segs[k].len : L) <= tau0) break;
            fv v[U][T];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                int lags = 0;
                const float* base = r;
                if (k + u < n_docs) {
                    const Seg& sg = segs[k + u];
                    lags = sg.len < L ? sg.len : L;
                    base = r + (static_cast<int64_t>(sg.row) * N + sg.start) * D + d;
                }
#pragma unroll
                for (int i = 0; i < T; ++i)
                    v[u][i] = tau0 + i < lags
                                  ? *reinterpret_cast<const fv*>(base + static_cast<int64_t>(tau0 + i) * D)
                                  : fv(0.0f);
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int i = 0; i < T; ++i) acc[i] += v[u][i];
        }
    }
#pragma unroll
    for (int i = 0; i < T; ++i)
#pragma unroll
        for (int e = 0; e < VEC; ++e) part[w][i][VEC * lane + e] = acc[i][e];
    __syncthreads();
    // write: 8 lanes along lags, 32 channels per instruction; waves added in order
    const int tl = threadIdx.x & (T - 1), jq = threadIdx.x >> 3;
    for (int j = jq; j < C; j += 256 / T) {
        const int dd = d0 + j, tau = tau0 + tl;
        if (dd < D && tau < L)
            dk[static_cast<int64_t>(dd) * L + tau] =
                ((part[0][tl][j] + part[1][tl][j]) + part[2][tl][j]) + part[3][tl][j];
    }
}

// The same sum for plans with few documents (fewer than one round per wave above, so
// most of those waves would idle): each wave owns 8 lags of the workgroup's 32 and sums
// every document itself, longest first, in document order; the workgroup's 32 x 256
// block of dk goes out through LDS with lanes along lags (128-byte runs per channel).
__global__ __launch_bounds__(256) void lag_sum_few_kernel(const float* __restrict__ r,
                                                         const Seg* __restrict__ segs, int n_docs,
                                                         int N, int D, int L, float* __restrict__ dk) {
    constexpr int C = 256;  // channels per workgroup, four per lane
    constexpr int T = 8;    // lags per wave
    constexpr int U = 4;    // documents per round of loads
    __shared__ float part[4 * T][C + 1];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int tau0 = blockIdx.x * (4 * T) + w * T, d0 = blockIdx.y * C;
    const int d = d0 + 4 * lane;
    float4 acc[T];
#pragma unroll
    for (int i = 0; i < T; ++i) acc[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (d < D && tau0 < L) {
        for (int k = 0; k < n_docs; k += U) {
            if ((segs[k].len < L ? segs[k].len : L) <= tau0) break;
            float4 v[U][T];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                int lags = 0;
                const float* base = r;
                if (k + u < n_docs) {
                    const Seg& sg = segs[k + u];
                    lags = sg.len < L ? sg.len : L;
                    base = r + (static_cast<int64_t>(sg.row) * N + sg.start) * D + d;
                }
#pragma unroll
                for (int i = 0; i < T; ++i)
                    v[u][i] = tau0 + i < lags
                                  ? *reinterpret_cast<const float4*>(base + static_cast<int64_t>(tau0 + i) * D)
                                  : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int i = 0; i < T; ++i) {
                    acc[i].x += v[u][i].x; acc[i].y += v[u][i].y;
                    acc[i].z += v[u][i].z; acc[i].w += v[u][i].w;
                }
        }
    }
#pragma unroll
    for (int i = 0; i < T; ++i) {
        float* row = &part[w * T + i][4 * lane];
        row[0] = acc[i].x; row[1] = acc[i].y; row[2] = acc[i].z; row[3] = acc[i].w;
    }
    __syncthreads();
    // write: 32 lanes along lags, 8 channels per instruction
    const int tl = threadIdx.x & 31, jq = threadIdx.x >> 5;
    const int tau = blockIdx.x * (4 * T) + tl;
    for (int j = jq; j < C; j += 8) {
        const int dd = d0 + j;
        if (dd < D && tau < L) dk[static_cast<int64_t>(dd) * L + tau] = part[tl][j];
    }
}

// The same transpose for tap rows whose stride is a multiple of 4 floats (taps <= stride):
// tiles of TC channels x 64 taps, 16-byte loads along taps (256-byte runs per channel)
// and 16-byte stores of four pairs along channels (2 TC-byte runs per tap).
template <int TC>
__global__ __launch_bounds__(256) void transpose_pairs4_kernel(const float* __restrict__ in, int D,
                                                               int taps, int in_ld,
                                                               uint32_t* __restrict__ out,
                                                               float* __restrict__ partials) {
    __shared__ float tile[TC][65];
    const int t0 = blockIdx.x * 64, c0 = blockIdx.y * TC;
    const int tid = threadIdx.x;
    {
        const int tx = tid & 15, cy = tid >> 4;  // 4 taps per thread, 16 channel rows per pass
        const int t = t0 + 4 * tx;
#pragma unroll
        for (int k = 0; k < TC / 16; ++k) {
            const int c = c0 + cy + 16 * k;
            float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            if (c < D && t < taps) {  // t + 3 < in_ld: in_ld is a multiple of 4, taps <= in_ld
                v = *reinterpret_cast<const float4*>(in + static_cast<int64_t>(c) * in_ld + t);
            }
            float* row = &tile[cy + 16 * k][4 * tx];
            row[0] = v.x; row[1] = v.y; row[2] = v.z; row[3] = v.w;
        }
    }
    __syncthreads();
    if (partials != nullptr) {  // per channel: sum of |k| over each 32-tap half of the tile
#pragma unroll
        for (int rb = 0; rb < TC; rb += 32)
#pragma unroll
            for (int th = 0; th < 2; ++th) {
                const int r = rb + (threadIdx.x >> 3), part = threadIdx.x & 7;
                float a = 0.0f;
#pragma unroll
                for (int i = 0; i < 4; ++i) a += fabsf(tile[r][32 * th + 4 * part + i]);
                a += __shfl_xor(a, 1);
                a += __shfl_xor(a, 2);
                a += __shfl_xor(a, 4);
                const int c = c0 + r;
                if (part == 0 && c < D) partials[static_cast<int64_t>(2 * blockIdx.x + th) * D + c] = a;
            }
    }
    const int half_d = D / 2;
    constexpr int QT = TC / 8;         // threads per tap row, 4 pairs each
    constexpr int RP = 256 / QT;       // tap rows per pass
    const int qx = tid % QT, ty = tid / QT;
#pragma unroll
    for (int k = 0; k < 64 / RP; ++k) {
        const int tt = ty + RP * k, t = t0 + tt;
        const int q0 = c0 / 2 + 4 * qx;
        if (t < taps && q0 < half_d) {
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int cl = 8 * qx + 2 * e;
                w[e] = __builtin_bit_cast(uint32_t, __float22half2_rn(make_float2(tile[cl][tt], tile[cl + 1][tt])));
            }
            uint32_t* dst = out + static_cast<int64_t>(t) * half_d + q0;
            if (q0 + 4 <= half_d) {
                *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
            } else {
                for (int e = 0; e < 4 && q0 + e < half_d; ++e) dst[e] = w[e];
            }
        }
    }
}

// ---------------------------------------------------------------- launchers
static int col_mode(int D) { return D % 32 == 0 ? kFull : (D % 2 == 0 ? kEven : kOdd); }

template <int R, class G, int MODE>
static hipError_t col_fwd_rgm(int x_dtype, const void* src, int64_t rs, int D, void* grid,
                              int64_t gs, const LaunchTables& t, GridScale sc, int n_cols, int npb,
                              hipStream_t stream) {
    const dim3 g(static_cast<unsigned>(n_cols) * npb), b(16 * R);
    G* gp = static_cast<G*>(grid);
    if (x_dtype == 0)
        hipLaunchKernelGGL((col_fwd_kernel<R, F32, G, MODE>), g, b, 0, stream, src, rs, D, gp, gs,
                           t, sc, npb);
    else
        hipLaunchKernelGGL((col_fwd_kernel<R, BF16, G, MODE>), g, b, 0, stream, src, rs, D, gp, gs,
                           t, sc, npb);
    return hipGetLastError();
}

template <int R, class G>
static hipError_t col_fwd_rg(int x_dtype, const void* src, int64_t rs, int D, void* grid,
                             int64_t gs, const LaunchTables& t, GridScale sc, int n_cols, int npb,
                             hipStream_t stream) {
    switch (col_mode(D)) {
        case kFull: return col_fwd_rgm<R, G, kFull>(x_dtype, src, rs, D, grid, gs, t, sc, n_cols, npb, stream);
        case kEven: return col_fwd_rgm<R, G, kEven>(x_dtype, src, rs, D, grid, gs, t, sc, n_cols, npb, stream);
        default: return col_fwd_rgm<R, G, kOdd>(x_dtype, src, rs, D, grid, gs, t, sc, n_cols, npb, stream);
    }
}

hipError_t launch_col_fwd(int r, bool half, int x_dtype, const void* src, int64_t src_row_stride,
                          int D, void* grid, int64_t grid_pb_stride, const LaunchTables& t,
                          GridScale sc, int n_cols, int npb, hipStream_t stream) {
    if (n_cols == 0) return hipSuccess;
    if (r == 16)
        return half ? col_fwd_rg<16, __half2>(x_dtype, src, src_row_stride, D, grid, grid_pb_stride,
                                              t, sc, n_cols, npb, stream)
                    : col_fwd_rg<16, float2>(x_dtype, src, src_row_stride, D, grid, grid_pb_stride,
                                             t, sc, n_cols, npb, stream);
    return half ? col_fwd_rg<8, __half2>(x_dtype, src, src_row_stride, D, grid, grid_pb_stride, t,
                                         sc, n_cols, npb, stream)
                : col_fwd_rg<8, float2>(x_dtype, src, src_row_stride, D, grid, grid_pb_stride, t,
                                        sc, n_cols, npb, stream);
}

template <int R, class G, int MODE>
static hipError_t col_inv_rgm(int y_dtype, const void* grid, int64_t gs, void* dst, int64_t rs,
                              int D, const LaunchTables& t, GridScale sc, int n_cols, int npb,
                              hipStream_t stream) {
    const dim3 g(static_cast<unsigned>(n_cols) * npb), b(16 * R);
    const G* gp = static_cast<const G*>(grid);
    if (y_dtype == 0)
        hipLaunchKernelGGL((col_inv_kernel<R, F32, G, MODE>), g, b, 0, stream, gp, gs, dst, rs, D,
                           t, sc, npb);
    else
        hipLaunchKernelGGL((col_inv_kernel<R, BF16, G, MODE>), g, b, 0, stream, gp, gs, dst, rs, D,
                           t, sc, npb);
    return hipGetLastError();
}

template <int R, class G>
static hipError_t col_inv_rg(int y_dtype, const void* grid, int64_t gs, void* dst, int64_t rs,
                             int D, const LaunchTables& t, GridScale sc, int n_cols, int npb,
                             hipStream_t stream) {
    switch (col_mode(D)) {
        case kFull: return col_inv_rgm<R, G, kFull>(y_dtype, grid, gs, dst, rs, D, t, sc, n_cols, npb, stream);
        case kEven: return col_inv_rgm<R, G, kEven>(y_dtype, grid, gs, dst, rs, D, t, sc, n_cols, npb, stream);
        default: return col_inv_rgm<R, G, kOdd>(y_dtype, grid, gs, dst, rs, D, t, sc, n_cols, npb, stream);
    }
}

hipError_t launch_col_inv(int r, bool half, int y_dtype, const void* grid, int64_t grid_pb_stride,
                          void* dst, int64_t dst_row_stride, int D, const LaunchTables& t,
                          GridScale sc, int n_cols, int npb, hipStream_t stream) {
    if (n_cols == 0) return hipSuccess;
    if (r == 16)
        return half ? col_inv_rg<16, __half2>(y_dtype, grid, grid_pb_stride, dst, dst_row_stride, D,
                                              t, sc, n_cols, npb, stream)
                    : col_inv_rg<16, float2>(y_dtype, grid, grid_pb_stride, dst, dst_row_stride, D,
                                             t, sc, n_cols, npb, stream);
    return half ? col_inv_rg<8, __half2>(y_dtype, grid, grid_pb_stride, dst, dst_row_stride, D, t,
                                         sc, n_cols, npb, stream)
                : col_inv_rg<8, float2>(y_dtype, grid, grid_pb_stride, dst, dst_row_stride, D, t,
                                        sc, n_cols, npb, stream);
}

hipError_t launch_row_conv(int n1, bool half, void* grid, int64_t grid_pb_stride,
                           const void* fgrid, int64_t fgrid_pb_stride, const LaunchTables& t,
                           int n_tasks, int npb, int lds_bytes, int corr, hipStream_t stream) {
    if (n_tasks == 0) return hipSuccess;
    const int run = 8 * kXcdRun;
    const dim3 g((n_tasks + run - 1) / run * run, npb), b(256);
    hipError_t e;
    if (half) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&row_conv_kernel<__half2>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(row_conv_kernel<__half2>, g, b, lds_bytes, stream,
                           static_cast<__half2*>(grid), grid_pb_stride,
                           static_cast<const __half2*>(fgrid), fgrid_pb_stride, t, n1, n_tasks, corr);
    } else {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&row_conv_kernel<float2>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(row_conv_kernel<float2>, g, b, lds_bytes, stream,
                           static_cast<float2*>(grid), grid_pb_stride,
                           static_cast<const float2*>(fgrid), fgrid_pb_stride, t, n1, n_tasks, corr);
    }
    return hipGetLastError();
}

template <int MAXLEN>
hipError_t launch_direct_len(int mode, int a_dtype, const void* a, int b_dtype, const void* b,
                             const float* taps, const Seg* docs, int n_docs, int N, int D, int L,
                             int out_dtype, void* out, hipStream_t stream) {
    const dim3 g(n_docs, (D + 63) / 64), blk(256);
    using U = uint16_t;
    if (mode == kDirectXcorr) {  // out fp32; a = dy, b = x
        if (a_dtype == 1 && b_dtype == 1)
            hipLaunchKernelGGL((direct_kernel<kDirectXcorr, MAXLEN, U, U, float>), g, blk, 0, stream,
                               static_cast<const U*>(a), static_cast<const U*>(b), taps, docs, N, D, L,
                               static_cast<float*>(out));
        else if (a_dtype == 1)
            hipLaunchKernelGGL((direct_kernel<kDirectXcorr, MAXLEN, U, float, float>), g, blk, 0, stream,
                               static_cast<const U*>(a), static_cast<const float*>(b), taps, docs, N,
                               D, L, static_cast<float*>(out));
        else if (b_dtype == 1)
            hipLaunchKernelGGL((direct_kernel<kDirectXcorr, MAXLEN, float, U, float>), g, blk, 0, stream,
                               static_cast<const float*>(a), static_cast<const U*>(b), taps, docs, N,
                               D, L, static_cast<float*>(out));
        else
            hipLaunchKernelGGL((direct_kernel<kDirectXcorr, MAXLEN, float, float, float>), g, blk, 0,
                               stream, static_cast<const float*>(a), static_cast<const float*>(b), taps,
                               docs, N, D, L, static_cast<float*>(out));
        return hipGetLastError();
    }
#define RUBICONV_DIRECT(M, TA, TO)                                                              \
    hipLaunchKernelGGL((direct_kernel<M, MAXLEN, TA, float, TO>), g, blk, 0, stream,           \
                       static_cast<const TA*>(a), static_cast<const float*>(nullptr), taps, docs, \
                       N, D, L, static_cast<TO*>(out))
    if (mode == kDirectConv) {
        if (a_dtype == 1) {
            if (out_dtype == 1) RUBICONV_DIRECT(kDirectConv, U, U); else RUBICONV_DIRECT(kDirectConv, U, float);
        } else {
            if (out_dtype == 1) RUBICONV_DIRECT(kDirectConv, float, U); else RUBICONV_DIRECT(kDirectConv, float, float);
        }
    } else {
        if (a_dtype == 1) {
            if (out_dtype == 1) RUBICONV_DIRECT(kDirectCorr, U, U); else RUBICONV_DIRECT(kDirectCorr, U, float);
        } else {
            if (out_dtype == 1) RUBICONV_DIRECT(kDirectCorr, float, U); else RUBICONV_DIRECT(kDirectCorr, float, float);
        }
    }
#undef RUBICONV_DIRECT
    return hipGetLastError();
}

hipError_t launch_direct(int mode, int max_len, int a_dtype, const void* a, int b_dtype,
                         const void* b, const float* taps, const Seg* docs, int n_docs, int N, int D,
                         int L, int out_dtype, void* out, hipStream_t stream) {
    if (n_docs == 0) return hipSuccess;
    if (max_len > kMaxDirect) return hipErrorInvalidValue;
    // LDS sized for the longest document the plan sends here
    return max_len <= 64 ? launch_direct_len<64>(mode, a_dtype, a, b_dtype, b, taps, docs, n_docs, N,
                                                 D, L, out_dtype, out, stream)
                         : launch_direct_len<kMaxDirect>(mode, a_dtype, a, b_dtype, b, taps, docs,
                                                         n_docs, N, D, L, out_dtype, out, stream);
}

hipError_t launch_lag_sum(const float* r, const Seg* segs, int n_docs, int N, int D, int L,
                          float* dk, hipStream_t stream) {
    if (D <= 0 || L <= 0) return hipSuccess;
    if (D % 4 == 0 && n_docs < 16) {  // fewer documents than the waves' rounds below
        const dim3 g((L + 31) / 32, (D + 255) / 256), b(256);
        hipLaunchKernelGGL(lag_sum_few_kernel, g, b, 0, stream, r, segs, n_docs, N, D, L, dk);
        return hipGetLastError();
    }
    if (D % 4 == 0) {  // whole float4 groups: 16-byte loads (r is 256-byte aligned)
        const dim3 g((L + 255) / 256 * 32, (D + 255) / 256), b(256);
        hipLaunchKernelGGL(lag_sum_kernel<4>, g, b, 0, stream, r, segs, n_docs, N, D, L, dk);
    } else {
        const dim3 g((L + 255) / 256 * 32, (D + 63) / 64), b(256);
        hipLaunchKernelGGL(lag_sum_kernel<1>, g, b, 0, stream, r, segs, n_docs, N, D, L, dk);
    }
    return hipGetLastError();
}

hipError_t launch_transpose_pairs(const float* in, int D, int taps, int in_ld, void* out,
                                  float* partials, int* ntiles, hipStream_t stream) {
    *ntiles = 0;
    if (D <= 0 || taps <= 0) return hipSuccess;
    // 16-byte paths: whole float4 groups of taps (aligned rows) and of pairs (D / 2).  Its
    // 64-tap tiles write the partial sums of two 32-tap tiles (a last one without taps as
    // zero): 2 ceil(taps / 64) tiles there, ceil(taps / 32) otherwise.
    if (taps <= in_ld && in_ld % 4 == 0 && (D / 2) % 4 == 0 &&
        reinterpret_cast<uintptr_t>(in) % 16 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0) {
        const dim3 g((taps + 63) / 64, (D + 63) / 64);
        *ntiles = 2 * static_cast<int>(g.x);
        hipLaunchKernelGGL(transpose_pairs4_kernel<64>, g, dim3(256), 0, stream, in, D, taps, in_ld,
                           static_cast<uint32_t*>(out), partials);
        return hipGetLastError();
    }
    const dim3 g((taps + 31) / 32, (D + 63) / 64);
    *ntiles = static_cast<int>(g.x);
    hipLaunchKernelGGL(transpose_pairs_kernel, g, dim3(256), 0, stream, in, D, taps, in_ld,
                       static_cast<uint32_t*>(out), partials);
    return hipGetLastError();
}

hipError_t launch_transpose(const float* in, int rows, int cols, int in_ld, float* out,
                            int out_ld, float* partials, hipStream_t stream) {
    if (rows == 0 || cols == 0) return hipSuccess;  // partials: ceil(cols / 32) tiles
    dim3 g((cols + 31) / 32, (rows + 31) / 32);
    hipLaunchKernelGGL(transpose_kernel, g, dim3(256), 0, stream, in, rows, cols, in_ld, out,
                       out_ld, partials);
    return hipGetLastError();
}

// ---------------------------------------------------------------- range scales (pow2_scale: kernels.hpp)

// One workgroup per 2 channel pairs (4 channels): thread t sums the tiles t / 4,
// t / 4 + 64, ... of channel t % 4 (four independent sums in flight), then the 64 partial
// sums of each channel are added in a fixed order (within each wave by shuffles, then the
// four waves).
__global__ __launch_bounds__(256) void filter_scale_kernel(const float* __restrict__ partials,
                                                           int ntiles, int D, int npairs,
                                                           float2* __restrict__ pair_scale) {
    __shared__ float part[4][4];
    const int c = threadIdx.x & 3, r = threadIdx.x >> 2;
    const int d = blockIdx.x * 4 + c;
    // sixteen loads in flight per lane while at least 16 rounds of tiles remain (long
    // filters have thousands of tiles per channel), then four, then one
    float acc[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) acc[u] = 0.0f;
    if (d < D) {
        int t = r;
        for (; t + 15 * 64 < ntiles; t += 16 * 64) {
#pragma unroll
            for (int u = 0; u < 16; ++u) acc[u] += partials[static_cast<int64_t>(t + 64 * u) * D + d];
        }
        for (; t + 3 * 64 < ntiles; t += 4 * 64) {
#pragma unroll
            for (int u = 0; u < 4; ++u) acc[u] += partials[static_cast<int64_t>(t + 64 * u) * D + d];
        }
        for (; t < ntiles; t += 64) acc[0] += partials[static_cast<int64_t>(t) * D + d];
    }
#pragma unroll
    for (int w = 8; w > 0; w >>= 1)
#pragma unroll
        for (int u = 0; u < w; ++u) acc[u] += acc[u + w];
    // the 16 partial sums of each channel in a wave (lanes c, c + 4, ...), then the four waves
    float a = acc[0];
#pragma unroll
    for (int o = 4; o < 64; o <<= 1) a += __shfl_xor(a, o);
    if ((threadIdx.x & 63) < 4) part[threadIdx.x >> 6][c] = a;
    __syncthreads();
    if (threadIdx.x < 2) {
        const int q = blockIdx.x * 2 + threadIdx.x;
        float g = 0.0f;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int cc = 2 * threadIdx.x + k;
            g = fmaxf(g, (part[0][cc] + part[1][cc]) + (part[2][cc] + part[3][cc]));
        }
        if (q < npairs) {
            const float sc = pow2_scale(g, kFilterGainExp);
            pair_scale[q] = make_float2(sc, 1.0f / sc);
        }
    }
}

// |v| as the bits of a non-negative float, for bf16 pairs (DT 1) or fp32 words
template <int DT>
__device__ __forceinline__ uint32_t abs_bits_max(uint32_t w, uint32_t m) {
    if constexpr (DT == 1) {
        m = max(m, w & 0x7fff0000u);
        return max(m, (w << 16) & 0x7fff0000u);
    } else {
        return max(m, w & 0x7fffffffu);
    }
}

// Stage 1: workgroup g reduces a grid-strided share of the words; one partial per group.
// Each thread keeps kAmaxUnroll 16-byte loads in flight per round.
constexpr int kAmaxUnroll = 8;
template <int DT>
__global__ __launch_bounds__(256) void amax_partial_kernel(const uint32_t* __restrict__ in, int64_t nwords,
                                                           uint32_t* __restrict__ parts) {
    __shared__ uint32_t red[4];
    uint32_t m0 = 0, m1 = 0;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * 256 * 4;  // words per round-robin step
    int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
    if ((reinterpret_cast<uintptr_t>(in) & 15) == 0) {
        for (; i + (kAmaxUnroll - 1) * stride + 3 < nwords; i += kAmaxUnroll * stride) {
            typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
            u32x4 w[kAmaxUnroll];
#pragma unroll
            for (int u = 0; u < kAmaxUnroll; ++u)
                w[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(in + i + u * stride));
#pragma unroll
            for (int u = 0; u < kAmaxUnroll; ++u) {
                m0 = abs_bits_max<DT>(w[u].x, m0);
                m1 = abs_bits_max<DT>(w[u].y, m1);
                m0 = abs_bits_max<DT>(w[u].z, m0);
                m1 = abs_bits_max<DT>(w[u].w, m1);
            }
        }
        for (; i + 3 < nwords; i += stride) {
            const uint4 w = *reinterpret_cast<const uint4*>(in + i);
            m0 = abs_bits_max<DT>(w.x, m0);
            m1 = abs_bits_max<DT>(w.y, m1);
            m0 = abs_bits_max<DT>(w.z, m0);
            m1 = abs_bits_max<DT>(w.w, m1);
        }
        for (; i < nwords; ++i) m0 = abs_bits_max<DT>(in[i], m0);  // the last partial group
    } else {
        for (; i < nwords; i += stride)
            for (int k = 0; k < 4 && i + k < nwords; ++k) m0 = abs_bits_max<DT>(in[i + k], m0);
    }
    uint32_t m = max(m0, m1);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), o)));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) parts[blockIdx.x] = max(max(red[0], red[1]), max(red[2], red[3]));
}

// Stage 2: one workgroup combines the partials (and a last odd bf16 element) into the scale.
__global__ __launch_bounds__(256) void amax_finish_kernel(const uint32_t* __restrict__ parts, int nparts,
                                                          const uint16_t* __restrict__ head,
                                                          const uint16_t* __restrict__ tail, float extra,
                                                          const float2* __restrict__ prev,
                                                          float2* __restrict__ out) {
    __shared__ uint32_t red[4];
    uint32_t m = 0;
    for (int i = threadIdx.x; i < nparts; i += 256) m = max(m, parts[i]);
    if (threadIdx.x == 0 && head != nullptr) m = max(m, (static_cast<uint32_t>(*head) << 16) & 0x7fff0000u);
    if (threadIdx.x == 0 && tail != nullptr) m = max(m, (static_cast<uint32_t>(*tail) << 16) & 0x7fff0000u);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), o)));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        const float a = __uint_as_float(max(max(red[0], red[1]), max(red[2], red[3])));
        const float s = pow2_scale(a, kDataAmaxExp) * extra;
        out[0] = make_float2(s, (prev != nullptr ? prev->y : 1.0f) / s);
    }
}

hipError_t launch_filter_scale(const float* partials, int ntiles, int D, int npairs,
                               float2* pair_scale, hipStream_t stream) {
    if (npairs <= 0) return hipSuccess;
    hipLaunchKernelGGL(filter_scale_kernel, dim3((npairs + 1) / 2), dim3(256), 0, stream,
                       partials, ntiles, D, npairs, pair_scale);
    return hipGetLastError();
}

hipError_t launch_prescale(int dtype, const void* in, int64_t n, float extra, const float2* prev,
                           float2* out, uint32_t* work, hipStream_t stream) {
    // whole aligned 32-bit words; a bf16 element before the first word (a tensor that starts
    // at an odd element) or after the last one goes to stage 2 on its own
    const uint16_t* head = nullptr;
    const uint16_t* tail = nullptr;
    const uint32_t* words = static_cast<const uint32_t*>(in);
    int64_t nwords = n;
    if (dtype == 1) {
        const uint16_t* e = static_cast<const uint16_t*>(in);
        int64_t ne = n;
        if (n > 0 && (reinterpret_cast<uintptr_t>(e) & 3) != 0) {
            head = e;
            ++e;
            --ne;
        }
        if (ne & 1) tail = e + (ne - 1);
        words = reinterpret_cast<const uint32_t*>(e);
        nwords = ne / 2;
    }
    const int64_t groups = (nwords + 1023) / 1024;
    const int nparts = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(kAmaxParts, groups)));
    if (dtype == 1)
        hipLaunchKernelGGL(amax_partial_kernel<1>, dim3(nparts), dim3(256), 0, stream, words, nwords, work);
    else
        hipLaunchKernelGGL(amax_partial_kernel<0>, dim3(nparts), dim3(256), 0, stream, words, nwords, work);
    hipLaunchKernelGGL(amax_finish_kernel, dim3(1), dim3(256), 0, stream, work, nparts, head, tail, extra,
                       prev, out);
    return hipGetLastError();
}

}  // namespace rubiconv
