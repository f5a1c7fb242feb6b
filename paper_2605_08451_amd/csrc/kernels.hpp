// kernels.hpp -- the three passes of the packed four-step convolution.
//
//   col_fwd : N1-point column DFTs of every document column (the left DFT of
//             Algorithm 1) and the per-document twiddle w_P^(u j);
//   row     : m-point row DFTs inside each document only (the block-diagonal
//             right DFT), then either the spectral product with conjugate-
//             symmetry separation and the inverse row DFT (convolution), or
//             the separation into the two filters' spectra (filter side);
//   col_inv : the conjugate twiddle and the inverse N1-point column DFT, the
//             store of positions t < L_i.
//
// Grid buffer layout (complex fp32): [pair block][segment grid point][16 pairs],
// grid point of (u, j) in a segment = grid_off + u * m + j.
// Spectrum layout: [pair block][class spectrum point][16 pairs][2], spectrum
// point of (u, v), u <= N1/2, = spec_off + u * m + v; entry 0 is S = (H_d +
// H_{d+1}) / (2P), entry 1 is Df = (H_d - H_{d+1}) / (2P).
#pragma once

#include <hip/hip_runtime.h>

#include "plan.hpp"

namespace rubiconv {

// Element type tags.
struct F32 {};
struct BF16 {};

struct LaunchTables {
    const Seg* segs;
    const int32_t* col_seg;
    const int32_t* task_seg;
    const float2* tw;      // per-class twiddles
    const float2* tw_n1;   // w_N1^s
    const int32_t* list;   // documents grouped by class / class identity list
};

hipError_t launch_col_fwd(int r, int x_dtype, const void* src, int64_t src_row_stride, int D,
                          float2* grid, int64_t grid_pb_stride, const LaunchTables& t,
                          int n_cols, int npb, hipStream_t stream);

hipError_t launch_col_inv(int r, int y_dtype, const float2* grid, int64_t grid_pb_stride,
                          void* dst, int64_t dst_row_stride, int D, const LaunchTables& t,
                          int n_cols, int npb, hipStream_t stream);

hipError_t launch_row_conv(int n1, float2* grid, int64_t grid_pb_stride, const float2* spec,
                           int64_t spec_pb_stride, const LaunchTables& t, int n_tasks, int npb,
                           int lds_bytes, hipStream_t stream);

hipError_t launch_row_spec(int n1, const float2* grid, int64_t grid_pb_stride, float2* spec,
                           int64_t spec_pb_stride, const LaunchTables& t, int n_tasks, int npb,
                           int lds_bytes, hipStream_t stream);

// Register-resident row pass for a listed row size m (row_sizes.hpp) over the
// nlist segments list[0..nlist) of that size; spec_mode selects the filter side.
hipError_t launch_row_fast(int m, bool spec_mode, float2* grid, int64_t grid_pb_stride,
                           float2* spec, int64_t spec_pb_stride, const Seg* segs,
                           const int32_t* list, int nlist, const float2* tw, int n1, int npb,
                           hipStream_t stream);

hipError_t launch_transpose(const float* in, int rows, int cols, int in_ld, float* out,
                            int out_ld, hipStream_t stream);

}  // namespace rubiconv
