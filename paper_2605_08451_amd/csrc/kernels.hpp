// kernels.hpp -- the three passes of the packed four-step convolution.
//
//   col_fwd : N1-point column DFTs of every document column (the left DFT of
//             Algorithm 1) and the per-document twiddle w_P^(u j);
//   row     : m-point row DFTs inside each document only (the block-diagonal
//             right DFT) of the document rows and of the same rows of the
//             filter class grid, the conjugate-symmetry separation of the
//             filter pair, the spectral product and the inverse row DFT;
//   col_inv : the conjugate twiddle and the inverse N1-point column DFT, the
//             store of positions t < L_i.
//
// Grid buffer layout (complex fp32, or complex fp16 for bf16 inputs):
// [pair block][segment grid point][16 pairs],
// grid point of (u, j) in a segment = grid_off + u * m + j.
// The filter "spectrum" is the filter pairs' class grids after the column stage,
// same layout, class grid point of (u, j) = spec_off + u * m + j.  The stored
// grids are the DFTs scaled by 1 / sqrt(N1) (folded into the w_P^r table); the
// row pass scales the filter spectra by sqrt(N1) / (2 m), so that
// 1/sqrt(N1) * 1/m * 1/sqrt(N1) = 1/P overall and fp16 values stay O(|x|).
#pragma once

#include <hip/hip_runtime.h>

#include "plan.hpp"

namespace rubiconv {

// Element type tags.
struct F32 {};
struct BF16 {};

// Power-of-two scales of the complex fp16 grids (device pointers, never null):
// pair[q] = {s, 1 / s} per channel pair q (pair block * 16 + lane pair), glob = {s, m}.
// A column pass into a grid multiplies its fp32 results by pair[q].x * glob->x before
// they are rounded to the grid type; an inverse column pass multiplies its fp32
// outputs by pair[q].y * glob->y.  The filter's per-pair normalisation and a
// call's data prescale travel this way, so every fp16 value stays in range.
struct GridScale {
    const float2* pair;
    const float2* glob;
};

struct LaunchTables {
    const Seg* segs;
    const int32_t* col_seg;
    const int32_t* task_seg;
    const float2* tw;      // per-class twiddles
    const float2* tw_n1;   // w_N1^s
    const int32_t* list;   // documents grouped by class / class identity list
};

// `half` selects complex fp16 grid and spectrum elements (complex fp32 otherwise).
hipError_t launch_col_fwd(int r, bool half, int x_dtype, const void* src, int64_t src_row_stride,
                          int D, void* grid, int64_t grid_pb_stride, const LaunchTables& t,
                          GridScale sc, int n_cols, int npb, hipStream_t stream);

hipError_t launch_col_inv(int r, bool half, int y_dtype, const void* grid, int64_t grid_pb_stride,
                          void* dst, int64_t dst_row_stride, int D, const LaunchTables& t,
                          GridScale sc, int n_cols, int npb, hipStream_t stream);

// Row pass: row DFTs of the filter class rows and the document rows, the
// separation and product, the inverse row DFT (generic kernel: long rows).
// Every row launcher takes `corr`: 0 multiplies by the filter spectrum F(f)
// (convolution), 1 by F(-f) = conj F(f) (correlation, the adjoint in x).
hipError_t launch_row_conv(int n1, bool half, void* grid, int64_t grid_pb_stride,
                           const void* fgrid, int64_t fgrid_pb_stride, const LaunchTables& t,
                           int n_tasks, int npb, int lds_bytes, int corr, hipStream_t stream);

// Register-resident row pass for a listed row size m (row_sizes.hpp) over the
// nlist documents list[0..nlist) of that size.
hipError_t launch_row_fast(int m, bool half, void* grid, int64_t grid_pb_stride, const void* fgrid,
                           int64_t fgrid_pb_stride, const Seg* segs, const int32_t* list,
                           int nlist, const float2* tw, int n1, int npb, int corr,
                           hipStream_t stream);

// Matrix-core row pass (complex fp16 grids) over `ngroups` groups, each a pair
// (first, count) of consecutive entries of `docs` (indices into segs) that share one
// size class and whose second-grid rows are those of the group's first document.
// Every document has ceil(m / 16) == nb (1 <= nb <= kMaxDenseBlocks); tabs = the
// plan's dense operand tables, addressed through Seg::dense_off.
// sum: every document of a group brings its own second-grid rows, the products of
// the group's documents are added, and the one inverse transform of the sum is written
// over the first document's rows (the others are left as they were); with sum, dscale
// (a power of two) multiplies the data rows' spectra before they are rounded to fp16,
// and out2 writes the inverse over the first document's second-grid rows instead, which
// leaves the grid itself as it was (both: 1 and false without sum).
// 16-byte entries of one class's tables for the rows of 3 to 8 blocks: nb * nb real
// operands of 64 lanes (the forward transform; the inverse takes their conjugates),
// then 16 nb complex fp16 twiddles w^(-j), 16 nb complex fp32 twiddles kappa w^j
// (w = exp(-2 pi i / m)) and kappa (fp32; the inverse's scale over the forward's),
// padded to whole 1 KB chunks.
constexpr int partner_tab_u4(int nb) { return (nb * nb * 64 + 12 * nb + 1 + 63) / 64 * 64; }

hipError_t launch_row_dense(int nb, void* grid, int64_t grid_pb_stride, const void* fgrid,
                            int64_t fgrid_pb_stride, const Seg* segs, const int32_t* docs,
                            const int32_t* groups, int ngroups, const void* tabs, int n1, int npb,
                            int corr, hipStream_t stream, bool sum = false, float dscale = 1.0f,
                            bool out2 = false);

// Long rows (fp16 grids): the first level of the row DFT of one document or class grid
// (LrItem) for its n1 grid rows and npb pair blocks, into its sub-row region, or the
// inverse from the region back (long_rows.hip).  grid_pb_stride in complex elements.
hipError_t launch_lr_step(bool inverse, void* grid, int64_t grid_pb_stride, const LrItem& it,
                          const float2* tw, int n1, int npb, hipStream_t stream);

// The same pass for rows of at most kMaxBatchM points, 16 / m documents of a group side
// by side in one matrix-core block; each document's second-grid rows are its own
// (Seg::spec_off), so the groups may also hold documents with different second grids.
// The grid and the second grid of a pair block must each span less than 2^31 bytes.
hipError_t launch_row_batch(void* grid, int64_t grid_pb_stride, const void* fgrid,
                            int64_t fgrid_pb_stride, const Seg* segs, const int32_t* docs,
                            const int32_t* groups, int ngroups, const void* tabs, int n1, int npb,
                            int corr, hipStream_t stream);

// Matrix-core column passes (N1 = 256, complex fp16 grids, D a multiple of 32).
// `mtab` holds the MFMA operand tables in lane order (16-byte entries, offsets
// below; see build_mfma_tables).
constexpr int kMtFwd1Bf16 = 0;     // forward stage 1, bf16 hi/lo: re_hi, re_lo, im_hi, im_lo
constexpr int kMtFwd1F16 = 256;    // forward stage 1, fp16: re, im
constexpr int kMtFwd2 = 384;       // forward stage 2 per k1: re, im
constexpr int kMtInv1 = 2432;      // inverse stage 1: re, im
constexpr int kMtInv2 = 2560;      // inverse stage 2 per n2: re, im
constexpr int kMtEntries = 4608;

// src_dtype 1: bf16 channels [rows][N][D] (x); 0: fp16 channel pairs [taps][D / 2] from
// launch_transpose_pairs (filter taps).
// amax_out (bf16 sources only; null for none): per column task, the largest bf16 magnitude
// bits of the x it loaded, the pass running at scale first_scale in place of sc.glob.
// amax_in (null for none; 16-byte aligned, from a launch with amax_out over the same tasks):
// this launch takes x's power-of-two range scale s = 2^(3 - e) extra (2^e at or above
// max |x|, extra a power of two), writes {s, p / s} to *used (p = prev->y, or 1 for a null
// prev) and s to *hint (host-mapped, may be null), and redoes the pass at s in place of
// sc.glob unless s equals first_scale (the scale the first launch used).
hipError_t launch_col_fwd_mfma(int src_dtype, const void* src, int64_t src_row_stride, int D,
                               void* grid, int64_t grid_pb_stride, const LaunchTables& t,
                               GridScale sc, const void* mtab, int n_cols, int npb,
                               hipStream_t stream, uint16_t* amax_out = nullptr,
                               const uint16_t* amax_in = nullptr, float2* used = nullptr,
                               float first_scale = 1.0f, float* hint = nullptr, float extra = 1.0f,
                               const float2* prev = nullptr);

hipError_t launch_col_inv_mfma(int y_dtype, const void* grid, int64_t grid_pb_stride, void* dst,
                               int64_t dst_row_stride, int D, const LaunchTables& t,
                               GridScale sc, const void* mtab, int n_cols, int npb,
                               hipStream_t stream);

// Direct-path modes (launch_direct, launch_direct_mfma)
constexpr int kDirectConv = 0;
constexpr int kDirectCorr = 1;
constexpr int kDirectXcorr = 2;

// The direct path on the matrix cores (direct_mfma.hip): the same three modes for bf16 a
// (x, or dy) and b (x, mode 2) of documents of at most kMaxDirectMfma tokens, D a multiple
// of 32, a, b and out 16-byte aligned.  taps: [D][T] bf16 pairs (launch_split_taps), T >=
// min(L, longest document); unused in mode 2.  Outputs: y or dx in bf16, the correlation
// in fp32 (as launch_direct).
hipError_t launch_direct_mfma(int mode, const void* a, const void* b, const uint32_t* taps, int T,
                              const Seg* docs, int n_docs, int N, int D, int L, void* out, hipStream_t stream);
// taps[d][t] = bf16(k[d][t]) | bf16(k[d][t] - bf16(k[d][t])) << 16, t < T (row stride ld of k)
hipError_t launch_split_taps(const float* filters, int D, int T, int ld, uint32_t* taps, hipStream_t stream);

// Documents computed by their defining sums (the direct path; kernels.hip):
// mode 0 out = y from a = x, mode 1 out = dx from a = dy, mode 2 out = the
// per-document correlation of a = dy with b = x at lags tau < min(len, L), written at
// the document's tokens (fp32).  Dtype codes: 0 fp32, 1 bf16.  taps: [T][D] fp32.
// max_len: no document in docs is longer (at most kMaxDirect).
hipError_t launch_direct(int mode, int max_len, int a_dtype, const void* a, int b_dtype,
                         const void* b, const float* taps, const Seg* docs, int n_docs, int N, int D,
                         int L, int out_dtype, void* out, hipStream_t stream);

// dk[d][tau] = sum over documents k < n_docs with tau < min(len_k, L) of
// r[row_k][start_k + tau][d] (r fp32 [B][N][D]); dk [D][L] fp32, fully written.
// segs must list the documents by non-increasing length.
hipError_t launch_lag_sum(const float* r, const Seg* segs, int n_docs, int N, int D, int L,
                          float* dk, hipStream_t stream);

// Filter taps [D][in_ld] fp32 -> [taps][D / 2] complex fp16 channel pairs (D even).
// partials (may be null): float [*ntiles][D], the sum of |k| of each channel over each
// tile of 32 taps (the input of launch_filter_scale); *ntiles <= tap_tile_rows(taps).
constexpr int tap_tile_rows(int taps) { return 2 * ((taps + 63) / 64); }
hipError_t launch_transpose_pairs(const float* in, int D, int taps, int in_ld, void* out,
                                  float* partials, int* ntiles, hipStream_t stream);

// out[c][r] = in[r][c] (r < rows, c < cols); partials as above with rows = channels and
// cols = taps (may be null), ceil(cols / 32) tiles.
hipError_t launch_transpose(const float* in, int rows, int cols, int in_ld, float* out,
                            int out_ld, float* partials, hipStream_t stream);

// Per channel pair q < npairs: g = max over its channels of the summed partials (the
// filter's absolute gain, sum over taps of |k|) and s = 2^(kFilterGainExp - e) with
// g < 2^e (1 when g is zero or not finite); pair_scale[q] = {s, 1 / s}.
constexpr int kFilterGainExp = 8;
hipError_t launch_filter_scale(const float* partials, int ntiles, int D, int npairs,
                               float2* pair_scale, hipStream_t stream);

// Exact power-of-two prescale of a [n] bf16 (dtype 1) or fp32 (dtype 0) tensor:
// a = max |v| (two passes, no atomics: a fixed result); s = 2^(kDataAmaxExp - e) with
// a < 2^e (1 when a is zero or not finite), times `extra` (a power of two);
// out = {s * extra, (prev ? prev->y : 1) / (s * extra)}.  work: kAmaxParts uint32.
constexpr int kDataAmaxExp = 3;
constexpr int kAmaxParts = 2048;

// 2^(target - e) for a = f 2^e (0.5 <= f < 1): the power of two that brings a into
// [2^(target-1), 2^target); 1 for a zero, negative, infinite or NaN a.
__device__ __forceinline__ float pow2_scale(float a, int target) {
    if (!(a > 0.0f) || !(a <= 3.0e38f)) return 1.0f;
    int e;
    (void)frexpf(a, &e);
    return ldexpf(1.0f, max(-126, min(127, target - e)));
}


hipError_t launch_prescale(int dtype, const void* in, int64_t n, float extra, const float2* prev,
                           float2* out, uint32_t* work, hipStream_t stream);

}  // namespace rubiconv
