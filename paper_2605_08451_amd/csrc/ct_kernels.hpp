// ct_kernels.hpp -- launchers of the masked Cooley-Tukey convolution (ct_kernels.hip).
//
// Data layout (ct_plan.hpp): documents packed longest first in a flat array of
// points; channel pairs (d, d + 1) are one complex lane, kPairs lanes per block.
// The long-document grid is [pair block][point][kPairs] complex (fp16 or fp32).
// The spectrum is [size class][pair block][f <= P/2][kPairs] of (U, V), complex fp16
// for bf16 inputs and complex fp32 otherwise, with U = (H_d + H_{d+1}) / 2 and
// V = (H_d - H_{d+1}) / 2, so that the product of a pair's transform Z, scaled for the
// inverse, is W(f) = (Z(f) U(f) + conj(Z(-f)) V(f)) / P.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ct_plan.hpp"

namespace rubiconv::ct {

// Short documents (P <= kTile), one tile of whole documents per workgroup.
// mode 0: forward transform of x, product with the spectrum, inverse, into y.
// mode 1: forward transform of the filter taps (a: fp32 [taps][D]) into the spectrum.
// spec_half: spectrum entries in complex fp16 (8 bytes) instead of complex fp32 (16).
hipError_t launch_short(int mode, const Doc* docs, const int32_t* tile_docs, int n_tiles,
                        int64_t region_off, int a_dtype, const void* a, int N, int D, int npb,
                        bool spec_half, void* spec, int out_dtype, void* out, const float2* tw,
                        hipStream_t stream);

// Long documents: first kLogTile forward stages of every tile, from x (or the taps)
// into the grid.
hipError_t launch_front(const Doc* docs, const int32_t* tile_doc, int n_tiles, int a_dtype,
                        const void* a, int N, int D, int npb, bool half, void* grid,
                        int64_t long_points, const float2* tw, hipStream_t stream);

// Long documents: the remaining stages down every column of a tile-strided view.
// mode 0: forward stages, product, inverse stages, in place.  mode 1: forward stages,
// then the spectrum entries.
hipError_t launch_col(int mode, const Doc* docs, const int32_t* items, int n_items, bool half,
                      void* grid, int64_t long_points, int npb, bool spec_half, void* spec,
                      const float2* tw, hipStream_t stream);

// Long documents of more than 2^kMaxLogCols points per 512-point column: the middle
// stages (forward, or the inverse's, in place) on every middle-pass tile.
hipError_t launch_mid(bool inverse, const Doc* docs, const int32_t* tiles, int n_tiles, bool half,
                      void* grid, int64_t long_points, int npb, const float2* tw, hipStream_t stream);

// Long documents: the last kLogTile inverse stages of every tile, into y.
hipError_t launch_back(const Doc* docs, const int32_t* tile_doc, int n_tiles, bool half,
                       const void* grid, int64_t long_points, int npb, int out_dtype, void* out,
                       int N, int D, const float2* tw, hipStream_t stream);

}  // namespace rubiconv::ct
