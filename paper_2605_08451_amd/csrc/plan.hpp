// plan.hpp -- the plan's tables, as seen by the host builder and the kernels.
//
// A "segment" is one independent transform on the N1 x m grid: either a
// document of the packed input (Algorithm 1: one block of the block-diagonal
// second DFT per document) or one filter size class (the filter padded to that
// class's transform size).  Segments of the same kind are laid out back to back
// in a grid buffer; the kernels find their segment from a per-column or
// per-row-task table.
#pragma once

#include <cstdint>

namespace rubiconv {

constexpr int kPairsPerBlock = 16;  // channel pairs per block: 16 * 8 B = 128 B of complex fp32
constexpr int kMaxFactors = 14;     // radices of m (m <= 2048 has at most 11)
constexpr int kMaxM = 2048;         // largest row DFT
constexpr int kRowLdsBytes = 98304; // generic row kernel: three buffers of two rows each
constexpr int kMaxDenseBlocks = 8;  // matrix-core row pass: m <= 16 * kMaxDenseBlocks

// Longest document the direct path may take (its per-output sums stay short).
constexpr int kMaxDirect = 128;
// Longest document the direct path takes on the matrix cores (bf16 inputs, D a multiple of
// 32): its sums run as blocked Toeplitz products, one LDS row of this many tokens per
// channel; it is also that path's default limit (measured: rows of 1024 tokens leave one
// workgroup per CU and made the LM-packing workload 6% slower than the transforms, rows of
// 512 three workgroups and 7% faster)
constexpr int kMaxDirectMfma = 512;
// Default: documents of at most this many tokens take the direct path, when together
// they would hold at least 1/kDirectMinShare of the transform grid (measured: a few
// short documents among long ones cost more on their own launch than they save).
constexpr int kDefaultDirect = 64;
constexpr int kDirectMinShare = 16;
// Size-class merging: bytes moved per grid point and channel pair, in units of one
// grid element.  A document's point costs five (column pass write, row pass read,
// write and filter-class read, inverse column pass read); a filter class's point
// costs one and a half (its column pass write and about half a point of taps read).
constexpr int kDocPointCost = 10;
constexpr int kClassPointCost = 3;
// Documents of one size class that share a row task of the matrix-core row pass
constexpr int kMaxGroupDocs = 4;
// Filter gradient: documents of one size class whose correlation products the
// matrix-core row pass adds before its one inverse transform (fp16 sums: the bound on
// one document's product leaves room for far more)
constexpr int kMaxSumDocs = 8;
// Rows of at most this many points are batched 16 / m to a matrix-core block, when
// they hold at least 1 / kBatchMinShare of the grid (measured: +2.5% on a batch of
// mostly 1-8-point rows, -1% when three such documents sit among long ones)
constexpr int kMaxBatchM = 8;
constexpr int kBatchMinShare = 4;

struct Seg {
    int32_t row;       // source row of x (documents) / 0 (filter classes)
    int32_t start;     // first token in the row / 0
    int32_t len;       // tokens that are read (document length / filter taps kept)
    int32_t m;         // row DFT size; P = N1 * m
    int32_t P;
    int32_t cls;       // size class
    int64_t grid_off;  // first grid point of this segment in its grid buffer
    int32_t tw_off;    // class roots w_m^h, h < m, at [tw_off, tw_off + m) (complex)
    int32_t twf_off;   // class roots w_P^r / sqrt(N1), r < P, at [twf_off, twf_off + P)
    int32_t spec_off;  // first grid point of the class's filter grid (the "spectrum" buffer)
    int32_t col0;      // first global column index of this segment
    int32_t task0;     // first global row-task index of this segment (generic row kernel)
    int32_t spb;       // pairs per row task (16, or fewer for long rows)
    int32_t list0;     // classes: first entry of this class in the class-ordered document list
    int32_t nlist;     // classes: number of documents in the class
    int32_t nfac;      // radices of m, applied in order
    int8_t fac[kMaxFactors];
    int8_t pad_[2];
    int32_t dense_off; // matrix-core row pass: first 16-byte entry of the class's DFT operands
};
static_assert(sizeof(Seg) % 8 == 0, "Seg must stay 8-byte aligned in arrays");

// Rows longer than kMaxFastM points on fp16 grids take a second four-step level: a row of
// m = m1 * m2 points (j = m2 j1 + j2) becomes m1 sub-rows of m2 points, sub-row k1 of
// grid row u at sub-row index k1 N1 + u of a virtual document of N1 m1 rows, whose
// partner rows and columns then follow the same rules as the grid's own rows.  The
// sub-rows live in a region of the same grid buffer past the documents' grids.
struct LrItem {
    int64_t real_off;  // first grid point of the document (or class) grid
    int64_t virt_off;  // first point of its sub-row region
    int32_t m, m1, m2;
    int32_t tw_off;    // w_m^h, h < m, in the plan's twiddles
};
static_assert(sizeof(LrItem) % 8 == 0, "LrItem must stay 8-byte aligned in arrays");
// sub-row counts the first level may take (register-resident DFTs), smallest first
constexpr int kLrRadices[] = {2, 3, 4, 5, 6, 8, 9, 10, 12, 15, 16, 20, 24, 25, 30, 32};

}  // namespace rubiconv
