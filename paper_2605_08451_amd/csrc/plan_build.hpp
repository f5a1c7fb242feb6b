// plan_build.hpp -- host-side construction of a plan's tables (no HIP calls).
#pragma once

#include <cstdint>
#include <vector>

#include "plan.hpp"

namespace rubiconv {

enum class BuildError { kOk, kArg, kSeqlens, kUnsupported };

struct HostPlan {
    int B = 0, N = 0, D = 0, L = 0, max_docs = 0, n1 = 0, r = 0;  // n1 = r * r
    int x_dtype = 0, y_dtype = 0;
    bool grid_half = false;             // complex fp16 grids and spectra (else complex fp32)
    int npb = 0;                        // channel-pair blocks of kPairsPerBlock pairs
    std::vector<Seg> docs;              // one per non-empty document, row order
    std::vector<int32_t> doc_index;     // index of each document inside its row
    // Documents of at most direct_max tokens skip the transforms: their outputs are the
    // defining sums, computed directly (direct_docs: row, start, len; m = P = 0).
    int direct_max = 0;
    int direct_taps = 0;                // taps the direct path reads: min(L, direct_max)
    bool direct_mfma = false;           // the direct path on the matrix cores (taps [D][T] as bf16 hi, lo)
    std::vector<Seg> direct_docs;
    std::vector<int32_t> direct_index;  // index of each direct document inside its row
    // every non-empty document in row order (transformed ones with their m and P,
    // direct ones with m = P = 0): the plan's document table
    std::vector<Seg> all_docs;
    std::vector<int32_t> all_index;
    std::vector<Seg> classes;           // one per distinct m, ascending m
    std::vector<int32_t> doc_col_seg;   // global column -> document
    std::vector<int32_t> doc_task_seg;  // global row task -> document
    std::vector<int32_t> cls_col_seg;   // global column -> class
    std::vector<int32_t> class_docs;    // documents grouped by class (class order)
    std::vector<int32_t> class_ident;   // 0, 1, ..., n_classes - 1
    std::vector<float> tw;              // complex pairs (re, im), per class: N1 then m entries
    std::vector<float> tw_n1;           // complex pairs, w_N1^s for s < N1
    std::vector<uint32_t> mfma_tab;     // matrix-core operand tables (N1 = 256 only)
    bool col_mfma = false;              // column passes on the matrix cores
    bool row_dense = false;             // row pass on the matrix cores for m <= 16 * kMaxDenseBlocks
    std::vector<uint32_t> dense_tab;    // per class: forward then inverse row DFT operands
    std::vector<int32_t> dense_docs;    // documents grouped by 16-point block count nb = ceil(m / 16)
    int32_t dense_list0[kMaxDenseBlocks + 1] = {};  // first entry of block count nb in dense_docs
    int32_t dense_count[kMaxDenseBlocks + 1] = {};  // documents with block count nb
    // row-task groups, pairs (first entry in dense_docs, documents): the documents of
    // one size class, at most kMaxGroupDocs per group, share one load and transform of
    // the class's filter rows
    std::vector<int32_t> dense_groups;
    int32_t dense_grp0[kMaxDenseBlocks + 1] = {};   // class groups of block count nb (pair index)
    int32_t dense_grp_n[kMaxDenseBlocks + 1] = {};
    // filter gradient (each document's second operand its own grid): sum groups, pairs
    // (first entry in dense_sdocs, documents), of at most kMaxSumDocs documents of one
    // size class, longest first; the row pass adds their correlation products and writes
    // the inverse of the sum over the first document's rows
    std::vector<int32_t> dense_sdocs;
    std::vector<int32_t> dense_sgroups;
    int32_t dense_sgrp0[kMaxDenseBlocks + 1] = {};  // sum groups of block count nb (pair index)
    int32_t dense_sgrp_n[kMaxDenseBlocks + 1] = {};
    // filter gradient outputs: the documents whose rows hold correlations after the row
    // pass (sum-group leaders and every document outside the sum groups), as copies of
    // their segments with the second rows their own and columns renumbered (dk_segs,
    // dk_col_seg: the inverse column pass), and with the direct documents, longest first
    // (ties in table order), for the lag sum (dk_sum_segs)
    std::vector<Seg> dk_segs;
    std::vector<int32_t> dk_col_seg;
    std::vector<Seg> dk_sum_segs;
    // rows of at most kMaxBatchM points: class groups of the batched kernel, which puts
    // 16 / m documents side by side in one block (for the filter gradient as well, as it
    // takes each document's second rows from that document)
    int32_t dense_bgrp0 = 0, dense_bgrp_n = 0;
    double dense_bwork = 0;                          // their summed row sizes
    // long rows: the documents' and classes' first-level items, the virtual documents
    // (m = m2, offsets into the sub-row regions; spec_off of lr_segs points at the
    // class's sub-rows, of lr_gsegs at the document's own), identity indices, and per
    // long class one row launch of N1 m1 rows with its class groups and one-document
    // groups (pairs into lr_idx)
    std::vector<LrItem> lr_doc_items, lr_cls_items;
    std::vector<Seg> lr_segs, lr_gsegs;
    std::vector<int32_t> lr_idx, lr_groups;
    struct LrLaunch { int m1, nb, grp0, grp_n, dgrp0, dgrp_n; double work; };
    std::vector<LrLaunch> lr_launches;
    int64_t grid_points_lr = 0, class_points_lr = 0;  // the sub-row regions
    int64_t grid_points = 0;            // sum over documents of P_i
    int64_t class_points = 0;           // sum over classes of P
    int32_t taps_max = 0;               // largest number of filter taps any class keeps
    int32_t row_lds_docs = 0;           // dynamic LDS bytes of the generic row kernel
};

// Smallest 2^a 3^b 5^c >= v (v >= 1).
int smooth_ceil(int v);

// The direct path can run on the matrix cores: bf16 x and dy (dtype 1), channels in
// blocks of 32.
inline bool direct_mfma_possible(int x_dtype, int y_dtype, int D) {
    return x_dtype == 1 && y_dtype == 1 && D % 32 == 0;
}

// MFMA operand tables of the N1 = 256 matrix-core column passes (kMtEntries
// 16-byte entries, 4 x uint32 each, in the order of kernels.hpp's kMt* offsets).
void build_mfma_tables(std::vector<uint32_t>* out);

// Operands of the matrix-core row pass for one size class (m <= 16 * kMaxDenseBlocks,
// nb = ceil(m / 16)): the forward m-point DFT with entries w_m^(-k j) / sqrt(m) and the
// inverse with entries (sqrt(n1) / 4) w_m^(k j), zero outside k, j < m, each as nb x nb
// blocks (output block major) of the two 16 x 32 real operands; 4 * nb^2 * 64 entries.
void build_dense_tables(int m, int n1, std::vector<uint32_t>* out);
// Matrix-core row pass for 32 < m <= 16 * kMaxDenseBlocks: one real operand per block
// and direction, then the partner-row twiddles (kernels.hpp: kPartnerTabU4).
void build_partner_tables(int m, int n1, std::vector<uint32_t>* out);
// Batched rows (m <= kMaxBatchM): the tables of build_dense_tables in block-diagonal form
// for 16 / m rows side by side (row r at slots r m .. r m + m - 1).
void build_batch_tables(int m, int n1, std::vector<uint32_t>* out);

// Validates cu_seqlens and fills every table of *out.
// direct_max: documents of at most this many tokens take the direct path (0: none);
// with direct_by_share they do so only when they would hold at least 1/kDirectMinShare
// of the transform grid (plan.hpp).
// merge_classes: documents may take a larger listed row size than their own when
// that removes a filter class and saves bytes overall (merge_size_classes).
BuildError build_host_plan(HostPlan* out, int B, int N, int D, int L, int max_docs,
                           const int32_t* cu_seqlens, int x_dtype, int y_dtype, int n1,
                           int direct_max, bool direct_by_share, bool merge_classes,
                           bool direct_mfma = false);

// Row sizes after class merging, one per entry of m0 (each a valid size for its
// document).  Sizes u_1 < ... < u_k with document counts c_t; a class of size u_j
// serving the sizes u_i..u_j costs kClassPointCost u_j + kDocPointCost u_j (c_i + ... + c_j),
// and the cheapest split into consecutive groups is found by dynamic programming.
// A size above max_merge_m never absorbs a smaller one.
std::vector<int> merge_size_classes(const std::vector<int>& m0, int max_merge_m);

}  // namespace rubiconv
