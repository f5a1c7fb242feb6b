// ct_plan.hpp -- host tables of the masked Cooley-Tukey convolution (Algorithm 2).
//
// Every non-empty document i gets the power-of-two size P_i, the smallest power of
// two >= L_i + min(L_i, L) - 1 (the causal zero padding of Algorithm 1 with the
// power-of-two length Algorithm 2 needs).  The documents of all rows are packed
// back to back in one flat array, longest first: every document then starts at a
// multiple of its own size, the documents longer than a tile of kTile points form
// a prefix made of whole tiles, and each later tile holds whole documents only.
// No HIP calls here.
#pragma once

#include <cstdint>
#include <vector>

namespace rubiconv::ct {

constexpr int kLogTile = 9;
constexpr int kTile = 1 << kLogTile;          // points one workgroup transforms in LDS
constexpr int kMaxLogCols = 6;                // column pass: up to 64 points per column
constexpr int kMaxLogMid = 4;                 // middle pass: up to 4 stages before the column pass
constexpr int kMaxLogP = kLogTile + kMaxLogMid + kMaxLogCols;  // largest transform, 2^19 points
constexpr int kItemBits = kMaxLogMid + kMaxLogCols;  // work-item index inside a document
constexpr int kPairs = 16;                    // channel pairs per block (32 channels)

// One transformed array of the flat layout: a document, or a filter size class.
struct Doc {
    int32_t row, start, len;  // tokens [start, start + len) of row `row`
    int32_t logp;             // P = 2^logp
    int32_t off;              // first point in the flat layout (a multiple of P)
    int32_t spec;             // first spectrum entry of its size class
    int32_t index;            // index inside its row (documents) / 0 (filter classes)
    int32_t pad;
};
static_assert(sizeof(Doc) == 32, "Doc is read as two 16-byte words");

struct Layout {
    std::vector<Doc> docs;                // longest first
    int32_t n_long = 0;                   // documents with P > kTile (a prefix of docs)
    int64_t long_points = 0;              // their points (whole tiles)
    int64_t points = 0;                   // all points, the short region rounded up to a tile
    std::vector<int32_t> long_tile_doc;   // tile of the long region -> its document
    std::vector<int32_t> short_tile_docs; // tile of the short region -> first and end document
    std::vector<int32_t> col_items;       // column work item -> document << kItemBits | group
    std::vector<int32_t> mid_tiles;       // middle-pass tile -> document << kItemBits | tile
};

struct CtHostPlan {
    int B = 0, N = 0, D = 0, L = 0, max_docs = 0, x_dtype = 0, y_dtype = 0;
    bool grid_half = false;   // long-document grid in complex fp16 (bf16 inputs)
    int npb = 0;              // channel-pair blocks
    Layout data;              // the documents
    Layout filt;              // one array per size class, its filter taps as the "document"
    int32_t taps_max = 0;     // most taps any size class keeps
    int64_t spec_entries = 0; // 16-byte spectrum entries (U and V of one channel pair)
    std::vector<float> tw;    // (re, im) of exp(-2 pi i j / 2^kMaxLogP), j < 2^(kMaxLogP - 1)
};

enum class CtError { kOk, kArg, kSeqlens, kUnsupported };

// P_i's exponent for a document of `len` tokens and filters of L taps.
int ct_log_size(int len, int L);

// Validates cu_seqlens ([B][max_docs + 1], host) and fills *out.
CtError build_ct_plan(CtHostPlan* out, int B, int N, int D, int L, int max_docs,
                      const int32_t* cu_seqlens, int x_dtype, int y_dtype);

}  // namespace rubiconv::ct
