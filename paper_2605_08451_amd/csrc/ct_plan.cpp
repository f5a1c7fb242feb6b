// ct_plan.cpp -- host tables of the masked Cooley-Tukey convolution (ct_plan.hpp).
#include "ct_plan.hpp"

#include <algorithm>
#include <cmath>
#include <limits>

namespace rubiconv::ct {

int ct_log_size(int len, int L) {
    const int64_t need = std::max<int64_t>(1, static_cast<int64_t>(len) + std::min(len, L) - 1);
    int lg = 0;
    while ((int64_t(1) << lg) < need) ++lg;
    return lg;
}

namespace {

// Packs `docs` longest first and fills the tile and work tables.  The spec field of
// every entry is set from class_spec (indexed by logp).
void pack(std::vector<Doc> docs, const int64_t* class_spec, Layout* out) {
    std::stable_sort(docs.begin(), docs.end(),
                     [](const Doc& a, const Doc& b) { return a.logp > b.logp; });
    int64_t off = 0;
    out->n_long = 0;
    for (Doc& d : docs) {
        d.off = static_cast<int32_t>(off);
        d.spec = static_cast<int32_t>(class_spec[d.logp]);
        off += int64_t(1) << d.logp;
        if (d.logp > kLogTile) {
            ++out->n_long;
            out->long_points = off;
        }
    }
    out->points = (off + kTile - 1) / kTile * kTile;
    out->long_tile_doc.clear();
    out->col_items.clear();
    for (int i = 0; i < out->n_long; ++i) {
        for (int64_t t = 0; t < (int64_t(1) << docs[i].logp) / kTile; ++t) out->long_tile_doc.push_back(i);
    }
    // column items: M = P / kTile per document (each holds kTile points of every
    // pair lane), document by document, so that the items reading adjacent columns
    // of one document are dispatched together; documents with more than 2^kMaxLogCols
    // points per column also get M middle-pass tiles
    out->mid_tiles.clear();
    for (int i = 0; i < out->n_long; ++i) {
        const int lg_m = docs[i].logp - kLogTile;
        const int M = 1 << lg_m;
        for (int g = 0; g < M; ++g) out->col_items.push_back((i << kItemBits) | g);
        if (lg_m > kMaxLogCols)
            for (int t = 0; t < M; ++t) out->mid_tiles.push_back((i << kItemBits) | t);
    }
    out->short_tile_docs.clear();
    const int64_t n_short_tiles = (out->points - out->long_points) / kTile;
    size_t d = static_cast<size_t>(out->n_long);
    for (int64_t t = 0; t < n_short_tiles; ++t) {
        const int64_t lo = out->long_points + t * kTile, hi = lo + kTile;
        const size_t first = d;
        while (d < docs.size() && docs[d].off < hi) ++d;
        (void)lo;
        out->short_tile_docs.push_back(static_cast<int32_t>(first));
        out->short_tile_docs.push_back(static_cast<int32_t>(d));
    }
    out->docs = std::move(docs);
}

}  // namespace

CtError build_ct_plan(CtHostPlan* out, int B, int N, int D, int L, int max_docs,
                      const int32_t* cu, int x_dtype, int y_dtype) {
    if (!out || !cu || B < 1 || N < 1 || D < 2 || L < 1 || max_docs < 1) return CtError::kArg;
    if (x_dtype < 0 || x_dtype > 1 || y_dtype < 0 || y_dtype > 1) return CtError::kArg;
    if (D % 2) return CtError::kUnsupported;  // channels are transformed in pairs
    if (static_cast<int64_t>(B) * N * D > (int64_t(1) << 40)) return CtError::kUnsupported;
    for (int b = 0; b < B; ++b) {
        const int32_t* c = cu + static_cast<int64_t>(b) * (max_docs + 1);
        if (c[0] != 0 || c[max_docs] != N) return CtError::kSeqlens;
        for (int k = 0; k < max_docs; ++k)
            if (c[k + 1] < c[k] || c[k + 1] > N) return CtError::kSeqlens;
    }
    CtHostPlan p;
    p.B = B; p.N = N; p.D = D; p.L = L; p.max_docs = max_docs;
    p.x_dtype = x_dtype; p.y_dtype = y_dtype;
    p.grid_half = x_dtype == 1;
    p.npb = (D / 2 + kPairs - 1) / kPairs;

    std::vector<Doc> docs;
    bool present[kMaxLogP + 1] = {};
    for (int b = 0; b < B; ++b) {
        const int32_t* c = cu + static_cast<int64_t>(b) * (max_docs + 1);
        for (int k = 0; k < max_docs; ++k) {
            const int len = c[k + 1] - c[k];
            if (len == 0) continue;
            const int lg = ct_log_size(len, L);
            if (lg > kMaxLogP) return CtError::kUnsupported;
            present[lg] = true;
            docs.push_back(Doc{b, c[k], len, lg, 0, 0, k, 0});
        }
    }
    // spectrum: per size class (longest first) [pair block][f <= P/2][16 pairs]
    int64_t class_spec[kMaxLogP + 1];
    int64_t entries = 0;
    std::vector<Doc> classes;
    for (int lg = kMaxLogP; lg >= 0; --lg) {
        class_spec[lg] = -1;
        if (!present[lg]) continue;
        class_spec[lg] = entries;
        entries += static_cast<int64_t>(p.npb) * ((int64_t(1) << lg) / 2 + 1) * kPairs;
        // taps every document of this class needs, and no more than the padding allows
        // without wrapping onto an output position: min(L, floor((P + 1) / 2))
        const int taps = static_cast<int>(std::min<int64_t>(L, ((int64_t(1) << lg) + 1) / 2));
        p.taps_max = std::max(p.taps_max, taps);
        classes.push_back(Doc{0, 0, taps, lg, 0, 0, 0, 0});
    }
    if (entries > std::numeric_limits<int32_t>::max()) return CtError::kUnsupported;
    p.spec_entries = entries;
    pack(std::move(docs), class_spec, &p.data);
    pack(std::move(classes), class_spec, &p.filt);
    if (p.data.points > std::numeric_limits<int32_t>::max()) return CtError::kUnsupported;

    const int half = 1 << (kMaxLogP - 1);
    p.tw.resize(2 * static_cast<size_t>(half));
    for (int j = 0; j < half; ++j) {
        const double a = -2.0 * M_PI * j / static_cast<double>(1 << kMaxLogP);
        p.tw[2 * j] = static_cast<float>(std::cos(a));
        p.tw[2 * j + 1] = static_cast<float>(std::sin(a));
    }
    *out = std::move(p);
    return CtError::kOk;
}

}  // namespace rubiconv::ct
