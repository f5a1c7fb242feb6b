// ct_api.cpp -- the C ABI declared in include/rubiconv_ct.h.
//
// rubiconv_ct_plan builds the flat layout on the host (ct_plan.cpp) and uploads
// its tables in one device allocation; the stream calls enqueue the kernels of
// ct_kernels.hip on the caller's stream.
#include "rubiconv_ct.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "ct_kernels.hpp"
#include "ct_plan.hpp"
#include "kernels.hpp"

using rubiconv::ct::CtError;
using rubiconv::ct::CtHostPlan;
using rubiconv::ct::Doc;
using rubiconv::ct::kPairs;
using rubiconv::ct::kTile;
using rubiconv::ct::Layout;

namespace {

struct DevLayout {
    const Doc* docs = nullptr;
    const int32_t* long_tile_doc = nullptr;
    const int32_t* short_tile_docs = nullptr;
    const int32_t* col_items = nullptr;
    const int32_t* mid_tiles = nullptr;
    int n_long_tiles = 0, n_short_tiles = 0, n_items = 0, n_mid = 0;
};

}  // namespace

struct rubiconv_ct_plan_s {
    CtHostPlan h;
    void* dev = nullptr;
    bool device_ready = false;
    DevLayout data, filt;
    const float2* tw = nullptr;
    size_t spec_bytes = 0;
    size_t ws_bytes = 0;
    size_t taps_bytes = 0;   // filter call: transposed taps, then the long classes' grid
};

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct Blob {
    std::vector<unsigned char> img;
    size_t add(const void* p, size_t bytes) {
        const size_t off = img.size();
        img.resize(align_up(off + std::max<size_t>(bytes, 1)), 0);
        if (bytes) std::memcpy(img.data() + off, p, bytes);
        return off;
    }
};

struct LayoutOffsets {
    size_t docs, ltd, std_, items, mid;
};

LayoutOffsets add_layout(Blob& b, const Layout& l) {
    LayoutOffsets o;
    o.docs = b.add(l.docs.data(), l.docs.size() * sizeof(Doc));
    o.ltd = b.add(l.long_tile_doc.data(), l.long_tile_doc.size() * 4);
    o.std_ = b.add(l.short_tile_docs.data(), l.short_tile_docs.size() * 4);
    o.items = b.add(l.col_items.data(), l.col_items.size() * 4);
    o.mid = b.add(l.mid_tiles.data(), l.mid_tiles.size() * 4);
    return o;
}

DevLayout dev_layout(const unsigned char* base, const LayoutOffsets& o, const Layout& l) {
    DevLayout d;
    d.docs = reinterpret_cast<const Doc*>(base + o.docs);
    d.long_tile_doc = reinterpret_cast<const int32_t*>(base + o.ltd);
    d.short_tile_docs = reinterpret_cast<const int32_t*>(base + o.std_);
    d.col_items = reinterpret_cast<const int32_t*>(base + o.items);
    d.n_long_tiles = static_cast<int>(l.long_tile_doc.size());
    d.n_short_tiles = static_cast<int>(l.short_tile_docs.size() / 2);
    d.n_items = static_cast<int>(l.col_items.size());
    d.mid_tiles = reinterpret_cast<const int32_t*>(base + o.mid);
    d.n_mid = static_cast<int>(l.mid_tiles.size());
    return d;
}

rubiconv_status_t upload(rubiconv_ct_plan_s* pl) {
    const CtHostPlan& h = pl->h;
    Blob b;
    const LayoutOffsets od = add_layout(b, h.data);
    const LayoutOffsets of = add_layout(b, h.filt);
    const size_t o_tw = b.add(h.tw.data(), h.tw.size() * sizeof(float));
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e == hipErrorNoDevice || (e == hipSuccess && count == 0)) {
        (void)hipGetLastError();
        return RUBICONV_OK;  // host-only plan: the stream calls report RUBICONV_ERR_HIP
    }
    if (e != hipSuccess) return RUBICONV_ERR_HIP;
    void* d = nullptr;
    e = hipMalloc(&d, b.img.size());
    if (e == hipErrorOutOfMemory) return RUBICONV_ERR_ALLOC;
    if (e != hipSuccess) return RUBICONV_ERR_HIP;
    if (hipMemcpy(d, b.img.data(), b.img.size(), hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(d);
        return RUBICONV_ERR_HIP;
    }
    pl->dev = d;
    const unsigned char* base = static_cast<const unsigned char*>(d);
    pl->data = dev_layout(base, od, h.data);
    pl->filt = dev_layout(base, of, h.filt);
    pl->tw = reinterpret_cast<const float2*>(base + o_tw);
    pl->device_ready = true;
    return RUBICONV_OK;
}

}  // namespace

extern "C" {

rubiconv_status_t rubiconv_ct_plan(rubiconv_ct_plan_t* out, int B, int N, int D, int L,
                                   int max_docs, const int32_t* cu_seqlens_host,
                                   rubiconv_dtype_t x_dtype, rubiconv_dtype_t y_dtype) {
    if (!out) return RUBICONV_ERR_ARG;
    *out = nullptr;
    rubiconv_ct_plan_s* pl = new (std::nothrow) rubiconv_ct_plan_s();
    if (!pl) return RUBICONV_ERR_ALLOC;
    const CtError be = rubiconv::ct::build_ct_plan(&pl->h, B, N, D, L, max_docs, cu_seqlens_host,
                                                   static_cast<int>(x_dtype), static_cast<int>(y_dtype));
    if (be != CtError::kOk) {
        delete pl;
        if (be == CtError::kArg) return RUBICONV_ERR_ARG;
        if (be == CtError::kSeqlens) return RUBICONV_ERR_SEQLENS;
        return RUBICONV_ERR_UNSUPPORTED;
    }
    const CtHostPlan& h = pl->h;
    const size_t esz = h.grid_half ? 4 : 8;
    pl->spec_bytes = std::max(kAlign, align_up(static_cast<size_t>(h.spec_entries) * (h.grid_half ? 8 : 16)));
    const size_t conv_ws = align_up(static_cast<size_t>(h.npb) * h.data.long_points * kPairs * esz);
    pl->taps_bytes = align_up(static_cast<size_t>(h.taps_max) * h.D * 4);
    const size_t filt_ws = pl->taps_bytes + align_up(static_cast<size_t>(h.npb) * h.filt.long_points * kPairs * 8);
    pl->ws_bytes = std::max({conv_ws, filt_ws, kAlign});
    const rubiconv_status_t st = upload(pl);
    if (st != RUBICONV_OK) {
        if (pl->dev) (void)hipFree(pl->dev);
        delete pl;
        return st;
    }
    *out = pl;
    return RUBICONV_OK;
}

void rubiconv_ct_plan_destroy(rubiconv_ct_plan_t plan) {
    if (!plan) return;
    if (plan->dev) (void)hipFree(plan->dev);
    delete plan;
}

size_t rubiconv_ct_spectrum_bytes(rubiconv_ct_plan_t plan) { return plan ? plan->spec_bytes : 0; }

size_t rubiconv_ct_workspace_bytes(rubiconv_ct_plan_t plan) { return plan ? plan->ws_bytes : 0; }

rubiconv_status_t rubiconv_ct_filter_spectrum(rubiconv_ct_plan_t plan, const float* filters,
                                              void* spectrum, void* workspace, hipStream_t stream) {
    if (!plan || !filters || !spectrum || !workspace) return RUBICONV_ERR_ARG;
    if (!aligned(spectrum, kAlign) || !aligned(workspace, kAlign) || !aligned(filters, 4))
        return RUBICONV_ERR_ARG;
    if (!plan->device_ready) return RUBICONV_ERR_HIP;
    const CtHostPlan& h = plan->h;
    float* taps = static_cast<float*>(workspace);
    void* fgrid = static_cast<char*>(workspace) + plan->taps_bytes;
    const DevLayout& f = plan->filt;
    hipError_t e = rubiconv::launch_transpose(filters, h.D, h.taps_max, h.L, taps, h.D, nullptr, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_front(f.docs, f.long_tile_doc, f.n_long_tiles, 0, taps, 0, h.D, h.npb,
                                       false, fgrid, h.filt.long_points, plan->tw, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_mid(false, f.docs, f.mid_tiles, f.n_mid, false, fgrid, h.filt.long_points,
                                     h.npb, plan->tw, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_col(1, f.docs, f.col_items, f.n_items, false, fgrid, h.filt.long_points,
                                     h.npb, h.grid_half, spectrum, plan->tw, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_short(1, f.docs, f.short_tile_docs, f.n_short_tiles, h.filt.long_points, 0,
                                       taps, 0, h.D, h.npb, h.grid_half, spectrum, 0, nullptr, plan->tw,
                                       stream);
    return e == hipSuccess ? RUBICONV_OK : RUBICONV_ERR_HIP;
}

rubiconv_status_t rubiconv_ct_packed_conv(rubiconv_ct_plan_t plan, const void* x,
                                          const void* spectrum, void* y, void* workspace,
                                          hipStream_t stream) {
    if (!plan || !x || !spectrum || !y || !workspace) return RUBICONV_ERR_ARG;
    const CtHostPlan& h = plan->h;
    // channel pairs are read and written as one 8-byte (fp32) or 4-byte (bf16) word
    const size_t xa = h.x_dtype == RUBICONV_F32 ? 8 : 4, ya = h.y_dtype == RUBICONV_F32 ? 8 : 4;
    if (!aligned(spectrum, kAlign) || !aligned(workspace, kAlign) || !aligned(x, xa) || !aligned(y, ya))
        return RUBICONV_ERR_ARG;
    if (!plan->device_ready) return RUBICONV_ERR_HIP;
    const DevLayout& d = plan->data;
    void* spec = const_cast<void*>(spectrum);  // read only by the convolution's kernels
    hipError_t e = rubiconv::ct::launch_short(0, d.docs, d.short_tile_docs, d.n_short_tiles,
                                              h.data.long_points, h.x_dtype, x, h.N, h.D, h.npb,
                                              h.grid_half, spec, h.y_dtype, y, plan->tw, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_front(d.docs, d.long_tile_doc, d.n_long_tiles, h.x_dtype, x, h.N, h.D,
                                       h.npb, h.grid_half, workspace, h.data.long_points, plan->tw, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_mid(false, d.docs, d.mid_tiles, d.n_mid, h.grid_half, workspace,
                                     h.data.long_points, h.npb, plan->tw, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_col(0, d.docs, d.col_items, d.n_items, h.grid_half, workspace,
                                     h.data.long_points, h.npb, h.grid_half, spec, plan->tw, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_mid(true, d.docs, d.mid_tiles, d.n_mid, h.grid_half, workspace,
                                     h.data.long_points, h.npb, plan->tw, stream);
    if (e == hipSuccess)
        e = rubiconv::ct::launch_back(d.docs, d.long_tile_doc, d.n_long_tiles, h.grid_half, workspace,
                                      h.data.long_points, h.npb, h.y_dtype, y, h.N, h.D, plan->tw, stream);
    return e == hipSuccess ? RUBICONV_OK : RUBICONV_ERR_HIP;
}

rubiconv_status_t rubiconv_ct_plan_doc_table(rubiconv_ct_plan_t plan, int32_t* out, int cap,
                                             int* n_docs) {
    if (!plan || !n_docs || cap < 0 || (cap > 0 && !out)) return RUBICONV_ERR_ARG;
    std::vector<Doc> docs(plan->h.data.docs);
    std::sort(docs.begin(), docs.end(), [](const Doc& a, const Doc& b) {
        return a.row != b.row ? a.row < b.row : a.start < b.start;
    });
    const int n = static_cast<int>(docs.size());
    *n_docs = n;
    for (int i = 0; i < n && i < cap; ++i) {
        int32_t* o = out + 6 * static_cast<int64_t>(i);
        o[0] = docs[i].row; o[1] = docs[i].index; o[2] = docs[i].start; o[3] = docs[i].len;
        o[4] = 1 << docs[i].logp; o[5] = docs[i].off;
    }
    return RUBICONV_OK;
}

}  // extern "C"
