// rubiconv.cpp -- the C ABI declared in include/rubiconv.h.
//
// rubiconv_plan validates the document boundaries and builds every table on the
// host (plan_build.cpp), then uploads them in one device allocation.  The two
// stream calls only enqueue kernels (kernels.hip) on the caller's stream.
#include "rubiconv.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "plan_build.hpp"
#include "row_sizes.hpp"

using rubiconv::BuildError;
using rubiconv::GridScale;
using rubiconv::HostPlan;
using rubiconv::kPairsPerBlock;
using rubiconv::LaunchTables;
using rubiconv::Seg;

struct rubiconv_plan_s {
    HostPlan h;
    void* dev = nullptr;  // all device tables, one allocation
    std::vector<unsigned char> host_image;  // their host copy, the source of the upload
    hipEvent_t uploaded = nullptr;          // recorded after the upload (destroy waits for it)
    const void* mfma_tab = nullptr;  // matrix-core operand tables (inside dev)
    const void* dense_tab = nullptr; // matrix-core row pass operands (inside dev)
    const int32_t* dense_docs = nullptr;  // documents by 16-point block count (inside dev)
    const int32_t* dense_groups = nullptr;  // row-task groups of dense_docs (inside dev)
    const int32_t* dense_sdocs = nullptr;   // filter gradient: sum-group documents (inside dev)
    const int32_t* dense_sgroups = nullptr; //   their groups
    const Seg* lr_segs = nullptr;           // long rows: sub-row documents (inside dev)
    const Seg* lr_gsegs = nullptr;          //   the same, second rows their own (filter gradient)
    const int32_t* lr_idx = nullptr;        //   identity indices
    const int32_t* lr_groups = nullptr;     //   groups of the sub-row launches
    const float2* ones = nullptr;           // {1, 1} per channel pair: the unit range scales
    const float2* dk_unscale = nullptr;     // {ed, 1 / ed} per channel pair (dk_split)
    bool device_ready = false;
    bool prescale_fwd = true;    // the forward prescales x as the gradients do dy (and x)
    // pinned host words, written by the matrix-core column passes: the range scales the
    // last calls found, per kind of call (forward x, dx dy, dk x, dk dy) and per input
    // buffer (kHintSlots slots hashed from its address, so that one plan shared by several
    // layers keeps each layer's scale).  A call starts its column pass at the scale of its
    // slot and redoes the pass only when its own scale differs; any value is correct, a
    // stale one costs the redo.
    static constexpr int kHintFwd = 0, kHintDx = 1, kHintDkX = 2, kHintDkDy = 3;
    static constexpr int kHintSlots = 64, kHints = 4 * kHintSlots;
    float* scale_hint = nullptr;      // host address
    float* scale_hint_dev = nullptr;  // the same words as kernels address them
    LaunchTables doc_t{};
    LaunchTables cls_t{};
    LaunchTables grad_t{};       // doc_t with each document's "filter" rows at its own grid rows
    LaunchTables dk_t{};         // grad_t restricted to the filter gradient's output documents
    const Seg* dk_sum_segs = nullptr;  // those and the direct documents, longest first (lag sum)
    const Seg* direct_segs = nullptr;  // documents of the direct path
    size_t dtaps_off = 0;        // spectrum: the direct path's taps, [direct_taps][D] fp32 or (matrix
                                 // cores) [D][direct_taps] bf16 pairs hi | lo << 16
    size_t sscale_off = 0;       // spectrum: the filter's range scales, float2 per channel pair
    size_t partials_off = 0;     // filter call's workspace: |k| sums per tap tile and channel
    size_t ws_hdr_off = 0;       // workspace: prescales of x and dy, then the amax partials
    size_t dk_hdr_off = 0;       // the same in the filter gradient's workspace
    int64_t grid_pb_stride = 0;  // grid elements per pair block, document grid
    int64_t cls_pb_stride = 0;   // same, filter class grids (the spectrum buffer)
    size_t taps_bytes = 0;       // transposed filter taps (workspace of the filter call)
    size_t spec_bytes = 0;
    size_t ws_bytes = 0;
    size_t grid_bytes = 0;       // one document grid (all pair blocks)
    size_t dk_ws_bytes = 0;      // rubiconv_packed_conv_dk: two grids and an fp32 [B][N][D] buffer
    // The row pass runs its size classes (independent launches) on side streams
    // forked from and joined back into the caller's stream with events; the mutex
    // keeps one call's record/wait sequence from interleaving with another's.
    static constexpr int kSideStreams = 2;
    hipStream_t side[kSideStreams] = {};
    hipEvent_t fork = nullptr;
    hipEvent_t direct_done = nullptr;  // the direct path's launch on its side stream
    hipEvent_t join[kSideStreams] = {};
    std::mutex launch_mu;
    // stage timing (rubiconv_profile_start / _read)
    static constexpr int kEventsPerCall = 16;  // before the first kernel + after each stage
    int prof_max = 0, prof_used = 0;
    // at least prof_max * kEventsPerCall events, created as profiling first needs them and
    // kept (re-recorded by later profiling) until the plan is destroyed
    std::vector<hipEvent_t> prof_events;
    std::vector<std::vector<std::string>> prof_names;
};

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) % kAlign) == 0; }

// The filter gradient's range split: x and dy carry ex and ed, together
// 2^-ceil(log2 P_max), as a correlation sums up to P products.
void dk_split(const HostPlan& h, float* ex, float* ed) {
    int pmax = 1;
    for (const Seg& d : h.docs) pmax = std::max(pmax, d.P);
    int lg = 0;
    while ((1 << lg) < pmax && lg < 30) ++lg;
    *ex = std::ldexp(1.0f, -(lg + 1) / 2);
    *ed = std::ldexp(1.0f, -(lg / 2));
}

rubiconv_status_t upload(rubiconv_plan_s* pl, hipStream_t stream) {
    const HostPlan& h = pl->h;
    const size_t n_segs = h.docs.size() + h.classes.size();
    size_t off = 0;
    const size_t o_segs = off;       off = align_up(off + n_segs * sizeof(Seg));
    const size_t o_gsegs = off;      off = align_up(off + h.docs.size() * sizeof(Seg));
    const size_t o_dsegs = off;      off = align_up(off + h.direct_docs.size() * sizeof(Seg));
    const size_t o_dcol = off;       off = align_up(off + h.doc_col_seg.size() * 4);
    const size_t o_dtask = off;      off = align_up(off + h.doc_task_seg.size() * 4);
    const size_t o_ccol = off;       off = align_up(off + h.cls_col_seg.size() * 4);
    const size_t o_tw = off;         off = align_up(off + h.tw.size() * 4);
    const size_t o_twn = off;        off = align_up(off + h.tw_n1.size() * 4);
    const size_t o_cdoc = off;       off = align_up(off + h.class_docs.size() * 4);
    const size_t o_cid = off;        off = align_up(off + h.class_ident.size() * 4);
    const size_t o_mt = off;         off = align_up(off + h.mfma_tab.size() * 4);
    const size_t o_dt = off;         off = align_up(off + h.dense_tab.size() * 4);
    const size_t o_dd = off;         off = align_up(off + h.dense_docs.size() * 4);
    const size_t o_dg = off;         off = align_up(off + h.dense_groups.size() * 4);
    const size_t o_sd = off;         off = align_up(off + h.dense_sdocs.size() * 4);
    const size_t o_sg = off;         off = align_up(off + h.dense_sgroups.size() * 4);
    const size_t o_ksegs = off;      off = align_up(off + h.dk_segs.size() * sizeof(Seg));
    const size_t o_kcol = off;       off = align_up(off + h.dk_col_seg.size() * 4);
    const size_t o_ksum = off;       off = align_up(off + h.dk_sum_segs.size() * sizeof(Seg));
    const size_t o_ls = off;         off = align_up(off + h.lr_segs.size() * sizeof(Seg));
    const size_t o_lg = off;         off = align_up(off + h.lr_gsegs.size() * sizeof(Seg));
    const size_t o_li = off;         off = align_up(off + h.lr_idx.size() * 4);
    const size_t o_lq = off;         off = align_up(off + h.lr_groups.size() * 4);
    const size_t n_ones = static_cast<size_t>(std::max(h.npb, 1)) * kPairsPerBlock;
    const size_t o_one = off;        off = align_up(off + n_ones * sizeof(float2));
    const size_t o_dku = off;        off = align_up(off + n_ones * sizeof(float2));
    const size_t total = off;

    // the host image stays with the plan: the copy below is stream-ordered and may still
    // be reading it when this call returns
    std::vector<unsigned char>& img = pl->host_image;
    img.assign(total, 0);
    std::vector<Seg> segs(h.docs);
    segs.insert(segs.end(), h.classes.begin(), h.classes.end());
    std::memcpy(img.data() + o_segs, segs.data(), n_segs * sizeof(Seg));
    if (!h.direct_docs.empty())
        std::memcpy(img.data() + o_dsegs, h.direct_docs.data(), h.direct_docs.size() * sizeof(Seg));
    {  // filter gradient: the second operand of a document's row stage is its own x grid
        std::vector<Seg> gsegs(h.docs);
        for (Seg& g : gsegs) g.spec_off = static_cast<int32_t>(g.grid_off);
        if (!gsegs.empty()) std::memcpy(img.data() + o_gsegs, gsegs.data(), gsegs.size() * sizeof(Seg));
    }
    std::memcpy(img.data() + o_dcol, h.doc_col_seg.data(), h.doc_col_seg.size() * 4);
    std::memcpy(img.data() + o_dtask, h.doc_task_seg.data(), h.doc_task_seg.size() * 4);
    std::memcpy(img.data() + o_ccol, h.cls_col_seg.data(), h.cls_col_seg.size() * 4);
    std::memcpy(img.data() + o_tw, h.tw.data(), h.tw.size() * 4);
    std::memcpy(img.data() + o_twn, h.tw_n1.data(), h.tw_n1.size() * 4);
    std::memcpy(img.data() + o_cdoc, h.class_docs.data(), h.class_docs.size() * 4);
    std::memcpy(img.data() + o_cid, h.class_ident.data(), h.class_ident.size() * 4);
    if (!h.mfma_tab.empty()) std::memcpy(img.data() + o_mt, h.mfma_tab.data(), h.mfma_tab.size() * 4);
    if (!h.dense_tab.empty()) std::memcpy(img.data() + o_dt, h.dense_tab.data(), h.dense_tab.size() * 4);
    if (!h.dense_docs.empty()) std::memcpy(img.data() + o_dd, h.dense_docs.data(), h.dense_docs.size() * 4);
    if (!h.dense_groups.empty())
        std::memcpy(img.data() + o_dg, h.dense_groups.data(), h.dense_groups.size() * 4);
    if (!h.dense_sdocs.empty()) {
        std::memcpy(img.data() + o_sd, h.dense_sdocs.data(), h.dense_sdocs.size() * 4);
        std::memcpy(img.data() + o_sg, h.dense_sgroups.data(), h.dense_sgroups.size() * 4);
    }
    if (!h.dk_segs.empty()) {
        std::memcpy(img.data() + o_ksegs, h.dk_segs.data(), h.dk_segs.size() * sizeof(Seg));
        std::memcpy(img.data() + o_kcol, h.dk_col_seg.data(), h.dk_col_seg.size() * 4);
    }
    if (!h.dk_sum_segs.empty())
        std::memcpy(img.data() + o_ksum, h.dk_sum_segs.data(), h.dk_sum_segs.size() * sizeof(Seg));
    {
        std::vector<float> ones(2 * n_ones, 1.0f);
        std::memcpy(img.data() + o_one, ones.data(), ones.size() * sizeof(float));
        float ex, ed;
        dk_split(h, &ex, &ed);
        std::vector<float2> dku(n_ones, make_float2(ed, 1.0f / ed));
        std::memcpy(img.data() + o_dku, dku.data(), dku.size() * sizeof(float2));
    }
    if (!h.lr_segs.empty()) {
        std::memcpy(img.data() + o_ls, h.lr_segs.data(), h.lr_segs.size() * sizeof(Seg));
        std::memcpy(img.data() + o_lg, h.lr_gsegs.data(), h.lr_gsegs.size() * sizeof(Seg));
        std::memcpy(img.data() + o_li, h.lr_idx.data(), h.lr_idx.size() * 4);
        std::memcpy(img.data() + o_lq, h.lr_groups.data(), h.lr_groups.size() * 4);
    }

    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e == hipErrorNoDevice || (e == hipSuccess && count == 0)) {
        (void)hipGetLastError();
        return RUBICONV_OK;  // host-only plan: tables exist, stream calls report ERR_HIP
    }
    if (e != hipSuccess) return RUBICONV_ERR_HIP;
    void* d = nullptr;
    e = hipMalloc(&d, total);
    if (e == hipErrorOutOfMemory) return RUBICONV_ERR_ALLOC;
    if (e != hipSuccess) return RUBICONV_ERR_HIP;
    e = hipMemcpyAsync(d, img.data(), total, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&pl->uploaded, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventRecord(pl->uploaded, stream);
    if (e != hipSuccess) {
        (void)hipStreamSynchronize(stream);
        (void)hipFree(d);
        return RUBICONV_ERR_HIP;
    }
    pl->dev = d;
    unsigned char* base = static_cast<unsigned char*>(d);
    const Seg* dsegs = reinterpret_cast<const Seg*>(base + o_segs);
    const float2* tw = reinterpret_cast<const float2*>(base + o_tw);
    const float2* twn = reinterpret_cast<const float2*>(base + o_twn);
    pl->doc_t = LaunchTables{dsegs, reinterpret_cast<const int32_t*>(base + o_dcol),
                             reinterpret_cast<const int32_t*>(base + o_dtask), tw, twn,
                             reinterpret_cast<const int32_t*>(base + o_cdoc)};
    pl->direct_segs = reinterpret_cast<const Seg*>(base + o_dsegs);
    pl->grad_t = pl->doc_t;
    pl->grad_t.segs = reinterpret_cast<const Seg*>(base + o_gsegs);
    pl->dk_t = pl->grad_t;
    pl->dk_t.segs = reinterpret_cast<const Seg*>(base + o_ksegs);
    pl->dk_t.col_seg = reinterpret_cast<const int32_t*>(base + o_kcol);
    pl->dk_sum_segs = reinterpret_cast<const Seg*>(base + o_ksum);
    pl->cls_t = LaunchTables{dsegs + h.docs.size(), reinterpret_cast<const int32_t*>(base + o_ccol),
                             nullptr, tw, twn,
                             reinterpret_cast<const int32_t*>(base + o_cid)};
    pl->mfma_tab = base + o_mt;
    pl->dense_tab = base + o_dt;
    pl->dense_docs = reinterpret_cast<const int32_t*>(base + o_dd);
    pl->dense_groups = reinterpret_cast<const int32_t*>(base + o_dg);
    pl->dense_sdocs = reinterpret_cast<const int32_t*>(base + o_sd);
    pl->dense_sgroups = reinterpret_cast<const int32_t*>(base + o_sg);
    pl->lr_segs = reinterpret_cast<const Seg*>(base + o_ls);
    pl->lr_gsegs = reinterpret_cast<const Seg*>(base + o_lg);
    pl->lr_idx = reinterpret_cast<const int32_t*>(base + o_li);
    pl->lr_groups = reinterpret_cast<const int32_t*>(base + o_lq);
    pl->ones = reinterpret_cast<const float2*>(base + o_one);
    pl->dk_unscale = reinterpret_cast<const float2*>(base + o_dku);
    // the fork and join events only order this device's streams: no system-scope fence
    // (the kernels' own release and acquire make their data visible across the device),
    // which spares a cache writeback and invalidation at every fork and join
    constexpr unsigned kOrderEvent = hipEventDisableTiming | hipEventDisableSystemFence;
    if (hipEventCreateWithFlags(&pl->fork, kOrderEvent) != hipSuccess ||
        hipEventCreateWithFlags(&pl->direct_done, kOrderEvent) != hipSuccess)
        return RUBICONV_ERR_HIP;
    for (int k = 0; k < rubiconv_plan_s::kSideStreams; ++k) {
        if (hipStreamCreateWithFlags(&pl->side[k], hipStreamNonBlocking) != hipSuccess ||
            hipEventCreateWithFlags(&pl->join[k], kOrderEvent) != hipSuccess)
            return RUBICONV_ERR_HIP;
    }
    if (hipHostMalloc(reinterpret_cast<void**>(&pl->scale_hint), rubiconv_plan_s::kHints * sizeof(float),
                      hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess)
        return RUBICONV_ERR_ALLOC;
    for (int i = 0; i < rubiconv_plan_s::kHints; ++i) pl->scale_hint[i] = 1.0f;
    if (hipHostGetDevicePointer(reinterpret_cast<void**>(&pl->scale_hint_dev), pl->scale_hint, 0) != hipSuccess)
        return RUBICONV_ERR_HIP;
    pl->device_ready = true;
    return RUBICONV_OK;
}

void destroy_side_streams(rubiconv_plan_s* pl) {
    for (int k = 0; k < rubiconv_plan_s::kSideStreams; ++k) {
        if (pl->side[k]) (void)hipStreamDestroy(pl->side[k]);
        if (pl->join[k]) (void)hipEventDestroy(pl->join[k]);
        pl->side[k] = nullptr;
        pl->join[k] = nullptr;
    }
    if (pl->fork) (void)hipEventDestroy(pl->fork);
    pl->fork = nullptr;
    if (pl->direct_done) (void)hipEventDestroy(pl->direct_done);
    pl->direct_done = nullptr;
}

void destroy_events(rubiconv_plan_s* pl) {
    for (hipEvent_t e : pl->prof_events) (void)hipEventDestroy(e);
    pl->prof_events.clear();
    pl->prof_names.clear();
    pl->prof_max = pl->prof_used = 0;
}

// Records an event before a call's first kernel and after each kernel while
// profiling slots remain; otherwise does nothing.
struct StageRecorder {
    rubiconv_plan_s* pl;
    hipStream_t stream;
    int slot = -1;
    int k = 0;
    StageRecorder(rubiconv_plan_s* p, hipStream_t s) : pl(p), stream(s) {
        if (pl->prof_used < pl->prof_max) {
            slot = pl->prof_used++;
            pl->prof_names[slot].clear();
            (void)hipEventRecord(pl->prof_events[slot * rubiconv_plan_s::kEventsPerCall], stream);
        }
    }
    bool active() const { return slot >= 0; }
    // records the stage's end; returns that event (null while not recording)
    hipEvent_t mark(const std::string& name) {
        if (slot < 0 || k + 1 >= rubiconv_plan_s::kEventsPerCall) return nullptr;
        ++k;
        hipEvent_t ev = pl->prof_events[slot * rubiconv_plan_s::kEventsPerCall + k];
        if (hipEventRecord(ev, stream) != hipSuccess) return nullptr;
        pl->prof_names[slot].push_back(name);
        return ev;
    }
};

// Starts the direct path's launch: on the last side stream, forked from `stream`, so
// that it runs beside the transforms; the caller joins with join_direct before the
// direct outputs are used or the call returns.  While stage timing records this call,
// the launch stays on `stream` so that its events time it.
template <class F>
hipError_t fork_direct(rubiconv_plan_s* plan, hipStream_t stream, StageRecorder& rec,
                       const char* name, F launch) {
    if (rec.active()) {
        const hipError_t e = launch(stream);
        rec.mark(name);
        return e;
    }
    hipStream_t side = plan->side[rubiconv_plan_s::kSideStreams - 1];
    hipError_t e = hipEventRecord(plan->fork, stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(side, plan->fork, 0);
    if (e == hipSuccess) e = launch(side);
    if (e == hipSuccess) e = hipEventRecord(plan->direct_done, side);
    return e;
}

hipError_t join_direct(rubiconv_plan_s* plan, hipStream_t stream, const StageRecorder& rec) {
    return rec.active() ? hipSuccess : hipStreamWaitEvent(stream, plan->direct_done, 0);
}

// The direct path's taps inside a spectrum buffer.
const float* direct_taps(const rubiconv_plan_s* plan, const void* spectrum) {
    return reinterpret_cast<const float*>(static_cast<const char*>(spectrum) + plan->dtaps_off);
}

// The matrix-core direct path moves 16-byte pieces of 8 channels: with it the tensors of
// a call must be 16-byte aligned.
bool direct_aligned(const rubiconv_plan_s* plan, std::initializer_list<const void*> ptrs) {
    if (!plan->h.direct_mfma) return true;
    for (const void* q : ptrs)
        if (reinterpret_cast<uintptr_t>(q) & 15) return false;
    return true;
}

// The direct path's sums (launch_direct's arguments): on the matrix cores when the plan
// says so, with the taps the filter call wrote for them.
hipError_t direct_sums(const rubiconv_plan_s* plan, int mode, int a_dtype, const void* a, int b_dtype,
                       const void* b, const float* taps, int out_dtype, void* out, hipStream_t s) {
    const HostPlan& h = plan->h;
    const int n = static_cast<int>(h.direct_docs.size());
    if (h.direct_mfma)
        return rubiconv::launch_direct_mfma(mode, a, b, reinterpret_cast<const uint32_t*>(taps), h.direct_taps,
                                            plan->direct_segs, n, h.N, h.D, h.L, out, s);
    return rubiconv::launch_direct(mode, h.direct_max, a_dtype, a, b_dtype, b, taps, plan->direct_segs, n, h.N,
                                   h.D, h.L, out_dtype, out, s);
}

// The filter's per-pair range scales inside a spectrum buffer (unit scales on fp32 grids).
const float2* filter_scales(const rubiconv_plan_s* plan, const void* spectrum) {
    if (!plan->h.grid_half) return plan->ones;
    return reinterpret_cast<const float2*>(static_cast<const char*>(spectrum) + plan->sscale_off);
}

// The two prescale words (x, dy) and the amax partials of a workspace header.
float2* prescale_words(void* workspace, size_t hdr_off) {
    return reinterpret_cast<float2*>(static_cast<char*>(workspace) + hdr_off);
}
uint32_t* prescale_work(void* workspace, size_t hdr_off) {
    return reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + hdr_off + kAlign);
}

// Prescale word of a [B][N][D] tensor (fp16 grids only; unit otherwise).
hipError_t prescale(rubiconv_plan_s* plan, int dtype, const void* in, float extra, const float2* prev,
                    float2* word, uint32_t* work, hipStream_t stream) {
    const HostPlan& h = plan->h;
    return rubiconv::launch_prescale(dtype, in, static_cast<int64_t>(h.B) * h.N * h.D, extra, prev, word,
                                     work, stream);
}

// Stage names in the profile: the forward's plain, the gradients' prefixed.
std::string stage(const char* tag, const char* name) { return std::string(tag) + name; }

// The data passes shared by the convolution and its gradients: column DFTs of `in`
// (dtype in_dtype, [B][N][D]) into `grid`; the row stage against the second grid
// `fgrid`, whose rows for each document are located by the spec_off of the segment
// table `t` (the filter class grids, or a document grid of the same plan); the
// product with F(f) (corr = 0) or F(-f) (corr = 1); the inverse passes into `out`
// (dtype out_dtype).  own_rows: every document's second grid rows are its own (the
// filter gradient), so the matrix-core row pass takes one document per task instead
// of groups of a size class.  The caller holds the plan's launch mutex.
// spec (matrix-core column pass, bf16 input only): the column pass runs at the guessed scale
// while recording |in|'s largest value per workgroup (four tasks) into spec->parts; a second
// launch takes the exact power-of-two scale from them, writes it to spec->used and redoes
// the pass at that scale only when it differs from the guess.
struct SpecScale {
    uint16_t* parts;
    float2* used;
    float guess;                  // the first pass's scale (a power of two)
    float* hint;                  // host-mapped word that receives the exact scale
    float extra = 1.0f;           // power of two the scale carries besides 2^(3 - e)
    const float2* prev = nullptr; // a scale word whose inverse the used word's inverse carries
};

// The hint word of a kind of call (rubiconv_plan_s::kHint*) and input buffer.
int hint_slot(int kind, const void* input) {
    const uint64_t a = reinterpret_cast<uintptr_t>(input) >> 8;
    return kind * rubiconv_plan_s::kHintSlots +
           static_cast<int>((a * 0x9E3779B97F4A7C15ull) >> 58);  // top 6 bits: 64 slots
}

// The scale a call's first column pass starts at: the last one its plan found for the
// slot (a power of two in the range pow2_scale gives, else 1).
float scale_guess(const rubiconv_plan_s* plan, int slot) {
    const float g = reinterpret_cast<const volatile float*>(plan->scale_hint)[slot];
    return g >= 0x1p-126f && g <= 0x1p127f ? g : 1.0f;
}

// The forward column pass of `in` into `grid` (and the long rows' first level); with
// spec, at a guessed scale, then the redo launch (SpecScale).
hipError_t enqueue_col_fwd(rubiconv_plan_s* plan, const void* in, int in_dtype, void* grid, GridScale in_sc,
                           hipStream_t stream, const SpecScale* spec) {
    const HostPlan& h = plan->h;
    const int n_cols = static_cast<int>(h.doc_col_seg.size());
    const int64_t rs = static_cast<int64_t>(h.N) * h.D;
    const bool half = h.grid_half;
    const bool mfma = h.col_mfma && in_dtype == RUBICONV_BF16;
    if (spec != nullptr && !mfma) return hipErrorInvalidValue;
    hipError_t e = mfma ? rubiconv::launch_col_fwd_mfma(in_dtype, in, rs, h.D, grid, plan->grid_pb_stride,
                                                        plan->doc_t, in_sc, plan->mfma_tab, n_cols, h.npb,
                                                        stream, spec ? spec->parts : nullptr, nullptr, nullptr,
                                                        spec ? spec->guess : 1.0f)
                        : rubiconv::launch_col_fwd(h.r, half, in_dtype, in, rs, h.D, grid,
                                                   plan->grid_pb_stride, plan->doc_t, in_sc, n_cols,
                                                   h.npb, stream);
    if (spec != nullptr && n_cols > 0 && e == hipSuccess)
        e = rubiconv::launch_col_fwd_mfma(in_dtype, in, rs, h.D, grid, plan->grid_pb_stride, plan->doc_t, in_sc,
                                          plan->mfma_tab, n_cols, h.npb, stream, nullptr, spec->parts, spec->used,
                                          spec->guess, spec->hint, spec->extra, spec->prev);
    // long rows: first level into the sub-row regions (both grids of the filter gradient)
    for (const rubiconv::LrItem& it : h.lr_doc_items)
        if (e == hipSuccess)
            e = rubiconv::launch_lr_step(false, grid, plan->grid_pb_stride, it, plan->doc_t.tw, h.n1,
                                         h.npb, stream);
    return e;
}

// The row stage on `grid` against the second grid `fgrid` (a filter spectrum, or x's grid
// for the filter gradient: own_rows, the sum groups), then the long rows' inverse first
// level.  dscale and out2 apply to the sum groups (launch_row_dense).
// `after`: an event just recorded on `stream` (a stage-timing mark), which the side
// streams then wait on in place of a fork event of their own (one marker less).
hipError_t enqueue_rows(rubiconv_plan_s* plan, const void* fgrid, int64_t fgrid_pb_stride, const LaunchTables& t,
                        void* grid, int corr, bool own_rows, hipStream_t stream, hipEvent_t after = nullptr,
                        float dscale = 1.0f, bool out2 = false) {
    const HostPlan& h = plan->h;
    const bool half = h.grid_half;
    hipError_t e = hipSuccess;
    // row pass: the generic kernel (long rows) and one launch per listed size
    // class, spread over the side streams (largest work first, least-loaded stream)
    struct Launch {
        int cls;       // -1: generic kernel; >= 0: register-resident kernel of that class
        int nb;        // > 0: matrix-core kernel for the documents of that block count
        double work;
        bool batch;    // the batched matrix-core kernel (rows of at most kMaxBatchM points)
        int lr = -1;   // >= 0: sub-row documents of long-row class launch lr
    };
    std::vector<Launch> launches;
    if (!h.doc_task_seg.empty()) launches.push_back({-1, 0, 1e30, false});
    for (size_t c = 0; c < h.classes.size(); ++c) {
        const int m = h.classes[c].m;
        if (m > rubiconv::kMaxFastM || (h.row_dense && m <= 16 * rubiconv::kMaxDenseBlocks)) continue;
        launches.push_back({static_cast<int>(c), 0, static_cast<double>(m) * h.classes[c].nlist, false});
    }
    // own_rows (the filter gradient): the sum groups, every matrix-core row size included
    if (h.row_dense)
        for (int nb = 1; nb <= rubiconv::kMaxDenseBlocks; ++nb) {
            if (h.dense_count[nb] == 0) continue;
            double w = 0;
            for (int k = 0; k < h.dense_count[nb]; ++k) w += h.docs[h.dense_docs[h.dense_list0[nb] + k]].m;
            if (nb == 1 && !own_rows) w -= h.dense_bwork;
            if ((own_rows ? h.dense_sgrp_n[nb] : h.dense_grp_n[nb]) > 0) launches.push_back({-1, nb, w, false});
        }
    if (h.row_dense && h.dense_bgrp_n > 0 && !own_rows) launches.push_back({-1, 1, h.dense_bwork, true});
    for (size_t k = 0; k < h.lr_launches.size(); ++k)
        launches.push_back({-1, h.lr_launches[k].nb, h.lr_launches[k].work, false, static_cast<int>(k)});
    std::sort(launches.begin(), launches.end(),
              [](const Launch& a, const Launch& b) { return a.work > b.work; });
    // the largest launch runs on the calling stream itself, the others on side streams
    const int nside = std::min<int>(rubiconv_plan_s::kSideStreams, static_cast<int>(launches.size()) - 1);
    auto launch_one = [&](const Launch& L, hipStream_t s) -> hipError_t {
        if (L.lr >= 0) {
            const HostPlan::LrLaunch& R = h.lr_launches[L.lr];
            return rubiconv::launch_row_dense(
                R.nb, grid, plan->grid_pb_stride, fgrid, fgrid_pb_stride, own_rows ? plan->lr_gsegs : plan->lr_segs,
                plan->lr_idx, plan->lr_groups + 2 * (own_rows ? R.dgrp0 : R.grp0), own_rows ? R.dgrp_n : R.grp_n,
                plan->dense_tab, h.n1 * R.m1, h.npb, corr, s);
        }
        if (L.batch)
            return rubiconv::launch_row_batch(grid, plan->grid_pb_stride, fgrid, fgrid_pb_stride, t.segs,
                                              plan->dense_docs, plan->dense_groups + 2 * h.dense_bgrp0,
                                              h.dense_bgrp_n, plan->dense_tab, h.n1, h.npb, corr, s);
        if (L.nb > 0 && own_rows)
            return rubiconv::launch_row_dense(
                L.nb, grid, plan->grid_pb_stride, fgrid, fgrid_pb_stride, t.segs, plan->dense_sdocs,
                plan->dense_sgroups + 2 * h.dense_sgrp0[L.nb], h.dense_sgrp_n[L.nb], plan->dense_tab, h.n1,
                h.npb, corr, s, true, dscale, out2);
        if (L.nb > 0)
            return rubiconv::launch_row_dense(
                L.nb, grid, plan->grid_pb_stride, fgrid, fgrid_pb_stride, t.segs, plan->dense_docs,
                plan->dense_groups + 2 * h.dense_grp0[L.nb], h.dense_grp_n[L.nb], plan->dense_tab, h.n1, h.npb,
                corr, s);
        if (L.cls < 0)
            return rubiconv::launch_row_conv(h.n1, half, grid, plan->grid_pb_stride, fgrid,
                                             fgrid_pb_stride, t,
                                             static_cast<int>(h.doc_task_seg.size()), h.npb,
                                             h.row_lds_docs, corr, s);
        const Seg& cs = h.classes[L.cls];
        return rubiconv::launch_row_fast(cs.m, half, grid, plan->grid_pb_stride, fgrid,
                                         fgrid_pb_stride, t.segs, plan->doc_t.list + cs.list0,
                                         cs.nlist, plan->doc_t.tw, h.n1, h.npb, corr, s);
    };
    if (nside < 1) {
        for (const Launch& L : launches)
            if (e == hipSuccess) e = launch_one(L, stream);
    } else if (e == hipSuccess) {
        hipEvent_t fork = after;
        if (fork == nullptr) {
            fork = plan->fork;
            e = hipEventRecord(fork, stream);
        }
        for (int k = 0; k < nside && e == hipSuccess; ++k) e = hipStreamWaitEvent(plan->side[k], fork, 0);
        std::vector<double> load(nside, 0.0);
        for (size_t i = 1; i < launches.size() && e == hipSuccess; ++i) {
            const Launch& L = launches[i];
            const int k = static_cast<int>(std::min_element(load.begin(), load.end()) - load.begin());
            load[k] += L.work;
            e = launch_one(L, plan->side[k]);
        }
        if (e == hipSuccess) e = launch_one(launches[0], stream);
        for (int k = 0; k < nside && e == hipSuccess; ++k) {
            e = hipEventRecord(plan->join[k], plan->side[k]);
            if (e == hipSuccess) e = hipStreamWaitEvent(stream, plan->join[k], 0);
        }
    }
    for (const rubiconv::LrItem& it : h.lr_doc_items)
        if (e == hipSuccess)
            e = rubiconv::launch_lr_step(true, grid, plan->grid_pb_stride, it, plan->doc_t.tw, h.n1,
                                         h.npb, stream);
    return e;
}

// The inverse column pass of `grid` into `out`.  own_rows (the filter gradient): its output
// documents only, the sum groups' followers having added their products to their
// leaders' rows.
hipError_t enqueue_col_inv(rubiconv_plan_s* plan, const void* grid, void* out, int out_dtype, bool own_rows,
                           GridScale out_sc, hipStream_t stream) {
    const HostPlan& h = plan->h;
    const int64_t rs = static_cast<int64_t>(h.N) * h.D;
    const LaunchTables& inv_t = own_rows ? plan->dk_t : plan->doc_t;
    const int inv_cols = own_rows ? static_cast<int>(h.dk_col_seg.size()) : static_cast<int>(h.doc_col_seg.size());
    return h.col_mfma ? rubiconv::launch_col_inv_mfma(out_dtype, grid, plan->grid_pb_stride, out, rs, h.D, inv_t,
                                                      out_sc, plan->mfma_tab, inv_cols, h.npb, stream)
                      : rubiconv::launch_col_inv(h.r, h.grid_half, out_dtype, grid, plan->grid_pb_stride, out, rs,
                                                 h.D, inv_t, out_sc, inv_cols, h.npb, stream);
}

hipError_t enqueue_conv(rubiconv_plan_s* plan, const void* in, int in_dtype, const void* fgrid,
                        int64_t fgrid_pb_stride, const LaunchTables& t, void* out, int out_dtype,
                        void* grid, int corr, bool own_rows, GridScale in_sc, GridScale out_sc,
                        const char* tag, hipStream_t stream, StageRecorder& rec,
                        const SpecScale* spec = nullptr) {
    hipError_t e = enqueue_col_fwd(plan, in, in_dtype, grid, in_sc, stream, spec);
    const hipEvent_t col_done = rec.mark(stage(tag, "col_fwd"));
    if (e == hipSuccess) e = enqueue_rows(plan, fgrid, fgrid_pb_stride, t, grid, corr, own_rows, stream, col_done);
    rec.mark(stage(tag, "row_conv"));
    if (e == hipSuccess) e = enqueue_col_inv(plan, grid, out, out_dtype, own_rows, out_sc, stream);
    rec.mark(stage(tag, "col_inv"));
    return e;
}

// The fused backward shares dy's column pass between dx and dk when every transform
// document takes the matrix-core passes on bf16 x and dy: no long rows and no VALU row
// launches, so that the filter gradient's row stage is the sum groups alone.
bool backward_fusable(const HostPlan& h) {
    if (!(h.grid_half && h.col_mfma && h.row_dense && h.x_dtype == RUBICONV_BF16 && h.y_dtype == RUBICONV_BF16))
        return false;
    if (!h.lr_doc_items.empty() || !h.doc_task_seg.empty()) return false;
    for (const Seg& c : h.classes)
        if (c.m > 16 * rubiconv::kMaxDenseBlocks) return false;
    return true;
}

}  // namespace

extern "C" {

rubiconv_status_t rubiconv_plan(rubiconv_plan_t* out, int B, int N, int D, int L, int max_docs,
                                const int32_t* cu_seqlens_host, rubiconv_dtype_t x_dtype,
                                rubiconv_dtype_t y_dtype, int n1, hipStream_t stream) {
    if (!out) return RUBICONV_ERR_ARG;
    *out = nullptr;
    rubiconv_plan_s* pl = new (std::nothrow) rubiconv_plan_s();
    if (!pl) return RUBICONV_ERR_ALLOC;
    // The direct path runs on the matrix cores where it can (bf16 x and dy, D a multiple of
    // 32; RUBICONV_DIRECT_MFMA = 0 keeps it on the VALU kernel), for documents of up to
    // kMaxDirectMfma tokens, else kDefaultDirect; RUBICONV_DIRECT_MAX (0 .. kMaxDirect, or
    // kMaxDirectMfma on the matrix cores) overrides that limit
    bool direct_mfma = true;
    if (const char* v = std::getenv("RUBICONV_DIRECT_MFMA")) {
        if (std::strcmp(v, "0") != 0 && std::strcmp(v, "1") != 0) {
            delete pl;
            return RUBICONV_ERR_ARG;
        }
        direct_mfma = v[0] == '1';
    }
    int direct_max = direct_mfma && rubiconv::direct_mfma_possible(x_dtype, y_dtype, D) ? rubiconv::kMaxDirectMfma
                                                                                      : rubiconv::kDefaultDirect;
    bool direct_by_share = true;  // an explicit limit applies as given
    if (const char* v = std::getenv("RUBICONV_DIRECT_MAX")) {
        direct_by_share = false;
        char* end = nullptr;
        const long n = std::strtol(v, &end, 10);
        if (end == v || *end != '\0' || n < 0 || n > rubiconv::kMaxDirectMfma) {
            delete pl;
            return RUBICONV_ERR_ARG;
        }
        direct_max = static_cast<int>(n);
    }
    // RUBICONV_CLASS_MERGE = 0 keeps every document at its own smallest row size
    bool merge = true;
    if (const char* v = std::getenv("RUBICONV_CLASS_MERGE")) {
        if (std::strcmp(v, "0") != 0 && std::strcmp(v, "1") != 0) {
            delete pl;
            return RUBICONV_ERR_ARG;
        }
        merge = v[0] == '1';
    }
    BuildError be = rubiconv::build_host_plan(&pl->h, B, N, D, L, max_docs, cu_seqlens_host,
                                              static_cast<int>(x_dtype), static_cast<int>(y_dtype),
                                              n1, direct_max, direct_by_share, merge, direct_mfma);
    if (be != BuildError::kOk) {
        delete pl;
        if (be == BuildError::kArg) return RUBICONV_ERR_ARG;
        if (be == BuildError::kSeqlens) return RUBICONV_ERR_SEQLENS;
        return RUBICONV_ERR_UNSUPPORTED;
    }
    const HostPlan& h = pl->h;
    // the grids hold the documents' (classes') points, then the sub-row regions of long rows
    pl->grid_pb_stride = (h.grid_points + h.grid_points_lr) * kPairsPerBlock;
    pl->cls_pb_stride = (h.class_points + h.class_points_lr) * kPairsPerBlock;
    const size_t esz = h.grid_half ? 4 : 8;  // complex fp16 / complex fp32 grid element
    pl->spec_bytes = align_up(static_cast<size_t>(h.npb) * pl->cls_pb_stride * esz);
    pl->dtaps_off = pl->spec_bytes;
    pl->spec_bytes += align_up(static_cast<size_t>(h.direct_taps) * h.D * 4);
    pl->sscale_off = pl->spec_bytes;
    pl->spec_bytes += align_up(static_cast<size_t>(std::max(h.npb, 1)) * kPairsPerBlock * sizeof(float2));
    pl->taps_bytes = align_up(static_cast<size_t>(h.taps_max) * h.D * 4);
    pl->partials_off = pl->taps_bytes;
    const size_t conv_ws = align_up(static_cast<size_t>(h.npb) * pl->grid_pb_stride * esz);
    const size_t filt_ws =
        pl->taps_bytes + align_up(static_cast<size_t>(rubiconv::tap_tile_rows(std::max(h.taps_max, 1))) * h.D * 4);
    // header: the scale words in the first kAlign bytes, then the amax
    // partials: kAmaxParts of the prescale pass, or one 16-bit word per workgroup of the
    // first forward column pass (four column tasks)
    const size_t n_tasks = h.doc_col_seg.size() * static_cast<size_t>(h.npb);
    // (dk keeps two sets of 16-bit magnitudes there, the second 16-byte aligned)
    const size_t hdr_bytes = kAlign + align_up(std::max<size_t>(rubiconv::kAmaxParts, n_tasks + 8) * 4);
    pl->ws_hdr_off = std::max(conv_ws, filt_ws);
    pl->ws_bytes = pl->ws_hdr_off + hdr_bytes;
    pl->grid_bytes = conv_ws;
    pl->dk_hdr_off = 2 * conv_ws + align_up(static_cast<size_t>(h.B) * h.N * h.D * 4);
    // (at least the convolution's: the fused backward may run dx and dk in sequence in it)
    pl->dk_ws_bytes = std::max(pl->dk_hdr_off + hdr_bytes, pl->ws_bytes);
    pl->spec_bytes = std::max(pl->spec_bytes, kAlign);
    // RUBICONV_PRESCALE = 0: the forward takes x as it is, without the power-of-two
    // scale from its largest magnitude (which costs one extra read of x); the gradients
    // always prescale dy (and x)
    if (const char* v = std::getenv("RUBICONV_PRESCALE")) {
        if (std::strcmp(v, "0") != 0 && std::strcmp(v, "1") != 0) {
            delete pl;
            return RUBICONV_ERR_ARG;
        }
        pl->prescale_fwd = v[0] == '1';
    }
    rubiconv_status_t st = upload(pl, stream);
    if (st != RUBICONV_OK) {
        if (pl->uploaded) {
            (void)hipEventSynchronize(pl->uploaded);
            (void)hipEventDestroy(pl->uploaded);
        }
        destroy_side_streams(pl);
        if (pl->dev) (void)hipFree(pl->dev);
        delete pl;
        return st;
    }
    *out = pl;
    return RUBICONV_OK;
}

void rubiconv_plan_destroy(rubiconv_plan_t plan) {
    if (!plan) return;
    if (plan->uploaded) {  // the upload reads the plan's host image until it completes
        (void)hipEventSynchronize(plan->uploaded);
        (void)hipEventDestroy(plan->uploaded);
    }
    destroy_events(plan);
    destroy_side_streams(plan);
    if (plan->scale_hint) (void)hipHostFree(plan->scale_hint);
    if (plan->dev) (void)hipFree(plan->dev);
    delete plan;
}

size_t rubiconv_spectrum_bytes(rubiconv_plan_t plan) { return plan ? plan->spec_bytes : 0; }

size_t rubiconv_workspace_bytes(rubiconv_plan_t plan) { return plan ? plan->ws_bytes : 0; }

rubiconv_status_t rubiconv_filter_spectrum(rubiconv_plan_t plan, const float* filters,
                                           void* spectrum, void* workspace, hipStream_t stream) {
    if (!plan || !filters || !spectrum || !workspace) return RUBICONV_ERR_ARG;
    if (!aligned(spectrum) || !aligned(workspace) || (reinterpret_cast<uintptr_t>(filters) % 4))
        return RUBICONV_ERR_ARG;
    if (!plan->device_ready) return RUBICONV_ERR_HIP;
    const HostPlan& h = plan->h;
    // taps as [taps_max][D] fp32, or as [taps_max][D / 2] fp16 channel pairs for the
    // matrix-core column pass (which computes in fp16)
    float* taps = static_cast<float*>(workspace);
    StageRecorder rec(plan, stream);
    // On fp16 grids the transpose also sums |k| per channel and tile of taps, and the
    // filter's range scale per channel pair follows from those sums: the column pass
    // normalises each pair's gain (sum of |k|) to 2^kFilterGainExp before fp16 rounding,
    // and the inverse column pass of every later call undoes it.
    float* partials = h.grid_half ? reinterpret_cast<float*>(static_cast<char*>(workspace) + plan->partials_off)
                                  : nullptr;
    float2* sscale = const_cast<float2*>(filter_scales(plan, spectrum));
    int ntiles = (h.taps_max + 31) / 32;
    hipError_t e = h.col_mfma
                       ? rubiconv::launch_transpose_pairs(filters, h.D, h.taps_max, h.L, taps, partials,
                                                          &ntiles, stream)
                       : rubiconv::launch_transpose(filters, h.D, h.taps_max, h.L, taps, h.D, partials,
                                                    stream);
    if (e == hipSuccess && h.grid_half)
        e = rubiconv::launch_filter_scale(partials, ntiles, h.D, h.npb * kPairsPerBlock, sscale, stream);
    rec.mark("filter_transpose");
    const rubiconv::GridScale fsc{sscale, plan->ones};
    if (e == hipSuccess)
        e = h.col_mfma
                ? rubiconv::launch_col_fwd_mfma(0, taps, 0, h.D, spectrum, plan->cls_pb_stride,
                                                plan->cls_t, fsc, plan->mfma_tab,
                                                static_cast<int>(h.cls_col_seg.size()), h.npb, stream)
                : rubiconv::launch_col_fwd(h.r, h.grid_half, 0, taps, 0, h.D, spectrum,
                                           plan->cls_pb_stride, plan->cls_t, fsc,
                                           static_cast<int>(h.cls_col_seg.size()), h.npb, stream);
    for (const rubiconv::LrItem& it : h.lr_cls_items)
        if (e == hipSuccess)
            e = rubiconv::launch_lr_step(false, spectrum, plan->cls_pb_stride, it, plan->doc_t.tw, h.n1,
                                         h.npb, stream);
    rec.mark("filter_col_fwd");
    if (e == hipSuccess && h.direct_taps > 0 && h.direct_mfma) {  // [D][T] bf16 hi, lo
        e = rubiconv::launch_split_taps(filters, h.D, h.direct_taps, h.L,
                                        reinterpret_cast<uint32_t*>(static_cast<char*>(spectrum) + plan->dtaps_off),
                                        stream);
        rec.mark("filter_direct_taps");
    } else if (e == hipSuccess && h.direct_taps > 0) {  // the direct path's taps, [T][D] fp32
        e = rubiconv::launch_transpose(filters, h.D, h.direct_taps, h.L,
                                       reinterpret_cast<float*>(static_cast<char*>(spectrum) + plan->dtaps_off),
                                       h.D, nullptr, stream);
        rec.mark("filter_direct_taps");
    }
    return e == hipSuccess ? RUBICONV_OK : RUBICONV_ERR_HIP;
}

rubiconv_status_t rubiconv_packed_conv(rubiconv_plan_t plan, const void* x, const void* spectrum,
                                       void* y, void* workspace, hipStream_t stream) {
    if (!plan || !x || !spectrum || !y || !workspace) return RUBICONV_ERR_ARG;
    if (!aligned(spectrum) || !aligned(workspace)) return RUBICONV_ERR_ARG;
    const size_t esz = plan->h.x_dtype == RUBICONV_F32 ? 4 : 2;
    const size_t ysz = plan->h.y_dtype == RUBICONV_F32 ? 4 : 2;
    if (reinterpret_cast<uintptr_t>(x) % esz || reinterpret_cast<uintptr_t>(y) % ysz || !direct_aligned(plan, {x, y}))
        return RUBICONV_ERR_ARG;
    if (!plan->device_ready) return RUBICONV_ERR_HIP;
    std::lock_guard<std::mutex> lock(plan->launch_mu);
    StageRecorder rec(plan, stream);
    const HostPlan& h = plan->h;
    const bool direct = !h.direct_docs.empty();
    hipError_t e = hipSuccess;
    if (direct)
        e = fork_direct(plan, stream, rec, "direct", [&](hipStream_t s) {
            return direct_sums(plan, 0, h.x_dtype, x, 0, nullptr, direct_taps(plan, spectrum), h.y_dtype, y, s);
        });
    // range scales: the filter's per pair, and x's power-of-two prescale when asked for.
    // On the matrix-core path the column pass first runs at the scale the plan's last
    // call found and records |x|'s largest value; it runs again only when that value asks
    // for another scale, which saves a read of x whenever x's range holds from call to call.
    const float2* xs = plan->ones;
    float2* w = prescale_words(workspace, plan->ws_hdr_off);
    const int slot = hint_slot(rubiconv_plan_s::kHintFwd, x);
    SpecScale spec{reinterpret_cast<uint16_t*>(prescale_work(workspace, plan->ws_hdr_off)), w,
                   scale_guess(plan, slot), plan->scale_hint_dev + slot};
    const bool speculative = h.grid_half && plan->prescale_fwd && h.col_mfma && h.x_dtype == RUBICONV_BF16;
    if (e == hipSuccess && h.grid_half && plan->prescale_fwd && !speculative) {
        e = prescale(plan, h.x_dtype, x, 1.0f, nullptr, w, prescale_work(workspace, plan->ws_hdr_off), stream);
        rec.mark("prescale");
        xs = w;
    }
    if (e == hipSuccess)
        e = enqueue_conv(plan, x, h.x_dtype, spectrum, plan->cls_pb_stride, plan->doc_t, y, h.y_dtype,
                         workspace, 0, false, {plan->ones, xs}, {filter_scales(plan, spectrum), speculative ? w : xs},
                         "", stream, rec, speculative ? &spec : nullptr);
    if (e == hipSuccess && direct) e = join_direct(plan, stream, rec);
    return e == hipSuccess ? RUBICONV_OK : RUBICONV_ERR_HIP;
}

rubiconv_status_t rubiconv_packed_conv_dx(rubiconv_plan_t plan, const void* dy, const void* spectrum,
                                          void* dx, void* workspace, hipStream_t stream) {
    if (!plan || !dy || !spectrum || !dx || !workspace) return RUBICONV_ERR_ARG;
    if (!aligned(spectrum) || !aligned(workspace)) return RUBICONV_ERR_ARG;
    const size_t xsz = plan->h.x_dtype == RUBICONV_F32 ? 4 : 2;
    const size_t ysz = plan->h.y_dtype == RUBICONV_F32 ? 4 : 2;
    if (reinterpret_cast<uintptr_t>(dy) % ysz || reinterpret_cast<uintptr_t>(dx) % xsz ||
        !direct_aligned(plan, {dy, dx}))
        return RUBICONV_ERR_ARG;
    if (!plan->device_ready) return RUBICONV_ERR_HIP;
    std::lock_guard<std::mutex> lock(plan->launch_mu);
    StageRecorder rec(plan, stream);
    // dy has y's dtype and dx has x's: the correlation runs the convolution's passes
    // with the roles of the two dtypes exchanged
    const HostPlan& h = plan->h;
    const bool direct = !h.direct_docs.empty();
    hipError_t e = hipSuccess;
    if (direct)
        e = fork_direct(plan, stream, rec, "dx_direct", [&](hipStream_t s) {
            return direct_sums(plan, 1, h.y_dtype, dy, 0, nullptr, direct_taps(plan, spectrum), h.x_dtype, dx, s);
        });
    // dy is prescaled by a power of two from its largest magnitude (upstream gradients are
    // often far below 1), the filter by its per-pair scale.  On the matrix-core path the
    // column pass starts at the scale of the plan's last dx call and is redone only when
    // dy's own scale differs (as in the forward).
    const float2* ds = plan->ones;
    float2* w = prescale_words(workspace, plan->ws_hdr_off) + 1;
    const int slot = hint_slot(rubiconv_plan_s::kHintDx, dy);
    SpecScale spec{reinterpret_cast<uint16_t*>(prescale_work(workspace, plan->ws_hdr_off)), w,
                   scale_guess(plan, slot), plan->scale_hint_dev + slot};
    const bool speculative = h.grid_half && h.col_mfma && h.y_dtype == RUBICONV_BF16;
    if (e == hipSuccess && h.grid_half && !speculative) {
        e = prescale(plan, h.y_dtype, dy, 1.0f, nullptr, w, prescale_work(workspace, plan->ws_hdr_off), stream);
        rec.mark("dx_prescale");
        ds = w;
    }
    if (e == hipSuccess)
        e = enqueue_conv(plan, dy, h.y_dtype, spectrum, plan->cls_pb_stride, plan->doc_t, dx,
                         h.x_dtype, workspace, 1, false, {plan->ones, ds},
                         {filter_scales(plan, spectrum), speculative ? w : ds}, "dx_", stream, rec,
                         speculative ? &spec : nullptr);
    if (e == hipSuccess && direct) e = join_direct(plan, stream, rec);
    return e == hipSuccess ? RUBICONV_OK : RUBICONV_ERR_HIP;
}

size_t rubiconv_dk_workspace_bytes(rubiconv_plan_t plan) { return plan ? plan->dk_ws_bytes : 0; }

rubiconv_status_t rubiconv_packed_conv_dk(rubiconv_plan_t plan, const void* x, const void* dy,
                                          float* dk, void* workspace, hipStream_t stream) {
    if (!plan || !x || !dy || !dk || !workspace) return RUBICONV_ERR_ARG;
    if (!aligned(workspace)) return RUBICONV_ERR_ARG;
    const HostPlan& h = plan->h;
    const size_t xsz = h.x_dtype == RUBICONV_F32 ? 4 : 2;
    const size_t ysz = h.y_dtype == RUBICONV_F32 ? 4 : 2;
    if (reinterpret_cast<uintptr_t>(x) % xsz || reinterpret_cast<uintptr_t>(dy) % ysz ||
        reinterpret_cast<uintptr_t>(dk) % 4 || !direct_aligned(plan, {x, dy}))
        return RUBICONV_ERR_ARG;
    // the x grid doubles as the "filter" grid: its offsets must fit the 32-bit field
    if (h.grid_points + h.grid_points_lr > INT32_MAX) return RUBICONV_ERR_UNSUPPORTED;
    if (!plan->device_ready) return RUBICONV_ERR_HIP;
    std::lock_guard<std::mutex> lock(plan->launch_mu);
    StageRecorder rec(plan, stream);
    char* ws = static_cast<char*>(workspace);
    void* xgrid = ws + plan->grid_bytes;
    float* r = reinterpret_cast<float*>(ws + 2 * plan->grid_bytes);
    const int n_cols = static_cast<int>(h.doc_col_seg.size());
    const int64_t rs = static_cast<int64_t>(h.N) * h.D;
    // direct documents: their correlations straight into r, beside the transforms
    const bool direct = !h.direct_docs.empty();
    hipError_t e = hipSuccess;
    if (direct)
        e = fork_direct(plan, stream, rec, "dk_direct", [&](hipStream_t s) {
            return direct_sums(plan, 2, h.y_dtype, dy, h.x_dtype, x, nullptr, 0, r, s);
        });
    // range: x and dy prescaled by powers of two from their largest magnitudes, and
    // together by 2^-ceil(log2 P_max) (half on each side), as a correlation sums up to P
    // products; the inverse pass undoes all of it (the dy word's second half)
    // On the matrix-core path both column passes find their scales themselves, starting
    // from the ones the plan's previous dk call found (as the forward does for x).
    const float2* xs = plan->ones;
    const float2* ds = plan->ones;
    float2* w = prescale_words(workspace, plan->dk_hdr_off);
    uint32_t* work = prescale_work(workspace, plan->dk_hdr_off);
    float ex, ed;
    dk_split(h, &ex, &ed);
    const bool speculative = h.grid_half && h.col_mfma && h.x_dtype == RUBICONV_BF16 && h.y_dtype == RUBICONV_BF16;
    // per-task magnitudes: x's in the first half of the partials area, dy's in the second
    uint16_t* parts = reinterpret_cast<uint16_t*>(work);
    const size_t n_tasks = static_cast<size_t>(n_cols) * h.npb;
    const int slot_x = hint_slot(rubiconv_plan_s::kHintDkX, x);
    const int slot_dy = hint_slot(rubiconv_plan_s::kHintDkDy, dy);
    SpecScale spec_x{parts, w, scale_guess(plan, slot_x), plan->scale_hint_dev + slot_x, ex, nullptr};
    SpecScale spec_dy{parts + (n_tasks + 7) / 8 * 8, w + 1, scale_guess(plan, slot_dy),
                      plan->scale_hint_dev + slot_dy, ed, w};
    if (e == hipSuccess && h.grid_half && !speculative) {
        e = prescale(plan, h.x_dtype, x, ex, nullptr, w, work, stream);
        if (e == hipSuccess)
            e = prescale(plan, h.y_dtype, dy, ed, w, w + 1, work, stream);
        rec.mark("dk_prescale");
    }
    if (h.grid_half) {
        xs = w;
        ds = w + 1;
    }
    // x's column DFTs into the second grid, then dy's passes against it with the
    // correlation product: document i's cross-correlation of dy with x lands at its
    // own token positions (lag = offset in the document) of r
    if (e == hipSuccess && speculative) {
        e = rubiconv::launch_col_fwd_mfma(h.x_dtype, x, rs, h.D, xgrid, plan->grid_pb_stride, plan->doc_t,
                                          {plan->ones, xs}, plan->mfma_tab, n_cols, h.npb, stream, spec_x.parts,
                                          nullptr, nullptr, spec_x.guess);
        if (e == hipSuccess && n_cols > 0)
            e = rubiconv::launch_col_fwd_mfma(h.x_dtype, x, rs, h.D, xgrid, plan->grid_pb_stride, plan->doc_t,
                                              {plan->ones, xs}, plan->mfma_tab, n_cols, h.npb, stream, nullptr,
                                              spec_x.parts, spec_x.used, spec_x.guess, spec_x.hint, spec_x.extra,
                                              spec_x.prev);
    } else if (e == hipSuccess) {
        e = h.col_mfma && h.x_dtype == RUBICONV_BF16
                       ? rubiconv::launch_col_fwd_mfma(h.x_dtype, x, rs, h.D, xgrid,
                                                       plan->grid_pb_stride, plan->doc_t,
                                                       {plan->ones, xs}, plan->mfma_tab, n_cols,
                                                       h.npb, stream)
                       : rubiconv::launch_col_fwd(h.r, h.grid_half, h.x_dtype, x, rs, h.D, xgrid,
                                                  plan->grid_pb_stride, plan->doc_t, {plan->ones, xs},
                                                  n_cols, h.npb, stream);
    }
    for (const rubiconv::LrItem& it : h.lr_doc_items)
        if (e == hipSuccess)
            e = rubiconv::launch_lr_step(false, xgrid, plan->grid_pb_stride, it, plan->doc_t.tw, h.n1,
                                         h.npb, stream);
    rec.mark("dk_col_fwd_x");
    if (e == hipSuccess)
        e = enqueue_conv(plan, dy, h.y_dtype, xgrid, plan->grid_pb_stride, plan->grad_t, r,
                         RUBICONV_F32, workspace, 1, true, {plan->ones, ds}, {plan->ones, ds}, "dk_",
                         stream, rec, speculative ? &spec_dy : nullptr);
    if (e == hipSuccess && direct) e = join_direct(plan, stream, rec);
    if (e == hipSuccess)
        e = rubiconv::launch_lag_sum(r, plan->dk_sum_segs, static_cast<int>(h.dk_sum_segs.size()), h.N,
                                     h.D, h.L, dk, stream);
    rec.mark("dk_lag_sum");
    return e == hipSuccess ? RUBICONV_OK : RUBICONV_ERR_HIP;
}


rubiconv_status_t rubiconv_packed_conv_backward(rubiconv_plan_t plan, const void* x, const void* dy,
                                                const void* spectrum, void* dx, float* dk, void* workspace,
                                                hipStream_t stream) {
    if (!plan || !x || !dy || !spectrum || !dx || !dk || !workspace) return RUBICONV_ERR_ARG;
    if (!aligned(spectrum) || !aligned(workspace)) return RUBICONV_ERR_ARG;
    const HostPlan& h = plan->h;
    const size_t xsz = h.x_dtype == RUBICONV_F32 ? 4 : 2;
    const size_t ysz = h.y_dtype == RUBICONV_F32 ? 4 : 2;
    if (reinterpret_cast<uintptr_t>(x) % xsz || reinterpret_cast<uintptr_t>(dy) % ysz ||
        reinterpret_cast<uintptr_t>(dx) % xsz || reinterpret_cast<uintptr_t>(dk) % 4 ||
        !direct_aligned(plan, {x, dy, dx}))
        return RUBICONV_ERR_ARG;
    if (!plan->device_ready) return RUBICONV_ERR_HIP;
    if (!backward_fusable(h)) {
        rubiconv_status_t st = rubiconv_packed_conv_dx(plan, dy, spectrum, dx, workspace, stream);
        if (st == RUBICONV_OK) st = rubiconv_packed_conv_dk(plan, x, dy, dk, workspace, stream);
        return st;
    }
    // the x grid doubles as the "filter" grid: its offsets must fit the 32-bit field
    if (h.grid_points + h.grid_points_lr > INT32_MAX) return RUBICONV_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(plan->launch_mu);
    StageRecorder rec(plan, stream);
    char* ws = static_cast<char*>(workspace);
    void* dygrid = ws;
    void* xgrid = ws + plan->grid_bytes;
    float* r = reinterpret_cast<float*>(ws + 2 * plan->grid_bytes);
    const int n_cols = static_cast<int>(h.doc_col_seg.size());
    hipError_t e = hipSuccess;
    // direct documents: dx's and dk's sums, one after the other beside the transforms
    const bool direct = !h.direct_docs.empty();
    if (direct)
        e = fork_direct(plan, stream, rec, "bwd_direct", [&](hipStream_t s) {
            hipError_t de = direct_sums(plan, 1, h.y_dtype, dy, 0, nullptr, direct_taps(plan, spectrum), h.x_dtype,
                                        dx, s);
            if (de == hipSuccess) de = direct_sums(plan, 2, h.y_dtype, dy, h.x_dtype, x, nullptr, 0, r, s);
            return de;
        });
    // range: dy's grid carries dx's scale s_dy (its magnitude alone); x's carries s_x ex
    // (as in dk), and the sum-group kernels multiply dy's spectra by ed before the
    // products, so that dk's products sit where dk's own passes put them.  dy's word is
    // {s_dy, 1 / s_dy} (dx's inverse); x's inverse factor also carries 1 / s_dy, and the
    // per-pair words 1 / ed: dk's inverse undoes all of it.
    float ex, ed;
    dk_split(h, &ex, &ed);
    float2* w = prescale_words(workspace, plan->dk_hdr_off);
    uint16_t* parts = reinterpret_cast<uint16_t*>(prescale_work(workspace, plan->dk_hdr_off));
    const size_t n_tasks = static_cast<size_t>(n_cols) * h.npb;
    const int slot_dy = hint_slot(rubiconv_plan_s::kHintDx, dy);
    const int slot_x = hint_slot(rubiconv_plan_s::kHintDkX, x);
    const SpecScale spec_dy{parts + (n_tasks + 7) / 8 * 8, w + 1, scale_guess(plan, slot_dy),
                            plan->scale_hint_dev + slot_dy, 1.0f, nullptr};
    const SpecScale spec_x{parts, w, scale_guess(plan, slot_x), plan->scale_hint_dev + slot_x, ex, w + 1};
    if (e == hipSuccess) e = enqueue_col_fwd(plan, dy, h.y_dtype, dygrid, {plan->ones, w + 1}, stream, &spec_dy);
    rec.mark("bwd_col_fwd_dy");
    if (e == hipSuccess) e = enqueue_col_fwd(plan, x, h.x_dtype, xgrid, {plan->ones, w}, stream, &spec_x);
    const hipEvent_t cols_done = rec.mark("bwd_col_fwd_x");
    // dk: the sum groups against x's grid, their sums written over x's grid (dy's stays)
    if (e == hipSuccess)
        e = enqueue_rows(plan, xgrid, plan->grid_pb_stride, plan->grad_t, dygrid, 1, true, stream, cols_done, ed,
                         true);
    rec.mark("bwd_dk_row_conv");
    if (e == hipSuccess) e = enqueue_col_inv(plan, xgrid, r, RUBICONV_F32, true, {plan->dk_unscale, w}, stream);
    rec.mark("bwd_dk_col_inv");
    if (e == hipSuccess && direct) e = join_direct(plan, stream, rec);
    if (e == hipSuccess)
        e = rubiconv::launch_lag_sum(r, plan->dk_sum_segs, static_cast<int>(h.dk_sum_segs.size()), h.N,
                                     h.D, h.L, dk, stream);
    const hipEvent_t dk_done = rec.mark("bwd_dk_lag_sum");
    // dx: the correlation with the filter on dy's grid, in place
    if (e == hipSuccess)
        e = enqueue_rows(plan, spectrum, plan->cls_pb_stride, plan->doc_t, dygrid, 1, false, stream, dk_done);
    rec.mark("bwd_dx_row_conv");
    if (e == hipSuccess)
        e = enqueue_col_inv(plan, dygrid, dx, h.x_dtype, false, {filter_scales(plan, spectrum), w + 1}, stream);
    rec.mark("bwd_dx_col_inv");
    return e == hipSuccess ? RUBICONV_OK : RUBICONV_ERR_HIP;
}

rubiconv_status_t rubiconv_plan_info(rubiconv_plan_t plan, rubiconv_plan_info_t* info) {
    if (!plan || !info) return RUBICONV_ERR_ARG;
    const HostPlan& h = plan->h;
    info->B = h.B; info->N = h.N; info->D = h.D; info->L = h.L;
    info->n1 = h.n1;
    info->n_docs = static_cast<int>(h.all_docs.size());
    info->n_classes = static_cast<int>(h.classes.size());
    info->n_pair_blocks = h.npb;
    info->grid_points = h.grid_points;
    info->class_points = h.class_points;
    int64_t tok = 0;
    for (const Seg& s : h.all_docs) tok += s.len;
    info->tokens = tok;
    info->direct_max = h.direct_max;
    info->n_direct = static_cast<int>(h.direct_docs.size());
    return RUBICONV_OK;
}

rubiconv_status_t rubiconv_plan_doc_table(rubiconv_plan_t plan, int32_t* out, int cap,
                                          int* n_docs) {
    if (!plan || !n_docs || cap < 0 || (cap > 0 && !out)) return RUBICONV_ERR_ARG;
    const HostPlan& h = plan->h;
    const int n = static_cast<int>(h.all_docs.size());
    *n_docs = n;
    for (int i = 0; i < n && i < cap; ++i) {
        const Seg& s = h.all_docs[i];
        int32_t* o = out + 6 * static_cast<int64_t>(i);
        o[0] = s.row; o[1] = h.all_index[i]; o[2] = s.start; o[3] = s.len; o[4] = s.m; o[5] = s.P;
    }
    return RUBICONV_OK;
}

rubiconv_status_t rubiconv_profile_start(rubiconv_plan_t plan, int max_calls) {
    if (!plan || max_calls < 0) return RUBICONV_ERR_ARG;
    plan->prof_max = plan->prof_used = 0;
    plan->prof_names.clear();
    if (max_calls == 0) return RUBICONV_OK;
    if (!plan->device_ready) return RUBICONV_ERR_HIP;
    const size_t n = static_cast<size_t>(max_calls) * rubiconv_plan_s::kEventsPerCall;
    while (plan->prof_events.size() < n) {
        hipEvent_t ev;
        // timing only: no system-scope fence at each stage boundary
        if (hipEventCreateWithFlags(&ev, hipEventDisableSystemFence) != hipSuccess) return RUBICONV_ERR_ALLOC;
        plan->prof_events.push_back(ev);
    }
    plan->prof_names.assign(max_calls, {});
    plan->prof_max = max_calls;
    return RUBICONV_OK;
}

rubiconv_status_t rubiconv_profile_read(rubiconv_plan_t plan, rubiconv_kernel_time_t* out, int cap,
                                        int* n) {
    if (!plan || !n || cap < 0 || (cap > 0 && !out)) return RUBICONV_ERR_ARG;
    std::vector<rubiconv_kernel_time_t> acc;
    for (int slot = 0; slot < plan->prof_used; ++slot) {
        const auto& names = plan->prof_names[slot];
        hipEvent_t* ev = plan->prof_events.data() + slot * rubiconv_plan_s::kEventsPerCall;
        if (!names.empty() && hipEventSynchronize(ev[names.size()]) != hipSuccess)
            return RUBICONV_ERR_HIP;
        for (size_t k = 0; k < names.size(); ++k) {
            float ms = 0.0f;
            if (hipEventElapsedTime(&ms, ev[k], ev[k + 1]) != hipSuccess) return RUBICONV_ERR_HIP;
            auto it = std::find_if(acc.begin(), acc.end(), [&](const rubiconv_kernel_time_t& a) {
                return names[k].compare(0, sizeof(a.name) - 1, a.name) == 0;
            });
            if (it == acc.end()) {
                rubiconv_kernel_time_t t{};
                std::strncpy(t.name, names[k].c_str(), sizeof(t.name) - 1);
                acc.push_back(t);
                it = acc.end() - 1;
            }
            it->launches += 1;
            it->total_ms += ms;
        }
    }
    *n = static_cast<int>(acc.size());
    for (int i = 0; i < *n && i < cap; ++i) out[i] = acc[i];
    return RUBICONV_OK;
}

const char* rubiconv_status_string(rubiconv_status_t status) {
    switch (status) {
        case RUBICONV_OK: return "ok";
        case RUBICONV_ERR_ARG: return "invalid argument";
        case RUBICONV_ERR_SEQLENS: return "invalid cu_seqlens";
        case RUBICONV_ERR_UNSUPPORTED: return "unsupported configuration";
        case RUBICONV_ERR_ALLOC: return "allocation failed";
        case RUBICONV_ERR_HIP: return "HIP error or no device";
    }
    return "unknown status";
}

}  // extern "C"
