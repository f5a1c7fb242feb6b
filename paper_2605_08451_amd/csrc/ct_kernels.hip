// ct_kernels.hip -- the masked Cooley-Tukey convolution (Algorithm 2) on gfx950.
//
// Algorithm 2 runs the radix-2 decimation-in-time stages over the whole packed
// array and masks them: at stage s (butterflies of size m = 2^s) an element whose
// document is shorter than m keeps its value, every other element takes the
// standard butterfly at its position inside its own document.  Here the same
// stages run on a flat array holding the documents longest first (ct_plan.hpp), so
// every document starts at a multiple of its size and the standard twiddle of an
// element depends on its flat position alone; only the mask needs the document.
//
// Stages are fused three at a time in registers (a radix-8 group holds the 8
// elements that three consecutive radix-2 stages combine), and a workgroup keeps a
// tile of kTile points x kPairs channel pairs in LDS:
//   * short documents (P <= kTile): one kernel takes a tile of whole documents from
//     x through the forward stages, the spectral product, the inverse stages and
//     into y;
//   * long documents (P = kTile * M, M <= 2^(kMaxLogMid + kMaxLogCols)): the first
//     kLogTile stages run on each tile (front), for M > 64 the next log2 M - 6 stages
//     on tiles of the column view (middle pass), the last stages (at most 6) on the
//     columns l = c + S * j of a view of stride S (column pass, which also takes the
//     product), and the inverse repeats the split in reverse (column pass, middle
//     pass, then back).
// The inverse uses decimation-in-frequency stages (the same butterflies with the
// conjugate twiddles, in reverse order), which take the spectrum in natural order
// and leave the time samples in bit-reversed order: the forward transform's load
// and the inverse's store use the same bit-reversed positions, and no separate
// reordering pass is needed.  Channels d and d + 1 share one complex transform;
// the filter spectrum separates them (ct_kernels.hpp).
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "ct_kernels.hpp"
#include "fft_core.hpp"
#include "pk_half.hpp"

namespace rubiconv::ct {
namespace {

constexpr int kThreads = 256;
constexpr int kSlots = kThreads / kPairs;      // 16 element slots per channel-pair lane
constexpr int kTileGroups = kTile / 8;         // radix-8 groups of one tile
constexpr int kMaxCols = 1 << kMaxLogCols;
static_assert(kMaxCols <= kTile / 4, "a column work item needs at least one low column pair");
static_assert(kMaxLogMid < kLogTile, "a middle-pass tile needs at least one column");

__device__ __forceinline__ int bitrev(int v, int bits) {
    return bits == 0 ? 0 : static_cast<int>(__builtin_bitreverse32(static_cast<uint32_t>(v)) >> (32 - bits));
}

__device__ __forceinline__ float2 sel(bool c, float2 a, float2 b) {
    return make_float2(c ? a.x : b.x, c ? a.y : b.y);
}

__device__ __forceinline__ float2 mul_conj(float2 a, float2 b) {  // a * conj(b)
    return make_float2(a.x * b.x + a.y * b.y, a.y * b.x - a.x * b.y);
}

__device__ __forceinline__ Doc load_doc(const Doc* docs, int i) {
    const int4* p = reinterpret_cast<const int4*>(docs + i);
    const int4 a = p[0], b = p[1];
    return Doc{a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
}

// ---------------------------------------------------------------- element I/O
// Channel pair p of token `tok` of row `row` as one complex value (zero past D).
template <int TA>
__device__ __forceinline__ float2 load_pair(const void* a, int row, int tok, int N, int D, int p) {
    if (2 * p >= D) return make_float2(0.f, 0.f);
    const int64_t i = (static_cast<int64_t>(row) * N + tok) * D + 2 * p;
    if constexpr (TA == 0) {
        return *reinterpret_cast<const float2*>(static_cast<const float*>(a) + i);
    } else {
        const uint32_t u = *reinterpret_cast<const uint32_t*>(static_cast<const uint16_t*>(a) + i);
        return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
    }
}

template <int TO>
__device__ __forceinline__ void store_pair(void* o, int row, int tok, int N, int D, int p, float2 v) {
    if (2 * p >= D) return;
    const int64_t i = (static_cast<int64_t>(row) * N + tok) * D + 2 * p;
    if constexpr (TO == 0) {
        *reinterpret_cast<float2*>(static_cast<float*>(o) + i) = v;
    } else {
        *reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(o) + i) = bf2_bits(v.x, v.y);
    }
}

template <bool HALF>
__device__ __forceinline__ float2 grid_load(const void* g, int64_t i) {
    if constexpr (HALF) {
        const uint32_t u = static_cast<const uint32_t*>(g)[i];
        return __half22float2(__builtin_bit_cast(__half2, u));
    } else {
        return static_cast<const float2*>(g)[i];
    }
}

template <bool HALF>
__device__ __forceinline__ void grid_store(void* g, int64_t i, float2 v) {
    if constexpr (HALF) static_cast<uint32_t*>(g)[i] = h2_bits(v.x, v.y);
    else static_cast<float2*>(g)[i] = v;
}

// ---------------------------------------------------------------- stage groups
// A group holds the 2^K elements l_i = base + i * h0 (h0 = 2^(sigma0 - 1), b0 = base
// mod h0).  Stage sigma = sigma0 + k pairs elements i and i + 2^k (bit k of i clear)
// with the twiddle w_{2^sigma}^r, r = b0 + (i mod 2^k) * h0 (the element's position
// inside its butterfly).  on(i, sigma) is the element's mask: its document holds at
// least 2^sigma points.
template <int K, class Tw, class On>
__device__ __forceinline__ void dit_group(float2 (&v)[1 << K], int b0, int h0, int sigma0, Tw tw, On on) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int sigma = sigma0 + k;
#pragma unroll
        for (int i = 0; i < (1 << K); ++i) {
            if (i & (1 << k)) continue;
            const int j = i | (1 << k);
            const float2 t = cmul(tw(b0 + (i & ((1 << k) - 1)) * h0, sigma), v[j]);
            const bool a = on(i, sigma);
            const float2 top = cadd(v[i], t), bot = csub(v[i], t);
            v[i] = sel(a, top, v[i]);
            v[j] = sel(a, bot, v[j]);
        }
    }
}

// The inverse (decimation in frequency): stages sigma0 + K - 1 down to sigma0, each
// (a, b) -> (a + b, (a - b) conj(w)) with the same pairs and twiddles.
template <int K, class Tw, class On>
__device__ __forceinline__ void dif_group(float2 (&v)[1 << K], int b0, int h0, int sigma0, Tw tw, On on) {
#pragma unroll
    for (int k = K - 1; k >= 0; --k) {
        const int sigma = sigma0 + k;
#pragma unroll
        for (int i = 0; i < (1 << K); ++i) {
            if (i & (1 << k)) continue;
            const int j = i | (1 << k);
            const bool a = on(i, sigma);
            const float2 top = cadd(v[i], v[j]);
            const float2 bot = mul_conj(csub(v[i], v[j]), tw(b0 + (i & ((1 << k) - 1)) * h0, sigma));
            v[i] = sel(a, top, v[i]);
            v[j] = sel(a, bot, v[j]);
        }
    }
}

// Group g of a radix-8 pass with element stride h0 over a tile: base and b0.
__device__ __forceinline__ int group_base(int g, int lg_h0) {
    return (g & ((1 << lg_h0) - 1)) + ((g >> lg_h0) << (lg_h0 + 3));
}

struct TileTw {  // w_{2^sigma}^r for sigma <= kLogTile, from w_kTile^k in LDS
    const float2* s;
    __device__ float2 operator()(int r, int sigma) const { return s[r << (kLogTile - sigma)]; }
};

struct GlobalTw {  // w_{2^sigma}^r for sigma <= kMaxLogP
    const float2* g;
    __device__ float2 operator()(int r, int sigma) const { return g[r << (kMaxLogP - sigma)]; }
};

struct AllOn {
    __device__ bool operator()(int, int) const { return true; }
};

__device__ __forceinline__ void load_tile_twiddles(float2* s_tw, const float2* tw) {
    for (int k = threadIdx.x; k < kTile / 2; k += kThreads) s_tw[k] = tw[k << (kMaxLogP - kLogTile)];
}

// One radix-8 pass over the LDS tile (forward or inverse), stride 2^lg_h0.
template <bool INV>
__device__ __forceinline__ void tile_pass(float2 (*s_z)[kPairs], const uint8_t* s_lp, TileTw tw,
                                          int lg_h0, int q, int slot) {
    const int h0 = 1 << lg_h0;
    #pragma unroll
    for (int g = slot; g < kTileGroups; g += kSlots) {
        const int base = group_base(g, lg_h0);
        float2 v[8];
        int lp[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            v[i] = s_z[base + i * h0][q];
            lp[i] = s_lp ? s_lp[base + i * h0] : kMaxLogP;
        }
        auto on = [&](int i, int sigma) { return lp[i] >= sigma; };
        if constexpr (INV) dif_group<3>(v, base & (h0 - 1), h0, lg_h0 + 1, tw, on);
        else dit_group<3>(v, base & (h0 - 1), h0, lg_h0 + 1, tw, on);
#pragma unroll
        for (int i = 0; i < 8; ++i) s_z[base + i * h0][q] = v[i];
    }
}

// ---------------------------------------------------------------- short documents
// Spectrum entry e: (U, V) of one channel pair at one frequency, complex fp16 pairs
// (8 bytes) or complex fp32 (16 bytes).  The entries hold (H_d + H_{d+1}) / 2 and
// (H_d - H_{d+1}) / 2; the product applies the inverse transform's 1/P.
template <bool SH>
__device__ __forceinline__ void spec_load(const void* spec, int64_t e, float2& u, float2& v) {
    if constexpr (SH) {
        const uint2 w = static_cast<const uint2*>(spec)[e];
        u = __half22float2(__builtin_bit_cast(__half2, w.x));
        v = __half22float2(__builtin_bit_cast(__half2, w.y));
    } else {
        const float4 w = static_cast<const float4*>(spec)[e];
        u = make_float2(w.x, w.y);
        v = make_float2(w.z, w.w);
    }
}

template <bool SH>
__device__ __forceinline__ void spec_store(void* spec, int64_t e, float2 u, float2 v) {
    if constexpr (SH) static_cast<uint2*>(spec)[e] = make_uint2(h2_bits(u.x, u.y), h2_bits(v.x, v.y));
    else static_cast<float4*>(spec)[e] = make_float4(u.x, u.y, v.x, v.y);
}

// W(f) / P for element f: (Z(f) U(f) + conj(Z(-f)) V(f)) / P; entries above P/2 are
// the conjugates of the stored entries at P - f (real filters).
template <bool SH>
__device__ __forceinline__ float2 spectral_product(float2 z, float2 zn, const void* spec, int64_t e,
                                                   bool upper, float inv_p) {
    float2 u, w;
    spec_load<SH>(spec, e, u, w);
    if (upper) {
        u = cconj(u);
        w = cconj(w);
    }
    return cscale(cadd(cmul(z, u), cmul(cconj(zn), w)), inv_p);
}

// U and V of the spectrum from the transform Zk of the taps pair (k_d + i k_{d+1}).
template <bool SH>
__device__ __forceinline__ void spectrum_entry(void* spec, int64_t e, float2 z, float2 zn) {
    const float2 c = cconj(zn);
    const float2 hd = cscale(cadd(z, c), 0.5f);                   // H_d
    const float2 dd = csub(z, c);
    const float2 hd1 = make_float2(0.5f * dd.y, -0.5f * dd.x);     // H_{d+1} = (z - conj zn) / (2i)
    spec_store<SH>(spec, e, cscale(cadd(hd, hd1), 0.5f), cscale(csub(hd, hd1), 0.5f));
}

template <int MODE, int TA, int TO, bool SH>
__global__ __launch_bounds__(kThreads, 2) void short_kernel(
    const Doc* __restrict__ docs, const int32_t* __restrict__ tile_docs, int64_t region_off,
    const void* __restrict__ a, int N, int D, void* __restrict__ spec, void* __restrict__ out,
    const float2* __restrict__ tw) {
    __shared__ float2 s_z[kTile][kPairs];
    __shared__ float2 s_tw[kTile / 2];
    __shared__ uint8_t s_lp[kTile];   // log2 of the point's document size (0: none)
    __shared__ int16_t s_doc[kTile];  // the point's document relative to d0 (-1: none)
    const int tile = blockIdx.y, pb = blockIdx.x;
    const int q = threadIdx.x & (kPairs - 1), slot = threadIdx.x / kPairs;
    const int p = pb * kPairs + q;
    const int d0 = tile_docs[2 * tile], d1 = tile_docs[2 * tile + 1];
    const int64_t base = region_off + static_cast<int64_t>(tile) * kTile;
    load_tile_twiddles(s_tw, tw);
    for (int u = threadIdx.x; u < kTile; u += kThreads) {
        int lp = 0, rel = -1;
        const int64_t pos = base + u;
        if (d1 > d0 && docs[d0].off <= pos) {
            int lo = d0, hi = d1;  // docs[lo].off <= pos < docs[hi].off
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (docs[mid].off <= pos) lo = mid;
                else hi = mid;
            }
            if (pos < static_cast<int64_t>(docs[lo].off) + (int64_t(1) << docs[lo].logp)) {
                lp = docs[lo].logp;
                rel = lo - d0;
            }
        }
        s_lp[u] = static_cast<uint8_t>(lp);
        s_doc[u] = static_cast<int16_t>(rel);
    }
    __syncthreads();
    const TileTw ttw{s_tw};
    // forward stages 1-3, loading the bit-reversed samples straight from global memory
    #pragma unroll
    for (int g = slot; g < kTileGroups; g += kSlots) {
        float2 v[8];
        int lp[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int u = 8 * g + i;
            const int rel = s_doc[u];
            lp[i] = s_lp[u];
            v[i] = make_float2(0.f, 0.f);
            if (rel >= 0) {
                const Doc d = load_doc(docs, d0 + rel);
                const int t = bitrev(static_cast<int>(base + u - d.off), d.logp);
                if (t < d.len) v[i] = load_pair<TA>(a, d.row, d.start + t, N, D, p);
            }
        }
        auto on = [&](int i, int sigma) { return lp[i] >= sigma; };
        dit_group<3>(v, 0, 1, 1, ttw, on);
#pragma unroll
        for (int i = 0; i < 8; ++i) s_z[8 * g + i][q] = v[i];
    }
    __syncthreads();
    tile_pass<false>(s_z, s_lp, ttw, 3, q, slot);
    __syncthreads();
    tile_pass<false>(s_z, s_lp, ttw, 6, q, slot);
    __syncthreads();
    constexpr int kPer = kTile / kSlots;  // points per thread
    if constexpr (MODE == 1) {
        // spectrum entries f <= P/2 of every size class in the tile
        for (int k = 0; k < kPer; ++k) {
            const int u = slot + kSlots * k;
            const int rel = s_doc[u];
            if (rel < 0) continue;
            const Doc d = load_doc(docs, d0 + rel);
            const int P = 1 << d.logp;
            const int f = static_cast<int>(base + u - d.off);
            if (2 * f > P) continue;
            const int nf = (P - f) & (P - 1);
            spectrum_entry<SH>(spec, d.spec + (static_cast<int64_t>(pb) * (P / 2 + 1) + f) * kPairs + q,
                               s_z[u][q], s_z[u - f + nf][q]);
        }
        return;
    } else {
        float2 w[kPer];
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int u = slot + kSlots * k;
            const int rel = s_doc[u];
            w[k] = make_float2(0.f, 0.f);
            if (rel >= 0) {
                const Doc d = load_doc(docs, d0 + rel);
                const int P = 1 << d.logp;
                const int f = static_cast<int>(base + u - d.off);
                const int nf = (P - f) & (P - 1);
                const bool upper = 2 * f > P;
                const int fi = upper ? P - f : f;
                w[k] = spectral_product<SH>(s_z[u][q], s_z[u - f + nf][q], spec,
                                            d.spec + (static_cast<int64_t>(pb) * (P / 2 + 1) + fi) * kPairs + q,
                                            upper, 1.0f / P);
            }
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kPer; ++k) s_z[slot + kSlots * k][q] = w[k];
        __syncthreads();
        tile_pass<true>(s_z, s_lp, ttw, 6, q, slot);
        __syncthreads();
        tile_pass<true>(s_z, s_lp, ttw, 3, q, slot);
        __syncthreads();
        // inverse stages 3-1, then every sample to its bit-reversed time in y
        #pragma unroll
    for (int g = slot; g < kTileGroups; g += kSlots) {
            float2 v[8];
            int lp[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                v[i] = s_z[8 * g + i][q];
                lp[i] = s_lp[8 * g + i];
            }
            auto on = [&](int i, int sigma) { return lp[i] >= sigma; };
            dif_group<3>(v, 0, 1, 1, ttw, on);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int u = 8 * g + i;
                const int rel = s_doc[u];
                if (rel < 0) continue;
                const Doc d = load_doc(docs, d0 + rel);
                const int t = bitrev(static_cast<int>(base + u - d.off), d.logp);
                if (t < d.len) store_pair<TO>(out, d.row, d.start + t, N, D, p, v[i]);
            }
        }
    }
}

// ---------------------------------------------------------------- long documents
// Tile k of document d holds, at point u, time c + M * bitrev(u) (forward input and
// inverse output alike), with M = P / kTile and c = bitrev(k) over log2 M bits.
template <int TA, bool HALF>
__global__ __launch_bounds__(kThreads, 2) void front_kernel(
    const Doc* __restrict__ docs, const int32_t* __restrict__ tile_doc, const void* __restrict__ a,
    int N, int D, void* __restrict__ grid, int64_t long_points, const float2* __restrict__ tw) {
    __shared__ float2 s_z[kTile][kPairs];
    __shared__ float2 s_tw[kTile / 2];
    const int tile = blockIdx.y, pb = blockIdx.x;
    const int q = threadIdx.x & (kPairs - 1), slot = threadIdx.x / kPairs;
    const int p = pb * kPairs + q;
    const Doc d = load_doc(docs, tile_doc[tile]);
    const int lg_m = d.logp - kLogTile;
    const int c = bitrev(static_cast<int>((static_cast<int64_t>(tile) * kTile - d.off) >> kLogTile), lg_m);
    load_tile_twiddles(s_tw, tw);
    __syncthreads();
    const TileTw ttw{s_tw};
    #pragma unroll
    for (int g = slot; g < kTileGroups; g += kSlots) {
        float2 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int t = c + (bitrev(8 * g + i, kLogTile) << lg_m);
            v[i] = t < d.len ? load_pair<TA>(a, d.row, d.start + t, N, D, p) : make_float2(0.f, 0.f);
        }
        dit_group<3>(v, 0, 1, 1, ttw, AllOn{});
#pragma unroll
        for (int i = 0; i < 8; ++i) s_z[8 * g + i][q] = v[i];
    }
    __syncthreads();
    tile_pass<false>(s_z, nullptr, ttw, 3, q, slot);
    __syncthreads();
    const int64_t row0 = static_cast<int64_t>(pb) * long_points + static_cast<int64_t>(tile) * kTile;
    #pragma unroll
    for (int g = slot; g < kTileGroups; g += kSlots) {  // stages 7-9, stride 64, to the grid
        float2 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = s_z[g + 64 * i][q];
        dit_group<3>(v, g, 64, 7, ttw, AllOn{});
#pragma unroll
        for (int i = 0; i < 8; ++i) grid_store<HALF>(grid, (row0 + g + 64 * i) * kPairs + q, v[i]);
    }
}

template <int TO, bool HALF>
__global__ __launch_bounds__(kThreads, 2) void back_kernel(
    const Doc* __restrict__ docs, const int32_t* __restrict__ tile_doc, const void* __restrict__ grid,
    int64_t long_points, void* __restrict__ out, int N, int D, const float2* __restrict__ tw) {
    __shared__ float2 s_z[kTile][kPairs];
    __shared__ float2 s_tw[kTile / 2];
    const int tile = blockIdx.y, pb = blockIdx.x;
    const int q = threadIdx.x & (kPairs - 1), slot = threadIdx.x / kPairs;
    const int p = pb * kPairs + q;
    const Doc d = load_doc(docs, tile_doc[tile]);
    const int lg_m = d.logp - kLogTile;
    const int c = bitrev(static_cast<int>((static_cast<int64_t>(tile) * kTile - d.off) >> kLogTile), lg_m);
    load_tile_twiddles(s_tw, tw);
    __syncthreads();
    const TileTw ttw{s_tw};
    const int64_t row0 = static_cast<int64_t>(pb) * long_points + static_cast<int64_t>(tile) * kTile;
    #pragma unroll
    for (int g = slot; g < kTileGroups; g += kSlots) {  // inverse stages 9-7 from the grid
        float2 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = grid_load<HALF>(grid, (row0 + g + 64 * i) * kPairs + q);
        dif_group<3>(v, g, 64, 7, ttw, AllOn{});
#pragma unroll
        for (int i = 0; i < 8; ++i) s_z[g + 64 * i][q] = v[i];
    }
    __syncthreads();
    tile_pass<true>(s_z, nullptr, ttw, 3, q, slot);
    __syncthreads();
    #pragma unroll
    for (int g = slot; g < kTileGroups; g += kSlots) {  // inverse stages 3-1, to y
        float2 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = s_z[8 * g + i][q];
        dif_group<3>(v, 0, 1, 1, ttw, AllOn{});
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int t = c + (bitrev(8 * g + i, kLogTile) << lg_m);
            if (t < d.len) store_pair<TO>(out, d.row, d.start + t, N, D, p, v[i]);
        }
    }
}

// Column pass over the columns l = c + S j (j < Mv) of one long document, S = kTile 2^A
// and Mv = M / 2^A: A = max(0, log2 M - kMaxLogCols) middle stages run first
// (mid_kernel), so that a column never holds more than 2^kMaxLogCols points.  A work
// item holds kTile points of every pair lane: G = kTile / (2 Mv) low columns
// c = g * G + s (s < G) and, in the high slots, their partners S - c, which hold the
// frequencies -f of the low columns' frequencies f = c + S j.  Column 0 is its own
// partner, so the high slot that would repeat it holds column S / 2, also its own
// partner.  A document of M points per 512-point column has M work items.
// LDS row of (slot, j): slot * Mv + j.
template <int K, bool INV>
__device__ __forceinline__ void col_pass(float2 (*s_c)[kPairs], const int* cols, int lg_v, int lg_s,
                                         int sigma0, GlobalTw tw, int q, int slot) {
    // stages sigma0 .. sigma0 + K - 1 (> lg_s): element stride over j is 2^(sigma0 - lg_s - 1)
    const int lg_hj = sigma0 - lg_s - 1;
    const int hj = 1 << lg_hj;
    const int lg_per = lg_v - K;  // groups per column: Mv / 2^K
    for (int e = slot; e < (kTile >> K); e += kSlots) {
        const int s = e >> lg_per, g = e & ((1 << lg_per) - 1);
        const int jb = (g & (hj - 1)) + ((g >> lg_hj) << (lg_hj + K));
        const int row = (s << lg_v) + jb;
        float2 v[1 << K];
#pragma unroll
        for (int i = 0; i < (1 << K); ++i) v[i] = s_c[row + i * hj][q];
        const int b0 = cols[s] + ((jb & (hj - 1)) << lg_s);
        if constexpr (INV) dif_group<K>(v, b0, hj << lg_s, sigma0, tw, AllOn{});
        else dit_group<K>(v, b0, hj << lg_s, sigma0, tw, AllOn{});
#pragma unroll
        for (int i = 0; i < (1 << K); ++i) s_c[row + i * hj][q] = v[i];
    }
}

// All stages of the column pass in one direction: passes of 3, then the remainder.
template <bool INV>
__device__ __forceinline__ void col_stages(float2 (*s_c)[kPairs], const int* cols, int lg_v, int lg_s,
                                           GlobalTw tw, int q, int slot) {
    const int n3 = lg_v / 3, rem = lg_v - 3 * n3;
    int sig[3], kk[3], n = 0;
    int s0 = lg_s + 1;
    for (int i = 0; i < n3; ++i) { sig[n] = s0; kk[n] = 3; ++n; s0 += 3; }
    if (rem) { sig[n] = s0; kk[n] = rem; ++n; }
    for (int t = 0; t < n; ++t) {
        const int i = INV ? n - 1 - t : t;
        if (kk[i] == 3) col_pass<3, INV>(s_c, cols, lg_v, lg_s, sig[i], tw, q, slot);
        else if (kk[i] == 2) col_pass<2, INV>(s_c, cols, lg_v, lg_s, sig[i], tw, q, slot);
        else col_pass<1, INV>(s_c, cols, lg_v, lg_s, sig[i], tw, q, slot);
        __syncthreads();
    }
}

// Middle stages kLogTile + 1 .. kLogTile + A of a document with M = 2^(kMaxLogCols + A)
// points per 512-point column (A >= 1).  With j = jhi 2^A + jlo, those stages pair
// j's that differ in jlo only; tile t = jhi 2^A + chunk holds the 512 points
// l = c + kTile (jhi 2^A + jlo) for the 2^(kLogTile - A) columns c of its chunk and every
// jlo (LDS row jlo 2^(kLogTile - A) + c - c0).  The forward runs the decimation-in-time
// stages upwards, the inverse the decimation-in-frequency stages downwards.
template <bool INV, bool HALF>
__global__ __launch_bounds__(kThreads, 2) void mid_kernel(const Doc* __restrict__ docs,
                                                          const int32_t* __restrict__ tiles,
                                                          void* __restrict__ grid, int64_t long_points,
                                                          const float2* __restrict__ tw) {
    __shared__ float2 s_z[kTile][kPairs];
    const int it = tiles[blockIdx.y], pb = blockIdx.x;
    const int q = threadIdx.x & (kPairs - 1), slot = threadIdx.x / kPairs;
    const Doc d = load_doc(docs, it >> kItemBits);
    const int t = it & ((1 << kItemBits) - 1);
    const int lg_a = d.logp - kLogTile - kMaxLogCols;  // 1 .. kMaxLogMid
    const int lg_cn = kLogTile - lg_a;                  // columns per tile
    const int c0 = (t & ((1 << lg_a) - 1)) << lg_cn, jhi = t >> lg_a;
    const int64_t row0 = static_cast<int64_t>(pb) * long_points + d.off + c0 +
                         (static_cast<int64_t>(jhi) << (kLogTile + lg_a));
    constexpr int kPer = kTile / kSlots;
    auto flat = [&](int e) {  // LDS row e -> offset from row0: c + kTile * jlo
        return (e & ((1 << lg_cn) - 1)) + ((e >> lg_cn) << kLogTile);
    };
    {
        float2 r[kPer];
#pragma unroll
        for (int k = 0; k < kPer; ++k) r[k] = grid_load<HALF>(grid, (row0 + flat(slot + kSlots * k)) * kPairs + q);
#pragma unroll
        for (int k = 0; k < kPer; ++k) s_z[slot + kSlots * k][q] = r[k];
    }
    __syncthreads();
    const GlobalTw gtw{tw};
    for (int st = 0; st < lg_a; ++st) {
        const int k = INV ? lg_a - 1 - st : st;   // stage kLogTile + 1 + k: jlo distance 2^k
        for (int b = slot; b < kTile / 2; b += kSlots) {
            const int cc = b & ((1 << lg_cn) - 1), jp = b >> lg_cn;
            const int jlo = ((jp >> k) << (k + 1)) | (jp & ((1 << k) - 1));  // bit k clear
            const int ea = (jlo << lg_cn) + cc, eb = ea + (1 << (lg_cn + k));
            const float2 w = gtw(c0 + cc + ((jlo & ((1 << k) - 1)) << kLogTile), kLogTile + 1 + k);
            const float2 a = s_z[ea][q], bb = s_z[eb][q];
            if constexpr (INV) {
                s_z[ea][q] = cadd(a, bb);
                s_z[eb][q] = mul_conj(csub(a, bb), w);
            } else {
                const float2 tb = cmul(w, bb);
                s_z[ea][q] = cadd(a, tb);
                s_z[eb][q] = csub(a, tb);
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const int e = slot + kSlots * k;
        grid_store<HALF>(grid, (row0 + flat(e)) * kPairs + q, s_z[e][q]);
    }
}

template <int MODE, bool HALF, bool SH>
__global__ __launch_bounds__(kThreads, 2) void col_kernel(
    const Doc* __restrict__ docs, const int32_t* __restrict__ items, void* __restrict__ grid,
    int64_t long_points, void* __restrict__ spec, const float2* __restrict__ tw) {
    __shared__ float2 s_c[kTile][kPairs];
    __shared__ int s_cols[kTile / 2];  // column of each slot (2G <= kTile / 2 slots)
    __shared__ int s_part[kTile / 2];  // slot holding the partner column
    const int item = items[blockIdx.y], pb = blockIdx.x;
    const int q = threadIdx.x & (kPairs - 1), slot = threadIdx.x / kPairs;
    const Doc d = load_doc(docs, item >> kItemBits);
    const int grp = item & ((1 << kItemBits) - 1);
    const int lg_m0 = d.logp - kLogTile;
    const int lg_a = lg_m0 > kMaxLogCols ? lg_m0 - kMaxLogCols : 0;  // stages of the middle pass
    const int lg_m = lg_m0 - lg_a;        // points per column of the view (Mv)
    const int lg_s = kLogTile + lg_a;     // the view's column stride S
    const int S = 1 << lg_s, M = 1 << lg_m, P = 1 << d.logp;
    const int lg_g = kLogTile - 1 - lg_m;  // G = kTile / (2 Mv) low columns
    const int G = 1 << lg_g;
    if (threadIdx.x < 2 * G) {
        const int s = threadIdx.x & (G - 1);
        const int lo = grp * G + s;
        const bool high = threadIdx.x >= G;
        const int c = !high ? lo : (lo == 0 ? S / 2 : S - lo);
        s_cols[threadIdx.x] = c;
        s_part[threadIdx.x] = (c == 0 || c == S / 2) ? threadIdx.x : (high ? s : G + s);
    }
    __syncthreads();
    const int64_t row0 = static_cast<int64_t>(pb) * long_points + d.off;
    constexpr int kPer = kTile / kSlots;  // elements per thread
    const int lg_2g = lg_g + 1;
    {
        float2 r[kPer];  // every load issued before the first LDS store
#pragma unroll
        for (int k = 0; k < kPer; ++k) {  // e = j * 2G + slot: adjacent columns adjacent
            const int e = slot + kSlots * k;
            const int s = e & ((2 << lg_g) - 1), j = e >> lg_2g;
            r[k] = grid_load<HALF>(grid, (row0 + s_cols[s] + (static_cast<int64_t>(j) << lg_s)) * kPairs + q);
        }
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int e = slot + kSlots * k;
            s_c[((e & ((2 << lg_g) - 1)) << lg_m) + (e >> lg_2g)][q] = r[k];
        }
    }
    __syncthreads();
    const GlobalTw gtw{tw};
    col_stages<false>(s_c, s_cols, lg_m, lg_s, gtw, q, slot);
    if constexpr (MODE == 1) {
        for (int e = slot; e < kTile; e += kSlots) {
            const int s = e & ((2 << lg_g) - 1), j = e >> lg_2g;
            const int c = s_cols[s];
            const int f = c + (j << lg_s);
            if (2 * f > P) continue;
            const int jn = c == 0 ? (M - j) & (M - 1) : M - 1 - j;
            spectrum_entry<SH>(spec, d.spec + (static_cast<int64_t>(pb) * (P / 2 + 1) + f) * kPairs + q,
                               s_c[(s << lg_m) + j][q], s_c[(s_part[s] << lg_m) + jn][q]);
        }
        return;
    } else {
        // each thread owns frequency pairs (f, -f) with f <= P/2: the elements j < M/2 of
        // every slot, and f = P/2 in column 0; it reads both values and one spectrum entry
        // and writes both products, so no other thread touches them
        const float inv_p = 1.0f / P;
        const int64_t sp0 = d.spec + static_cast<int64_t>(pb) * (P / 2 + 1) * kPairs + q;
        auto product = [&](int s, int j) {
            const int c = s_cols[s];
            const int f = c + (j << lg_s);
            const int jn = c == 0 ? (M - j) & (M - 1) : M - 1 - j;
            const int rf = (s << lg_m) + j, rn = (s_part[s] << lg_m) + jn;
            float2 u, v;
            spec_load<SH>(spec, sp0 + static_cast<int64_t>(f) * kPairs, u, v);
            const float2 z = s_c[rf][q], zn = s_c[rn][q];
            const float2 wn = cscale(cadd(cmul(zn, cconj(u)), cmul(cconj(z), cconj(v))), inv_p);
            const float2 wf = cscale(cadd(cmul(z, u), cmul(cconj(zn), v)), inv_p);
            s_c[rn][q] = wn;
            s_c[rf][q] = wf;  // last: for f = -f both are the same element and value
        };
        for (int e = slot; e < kTile / 2; e += kSlots) product(e & ((2 << lg_g) - 1), e >> lg_2g);
        if (grp == 0 && slot == 0) product(0, M / 2);
        __syncthreads();
        col_stages<true>(s_c, s_cols, lg_m, lg_s, gtw, q, slot);
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int e = slot + kSlots * k;
            const int s = e & ((2 << lg_g) - 1), j = e >> lg_2g;
            grid_store<HALF>(grid, (row0 + s_cols[s] + (static_cast<int64_t>(j) << lg_s)) * kPairs + q,
                             s_c[(s << lg_m) + j][q]);
        }
    }
}

}  // namespace

template <int V>
using IC = std::integral_constant<int, V>;

template <class F>
void dispatch2(int v, F f) {  // v in {0, 1}
    if (v) f(IC<1>{});
    else f(IC<0>{});
}

hipError_t launch_short(int mode, const Doc* docs, const int32_t* tile_docs, int n_tiles,
                        int64_t region_off, int a_dtype, const void* a, int N, int D, int npb,
                        bool spec_half, void* spec, int out_dtype, void* out, const float2* tw,
                        hipStream_t stream) {
    if (n_tiles == 0) return hipSuccess;
    const dim3 grid(npb, n_tiles);  // pair blocks of one tile adjacent: whole token rows
    dispatch2(spec_half, [&](auto sh) {
        if (mode == 1) {
            hipLaunchKernelGGL((short_kernel<1, 0, 0, decltype(sh)::value != 0>), grid, dim3(kThreads), 0,
                               stream, docs, tile_docs, region_off, a, N, D, spec, nullptr, tw);
            return;
        }
        dispatch2(a_dtype, [&](auto ta) {
            dispatch2(out_dtype, [&](auto to) {
                hipLaunchKernelGGL((short_kernel<0, decltype(ta)::value, decltype(to)::value,
                                                 decltype(sh)::value != 0>),
                                   grid, dim3(kThreads), 0, stream, docs, tile_docs, region_off, a, N, D,
                                   spec, out, tw);
            });
        });
    });
    return hipGetLastError();
}

hipError_t launch_front(const Doc* docs, const int32_t* tile_doc, int n_tiles, int a_dtype,
                        const void* a, int N, int D, int npb, bool half, void* grid,
                        int64_t long_points, const float2* tw, hipStream_t stream) {
    if (n_tiles == 0) return hipSuccess;
    const dim3 g(npb, n_tiles);  // pair blocks of one tile adjacent: whole token rows
    if (a_dtype == 0 && !half)
        hipLaunchKernelGGL((front_kernel<0, false>), g, dim3(kThreads), 0, stream, docs, tile_doc, a, N, D,
                           grid, long_points, tw);
    else if (a_dtype == 0)
        hipLaunchKernelGGL((front_kernel<0, true>), g, dim3(kThreads), 0, stream, docs, tile_doc, a, N, D,
                           grid, long_points, tw);
    else if (!half)
        hipLaunchKernelGGL((front_kernel<1, false>), g, dim3(kThreads), 0, stream, docs, tile_doc, a, N, D,
                           grid, long_points, tw);
    else
        hipLaunchKernelGGL((front_kernel<1, true>), g, dim3(kThreads), 0, stream, docs, tile_doc, a, N, D,
                           grid, long_points, tw);
    return hipGetLastError();
}

hipError_t launch_col(int mode, const Doc* docs, const int32_t* items, int n_items, bool half,
                      void* grid, int64_t long_points, int npb, bool spec_half, void* spec,
                      const float2* tw, hipStream_t stream) {
    if (n_items == 0) return hipSuccess;
    const dim3 g(npb, n_items);
    dispatch2(mode, [&](auto md) {
        dispatch2(half, [&](auto hf) {
            dispatch2(spec_half, [&](auto sh) {
                hipLaunchKernelGGL((col_kernel<decltype(md)::value, decltype(hf)::value != 0,
                                               decltype(sh)::value != 0>),
                                   g, dim3(kThreads), 0, stream, docs, items, grid, long_points, spec, tw);
            });
        });
    });
    return hipGetLastError();
}

hipError_t launch_mid(bool inverse, const Doc* docs, const int32_t* tiles, int n_tiles, bool half,
                      void* grid, int64_t long_points, int npb, const float2* tw, hipStream_t stream) {
    if (n_tiles == 0) return hipSuccess;
    const dim3 g(npb, n_tiles);
    dispatch2(inverse, [&](auto iv) {
        dispatch2(half, [&](auto hf) {
            hipLaunchKernelGGL((mid_kernel<decltype(iv)::value != 0, decltype(hf)::value != 0>), g,
                               dim3(kThreads), 0, stream, docs, tiles, grid, long_points, tw);
        });
    });
    return hipGetLastError();
}

hipError_t launch_back(const Doc* docs, const int32_t* tile_doc, int n_tiles, bool half,
                       const void* grid, int64_t long_points, int npb, int out_dtype, void* out,
                       int N, int D, const float2* tw, hipStream_t stream) {
    if (n_tiles == 0) return hipSuccess;
    const dim3 g(npb, n_tiles);  // pair blocks of one tile adjacent: whole token rows
    if (out_dtype == 0 && !half)
        hipLaunchKernelGGL((back_kernel<0, false>), g, dim3(kThreads), 0, stream, docs, tile_doc, grid,
                           long_points, out, N, D, tw);
    else if (out_dtype == 0)
        hipLaunchKernelGGL((back_kernel<0, true>), g, dim3(kThreads), 0, stream, docs, tile_doc, grid,
                           long_points, out, N, D, tw);
    else if (!half)
        hipLaunchKernelGGL((back_kernel<1, false>), g, dim3(kThreads), 0, stream, docs, tile_doc, grid,
                           long_points, out, N, D, tw);
    else
        hipLaunchKernelGGL((back_kernel<1, true>), g, dim3(kThreads), 0, stream, docs, tile_doc, grid,
                           long_points, out, N, D, tw);
    return hipGetLastError();
}

}  // namespace rubiconv::ct
