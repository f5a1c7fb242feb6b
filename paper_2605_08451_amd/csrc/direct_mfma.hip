// direct_mfma.hip -- the direct path on the matrix cores (bf16 inputs, documents of up to
// kMaxDirectMfma tokens).
//
// A document's causal convolution is the block-diagonal Toeplitz product of Section 3.2
// restricted to its own block.  Cut into 16-token blocks it reads, per channel,
//   out_b = sum_{c <= b} F_c g_{b - c},   F_c[i][j] = f[16 c + i - j]   (0 outside [0, nf)),
// so each 16 x 16 block F_c is one matrix-core operand, applied at once to 16 output
// blocks (the operand's 16 columns).  v_mfma_f32_16x16x32_bf16 takes two tap blocks per
// instruction: A = [F_c | F_{c+1}], B = [g_{b-c} ; g_{b-c-1}] for columns b.  The three
// modes are the same convolution:
//   kDirectConv  (y from x):   f = k, g = x, out = y;
//   kDirectCorr  (dx from dy): f = k, g = dy reversed in time, out = dx reversed;
//   kDirectXcorr (the filter gradient's correlation of dy with x): f = x, g = dy reversed,
//                out(w) = r(len - 1 - w) for lags len - 1 - w < min(len, L).
// Taps (fp32) enter as bf16 pairs hi + lo (two products), x and dy are bf16 as given;
// every sum runs in fp32 on the matrix cores.  A workgroup takes one document and 16
// channels, stages g and f (the taps, or x) channel-major in LDS, gives each wave two
// channels to compute and writes the outputs back through LDS as whole rows of its
// channels.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.hpp"

namespace rubiconv {

namespace {

typedef __bf16 b8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kRow = kMaxDirectMfma;   // tokens (or taps) per channel row in LDS
constexpr int kFront = 16;             // zeros in front of each row
constexpr int kStride = kFront + kRow; // LDS elements per row
constexpr int kWaves = 8;
constexpr int kCh = 16;                // channels per workgroup

__device__ __forceinline__ f4 mma_bf16(u4 a, u4 b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b8, a), __builtin_bit_cast(b8, b), c, 0,
                                                   0, 0);
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000);
}
__device__ __forceinline__ uint32_t bf16_rne(float v) {
    const uint32_t u = __float_as_uint(v);
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

template <int MODE>
__global__ __launch_bounds__(64 * kWaves) void direct_mfma_kernel(const uint16_t* __restrict__ a,
                                                                  const uint16_t* __restrict__ b,
                                                                  const uint32_t* __restrict__ taps, int T,
                                                                  const Seg* __restrict__ docs, int N, int D,
                                                                  int L, void* __restrict__ out) {
    constexpr bool kX = MODE == kDirectXcorr;
    constexpr int PER = kCh / kWaves;      // channels per wave
    // LDS (32-bit words): g rows [kCh][kStride] bf16, then f rows: x [kCh][kStride] bf16 for
    // the correlation, the taps [kCh][kStride] as bf16 pairs otherwise.  Each row holds
    // kFront zeros, then its data (zero past it): operands that reach before a row's start
    // read those zeros.  Reused for the outputs as [token][kCh] (bf16, or fp32).
    __shared__ uint32_t smem[kCh * kStride / 2 + (kX ? kCh * kStride / 2 : kCh * kStride)];
    uint16_t* gtile = reinterpret_cast<uint16_t*>(smem);
    uint16_t* xtile = reinterpret_cast<uint16_t*>(smem + kCh * kStride / 2);  // the correlation's f
    uint32_t* ttile = smem + kCh * kStride / 2;                                // the taps
    const Seg sg = docs[blockIdx.x];
    const int n = sg.len;
    const int nb = (n + 15) / 16, ng = (nb + 15) / 16;
    const int d0 = blockIdx.y * kCh;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int p = lane & 15, h = lane >> 4;
    const int64_t row0 = static_cast<int64_t>(sg.row) * N + sg.start;  // the document's first token

    // stage every row from kFront zeros up to what the operands read (256 ng + 15 tokens at
    // most, never past kRow); all loads of a thread are issued before its LDS writes
    const int fill = 256 * ng + 16 < kRow ? 256 * ng + 16 : kRow;
    {
        // g (and the correlation's x): 16 bytes (8 channels) per load, two per token each
        constexpr int kChunks = kX ? 4 : 2;
        constexpr int kTotal = (kFront + kRow) * kChunks;
        constexpr int kIters = (kTotal + 64 * kWaves - 1) / (64 * kWaves);
        u4 v[kIters];
#pragma unroll
        for (int j = 0; j < kIters; ++j) {
            const int i = static_cast<int>(threadIdx.x) + 64 * kWaves * j;
            const int t = (i < kTotal ? i / kChunks : kRow + kFront) - kFront, q = i % kChunks;
            const bool from_b = kX && q >= 2;
            // g reversed in time for dx and the correlation; f = x in order
            const int src = (MODE == kDirectConv || from_b) ? t : n - 1 - t;
            v[j] = u4{0u, 0u, 0u, 0u};
            if (t >= 0 && t < n) v[j] = *reinterpret_cast<const u4*>((from_b ? b : a) + (row0 + src) * D + d0 + 8 * (q & 1));
        }
#pragma unroll
        for (int j = 0; j < kIters; ++j) {
            const int i = static_cast<int>(threadIdx.x) + 64 * kWaves * j;
            const int t = (i < kTotal ? i / kChunks : kRow + kFront) - kFront, q = i % kChunks;
            if (t >= fill) continue;
            uint16_t* dst = ((kX && q >= 2) ? xtile : gtile) + (8 * (q & 1)) * kStride + kFront + t;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                dst[(2 * e) * kStride] = static_cast<uint16_t>(v[j][e] & 0xffffu);
                dst[(2 * e + 1) * kStride] = static_cast<uint16_t>(v[j][e] >> 16);
            }
        }
    }
    if constexpr (!kX) {
        // the taps k[tau], tau < T (every tap a document of at most T tokens reads), as
        // bf16 pairs; zero past T
        constexpr int kTotal = kCh * (kFront + kRow);
        constexpr int kIters = (kTotal + 64 * kWaves - 1) / (64 * kWaves);
        uint32_t w[kIters];
#pragma unroll
        for (int j = 0; j < kIters; ++j) {
            const int i = static_cast<int>(threadIdx.x) + 64 * kWaves * j;
            const int c = i / (kFront + kRow), tau = i % (kFront + kRow) - kFront;
            w[j] = (i < kTotal && tau >= 0 && tau < T && tau < fill) ? taps[static_cast<int64_t>(d0 + c) * T + tau]
                                                                      : 0u;
        }
#pragma unroll
        for (int j = 0; j < kIters; ++j) {
            const int i = static_cast<int>(threadIdx.x) + 64 * kWaves * j;
            const int c = i / (kFront + kRow), tau = i % (kFront + kRow) - kFront;
            if (i < kTotal && tau < fill) ttile[c * kStride + kFront + tau] = w[j];
        }
    }
    __syncthreads();

    f4 acc[PER][4];
#pragma unroll
    for (int k = 0; k < PER; ++k)
#pragma unroll
        for (int g = 0; g < 4; ++g) acc[k][g] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int c = 0; c < nb; c += 2) {
        // A: lane (p, h) holds f[e0 - t], t < 8, for K = 8 h + t (e0 - t >= -15: the zeros
        // in front of the row)
        const int e0 = 16 * c + p - 8 * h + (h >= 2 ? 32 : 0) + kFront;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int ch = wave + kWaves * k;
            u4 ahi, alo;
            if constexpr (kX) {
                const uint16_t* frow = xtile + ch * kStride;
                uint32_t v[8];
#pragma unroll
                for (int t = 0; t < 8; ++t) v[t] = frow[e0 - t];
#pragma unroll
                for (int q = 0; q < 4; ++q) ahi[q] = v[2 * q] | (v[2 * q + 1] << 16);
                alo = u4{0u, 0u, 0u, 0u};
            } else {
                const uint32_t* trow = ttile + ch * kStride;
                uint32_t w[8];  // packed taps: hi bf16 in the low half, lo bf16 in the high half
#pragma unroll
                for (int t = 0; t < 8; ++t) w[t] = trow[e0 - t];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    ahi[q] = __builtin_amdgcn_perm(w[2 * q + 1], w[2 * q], 0x05040100u);
                    alo[q] = __builtin_amdgcn_perm(w[2 * q + 1], w[2 * q], 0x07060302u);
                }
            }
            // B: lane (p, h) holds g[s0 + t], t < 8, of column 16 g + p; a chunk before the
            // row's start is all zero (s0 is a multiple of 8), read from the zeros in front
            const uint16_t* grow = gtile + ch * kStride + kFront;
            u4 bv[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int s0 = 16 * (16 * g + p - c) + 8 * h - (h >= 2 ? 32 : 0);
                bv[g] = *reinterpret_cast<const u4*>(grow + (s0 > -kFront ? s0 : -kFront));
            }
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                if (g >= ng || 16 * g + 15 < c) continue;  // wave-uniform
                acc[k][g] = mma_bf16(ahi, bv[g], acc[k][g]);
                if constexpr (!kX) acc[k][g] = mma_bf16(alo, bv[g], acc[k][g]);
            }
        }
    }
    __syncthreads();  // every wave is done with the staged rows

    // outputs into LDS as [token][kCh]: lane (p, h) of group g holds positions 16 (16 g + p) + 4 h + r
    const int lim = kX ? (n < L ? n : L) : n;  // rows to store
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int ch = wave + kWaves * k;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            if (g >= ng) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int w = 16 * (16 * g + p) + 4 * h + r;
                if (w >= n) continue;
                const int t = MODE == kDirectConv ? w : n - 1 - w;  // output row
                if (t >= lim) continue;
                if constexpr (kX)
                    reinterpret_cast<float*>(smem)[t * kCh + ch] = acc[k][g][r];
                else
                    reinterpret_cast<uint16_t*>(smem)[t * kCh + ch] = static_cast<uint16_t>(bf16_rne(acc[k][g][r]));
            }
        }
    }
    __syncthreads();

    // whole rows of the workgroup's channels, 16 bytes per lane: 64 bytes per token (fp32)
    // or 32 (bf16)
    constexpr int kPieces = kX ? 4 : 2;
    for (int i = threadIdx.x; i < lim * kPieces; i += 64 * kWaves) {
        const int t = i / kPieces, q = i % kPieces;
        if constexpr (kX) {
            float* o = static_cast<float*>(out) + (row0 + t) * D + d0 + 4 * q;
            *reinterpret_cast<u4*>(o) = reinterpret_cast<const u4*>(smem)[t * 4 + q];
        } else {
            uint16_t* o = static_cast<uint16_t*>(out) + (row0 + t) * D + d0 + 8 * q;
            *reinterpret_cast<u4*>(o) = reinterpret_cast<const u4*>(smem)[t * 2 + q];
        }
    }
}

}  // namespace

namespace {
// taps[d][t] = bf16(k) | bf16(k - bf16(k)) << 16 (round to nearest even), t < T
__global__ __launch_bounds__(256) void split_taps_kernel(const float* __restrict__ k, int D, int T, int ld,
                                                         uint32_t* __restrict__ taps) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= static_cast<int64_t>(D) * T) return;
    const int d = static_cast<int>(i / T), t = static_cast<int>(i % T);
    const float v = k[static_cast<int64_t>(d) * ld + t];
    const uint32_t hi = bf16_rne(v);
    const uint32_t lo = bf16_rne(v - __uint_as_float(hi << 16));
    taps[i] = hi | (lo << 16);
}
}  // namespace

hipError_t launch_split_taps(const float* filters, int D, int T, int ld, uint32_t* taps, hipStream_t stream) {
    const int64_t n = static_cast<int64_t>(D) * T;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(split_taps_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream,
                       filters, D, T, ld, taps);
    return hipGetLastError();
}

hipError_t launch_direct_mfma(int mode, const void* a, const void* b, const uint32_t* taps, int T,
                              const Seg* docs, int n_docs, int N, int D, int L, void* out, hipStream_t stream) {
    if (n_docs == 0) return hipSuccess;
    // 16-byte rows of 8 (bf16) or 4 (fp32) channels
    auto misaligned = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) != 0; };
    if (D % kCh != 0 || misaligned(a) || misaligned(out) || (mode == kDirectXcorr && misaligned(b)))
        return hipErrorInvalidValue;
    const dim3 blk(64 * kWaves);
    const auto* ap = static_cast<const uint16_t*>(a);
    const auto* bp = static_cast<const uint16_t*>(b);
    if (mode == kDirectXcorr)
        hipLaunchKernelGGL((direct_mfma_kernel<kDirectXcorr>), dim3(n_docs, D / kCh), blk, 0, stream, ap, bp,
                           taps, T, docs, N, D, L, out);
    else if (mode == kDirectCorr)
        hipLaunchKernelGGL((direct_mfma_kernel<kDirectCorr>), dim3(n_docs, D / kCh), blk, 0, stream, ap, bp,
                           taps, T, docs, N, D, L, out);
    else
        hipLaunchKernelGGL((direct_mfma_kernel<kDirectConv>), dim3(n_docs, D / kCh), blk, 0, stream, ap, bp,
                           taps, T, docs, N, D, L, out);
    return hipGetLastError();
}

}  // namespace rubiconv
