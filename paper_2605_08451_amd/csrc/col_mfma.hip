// col_mfma.hip -- column passes on the matrix cores (N1 = 256, complex fp16 grids).
//
// The N1 = 256-point column DFT of Algorithm 1 (the shared left DFT M1 = F_k) is
// applied as two dense 16 x 16 complex DFT stages on v_mfma_f32_16x16x32, the
// small DFT matrices being genuine dense contractions over a batch of 16
// channel pairs.  A complex 16 x 16 matrix M acts on [re; im] as the real
// 16 x 32 operands A_re = [Re M | -Im M] and A_im = [Im M | Re M], with the K
// index interleaving (re, im) per input, so the bf16/fp16 pair of a channel
// pair is one operand element pair as loaded.
//
// One wave = one grid column j of one document x one block of 16 channel pairs
// (lane l: pair p = l % 16, lane group h = l / 16).  With a = 16 n1 + n2 and
// u = k1 + 16 k2:
//   stage 1: for each n2, D[k1][p] = sum_n1 w16^(k1 n1) X[16 n1 + n2][p]
//            (lane group h holds n1 = h, h+4, h+8, h+12 on input, k1 = 4h..4h+3 on
//            output);
//   4 x 4 lane-group transposes (v_permlane32/16_swap) so that lane group h holds
//            n2 = 4h..4h+3 for every k1;
//   stage 2: for each k1, Y[k1 + 16 k2][p] = sum_n2 w16^(n2 k2) w256^(n2 k1) D[k1][n2][p]
//            (the inner twiddle is folded into one matrix per k1; lane group h
//            produces k2 = h, h+4, h+8, h+12);
//   the per-document twiddle w_P^(u j) / sqrt(N1) on the fp32 result, stored as fp16.
// The inverse runs the mirror image (conjugate twiddle on the fp16 input, inner
// twiddle folded per n2, output rounded to y's type).  Stage-1 matrices of the
// bf16 input are split hi + lo in bf16 so that the coefficients keep ~16 bits.
#include <hip/hip_bf16.h>
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "fft_core.hpp"
#include "kernels.hpp"
#include "pk_half.hpp"

namespace rubiconv {

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef __bf16 b8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_h2(float re, float im) {
    const __half2 h = __float22half2_rn(make_float2(re, im));
    return __builtin_bit_cast(uint32_t, h);
}
__device__ __forceinline__ float2 unpack_h2(uint32_t w) {
    return __half22float2(__builtin_bit_cast(__half2, w));
}
__device__ __forceinline__ uint32_t pack_bf2(float re, float im) { return bf2_bits(re, im); }

__device__ __forceinline__ f4 mma_f16(u4 a, u4 b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a), __builtin_bit_cast(h8, b),
                                                  c, 0, 0, 0);
}
__device__ __forceinline__ f4 mma_bf16(u4 a, u4 b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b8, a),
                                                   __builtin_bit_cast(b8, b), c, 0, 0, 0);
}

// 4 x 4 transpose of (register, lane group): afterwards r_g in lane group h holds
// what r_h held in lane group g.
__device__ __forceinline__ void lanegroup_transpose(uint32_t& r0, uint32_t& r1, uint32_t& r2,
                                                    uint32_t& r3) {
    const auto s02 = __builtin_amdgcn_permlane32_swap(r0, r2, false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(r1, r3, false, false);
    const auto t01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
    const auto t23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
    r0 = t01[0];
    r1 = t01[1];
    r2 = t23[0];
    r3 = t23[1];
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t doc_buffer(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes),
                                             0x00020000);
}
// The part [off, bytes) of a buffer of `bytes` bytes as a buffer of its own (empty
// when off >= bytes).  With wave-uniform arguments it costs scalar instructions
// only, and keeps the range check of every access exact: a lane offset v into it
// is in range exactly when off + v is in range of the whole buffer.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t sub_buffer(const void* base, int64_t bytes,
                                                             int64_t off) {
    const int64_t rest = bytes > off ? bytes - off : 0;
    return doc_buffer(static_cast<const char*>(base) + off, static_cast<uint32_t>(rest));
}

// Copies `chunks` 1 KB pieces of src into LDS, 16 bytes per lane, spread over the
// workgroup's four waves (buffer loads with the lds modifier: no registers).
__device__ __forceinline__ void copy_to_lds(const u4* src, u4* lds, int chunks, int wave, int lane) {
    const __amdgpu_buffer_rsrc_t rs = doc_buffer(src, static_cast<uint32_t>(chunks) * 1024);
    for (int c = wave; c < chunks; c += 4)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs, (__attribute__((address_space(3))) void*)(lds + c * 64), 16, c * 1024 + lane * 16, 0, 0, 0);
}

__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

constexpr int kTab2 = 16 * 2 * 64;  // stage-2 operands: 16 matrices x (re, im) x 64 lanes

constexpr int kF16In = 0;   // fp16 channel pairs (filter taps, packed by the pair transpose)
constexpr int kBf16In = 1;  // bf16 channel pairs (x): used as bf16 operands as loaded

// The largest of n bf16 magnitudes (16-bit words, 16-byte aligned), reduced by one wave on
// its own: every wave of the launch reads the same words and gets the same value.
__device__ __forceinline__ uint32_t wave_amax16(const uint16_t* __restrict__ a, int n, int lane) {
    const u4* v = reinterpret_cast<const u4*>(a);
    const int nv = n / 8;  // whole 16-byte groups
    uint32_t m = 0;
    for (int base = lane; base < nv; base += 8 * 64) {
        u4 w[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) w[u] = base + 64 * u < nv ? v[base + 64 * u] : u4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c) m = max(m, max(w[u][c] & 0xffffu, w[u][c] >> 16));
    }
    for (int i = nv * 8 + lane; i < n; i += 64) m = max(m, static_cast<uint32_t>(a[i]));
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), o)));
    return m;
}

// AMAX: the pass runs at scale first_scale in place of sc.glob, and each workgroup also
// writes the largest |x| its tasks loaded (bf16 magnitude bits) to amax_out[blockIdx.x]
// (launched with one workgroup per four tasks).  amax_in
// (the redo launch): the launch first takes the range scale s from the n_amax magnitudes
// a pass with AMAX recorded, times extra (a power of two), writes {s, p / s} to *used
// (p = prev->y, or 1 without prev) and s to *hint (workgroup 0), and does nothing more when
// s equals first_scale (the scale that pass used); otherwise it runs the pass at scale s.
template <int IN, bool AMAX>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void col_fwd_mfma_kernel(const void* __restrict__ src,
                                                           int64_t src_row_stride, int D,
                                                           uint32_t* __restrict__ grid,
                                                           int64_t grid_pb_stride, LaunchTables t,
                                                           GridScale sc,
                                                           const u4* __restrict__ mt, int npb,
                                                           int ntasks, uint16_t* __restrict__ amax_out,
                                                           const uint16_t* __restrict__ amax_in, int n_amax,
                                                           float2* __restrict__ used, float first_scale,
                                                           float* __restrict__ hint, float extra,
                                                           const float2* __restrict__ prev) {
    // stage-2 operands, shared by the workgroup's four column tasks
    __shared__ u4 tab2[kTab2];
    // per wave: one output row group (16 grid rows x 16 pairs) on its way to 16-byte stores
    __shared__ uint32_t ring_all[4][256];
    const int lane = threadIdx.x & 63;
    float glob_x = 1.0f;
    if (amax_in != nullptr) {
        glob_x = pow2_scale(__uint_as_float(wave_amax16(amax_in, n_amax, lane) << 16), kDataAmaxExp) * extra;
        if (blockIdx.x == 0 && threadIdx.x == 0) {
            used[0] = make_float2(glob_x, (prev != nullptr ? prev->y : 1.0f) / glob_x);
            if (hint != nullptr) *reinterpret_cast<volatile float*>(hint) = glob_x;
        }
        if (glob_x == first_scale) return;  // every wave of every workgroup alike, before any barrier
    } else {
        glob_x = AMAX ? first_scale : sc.glob->x;
    }
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    copy_to_lds(mt + kMtFwd2, tab2, kTab2 / 64, wave, lane);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // the only workgroup barrier (AMAX: and the one after the tasks)
    uint32_t wave_amax = 0;  // AMAX: the largest magnitude bits of the wave's tasks
    // wave-uniform task index: keeps the document's buffer resource in SGPRs.  A launch
    // with fewer workgroups than ntasks / 4 (the redo launch) loops over the tasks.
    for (int task = blockIdx.x * 4 + wave; task < ntasks; task += static_cast<int>(gridDim.x) * 4) {
        const int col = task / npb, pb = task - col * npb;
        const Seg* sg = t.segs + t.col_seg[col];
        const int j = col - sg->col0, m = sg->m, len = sg->len;
        const int p = lane & 15, h = lane >> 4;
        const int ch = 2 * (pb * kPairsPerBlock + p);
        constexpr int ES = 2;  // bytes per channel
        uint32_t* ring = ring_all[wave];

        const char* doc = static_cast<const char*>(src) +
                          (static_cast<int64_t>(sg->row) * src_row_stride +
                           static_cast<int64_t>(sg->start) * D) * ES;
        const int64_t doc_bytes = static_cast<int64_t>(len) * D * ES;

        // stage 1: one MFMA tile per n2 (bf16: hi and lo matrix halves accumulate).
        // Token t = m (16 n1 + n2) + j with n1 = 4i + h (operand slot 4h + i; the
        // matrix tables use the same interleaving): a lane part and a wave-uniform part.
        // All loads are issued before the first MFMA so that the wave waits once, at a
        // raised wave priority so that waves about to load issue ahead of waves that
        // compute (measured: the pass 2% faster)
        __builtin_amdgcn_s_setprio(3);
        u4 xb[16];
        {
            uint32_t lane_off[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                lane_off[i] = (static_cast<uint32_t>(m) * 16u * (4 * i + h) * D + ch) * ES;
#pragma unroll
            for (int n2 = 0; n2 < 16; ++n2) {
                const __amdgpu_buffer_rsrc_t rs =
                    sub_buffer(doc, doc_bytes, static_cast<int64_t>(m * n2 + j) * D * ES);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int off = static_cast<int>(lane_off[i]);
                    xb[n2][i] = __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
                }
            }
        }
        // per-document twiddle w_P^(u j) = w_P^(k1 j) * w_P^(16 k2 j), u = k1 + 16 k2: the first
        // factor is wave-uniform, the second has four values per lane (k2 = 4 r2 + h)
        const __amdgpu_buffer_rsrc_t rt = doc_buffer(t.tw + sg->twf_off, static_cast<uint32_t>(sg->P) * 8);
        uint32_t tw_lane[4];  // complex fp16
#pragma unroll
        for (int r2 = 0; r2 < 4; ++r2) {
            const auto w = __builtin_amdgcn_raw_buffer_load_b64(
                rt, static_cast<int>(16u * (4 * r2 + h) * j * 8), 0, 0);
            tw_lane[r2] = h2_bits(__uint_as_float(w[0]), __uint_as_float(w[1]));
        }
        u4 a[4];
        if constexpr (IN == kBf16In) {
#pragma unroll
            for (int o = 0; o < 4; ++o) a[o] = mt[kMtFwd1Bf16 + o * 64 + lane];
        } else {
#pragma unroll
            for (int o = 0; o < 2; ++o) a[o] = mt[kMtFwd1F16 + o * 64 + lane];
        }
        // range scale of this lane's pair, applied to the fp32 products before fp16 rounding
        const float in_mul = sc.pair[pb * kPairsPerBlock + p].x * glob_x;
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);

        uint32_t y[16][4];
        uint32_t amax_lo = 0, amax_hi = 0;  // the largest bf16 magnitude bits of the loaded x
#pragma unroll
        for (int n2 = 0; n2 < 16; ++n2) {
            const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
            f4 dre, dim;
            if constexpr (IN == kBf16In) {
                dre = mma_bf16(a[1], xb[n2], mma_bf16(a[0], xb[n2], zero));
                dim = mma_bf16(a[3], xb[n2], mma_bf16(a[2], xb[n2], zero));
            } else {
                dre = mma_f16(a[0], xb[n2], zero);
                dim = mma_f16(a[1], xb[n2], zero);
            }
            if constexpr (AMAX) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    amax_lo = max(amax_lo, xb[n2][i] & 0x7fffu);
                    amax_hi = max(amax_hi, xb[n2][i] & 0x7fff0000u);
                }
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) y[n2][r] = pack_h2(dre[r] * in_mul, dim[r] * in_mul);
        }
        const uint32_t amax_lane = max(amax_lo, amax_hi >> 16);
        // y[n2][r] = D[k1 = 4h + r][n2]; regroup so that lane group h holds n2 = 4h + r'
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int rp = 0; rp < 4; ++rp)
                lanegroup_transpose(y[rp][r], y[4 + rp][r], y[8 + rp][r], y[12 + rp][r]);

        // stage 2 per k1 = 4g + r, then the per-document twiddle and the fp16 store
        const float2* twf = t.tw + sg->twf_off;
        const uint32_t* gdoc = grid + pb * grid_pb_stride + sg->grid_off * kPairsPerBlock;
        const int64_t grid_bytes = static_cast<int64_t>(sg->P) * kPairsPerBlock * 4;
        const uint32_t g_lane = (static_cast<uint32_t>(j) * kPairsPerBlock + p) * 4;
        // 16-byte stores: lane l writes pairs 4 (l % 4) .. + 3 of grid row u = k1 + 16 (l / 4)
        const uint32_t st_lane = (static_cast<uint32_t>(16 * (lane >> 2)) * m + j) * (kPairsPerBlock * 4) +
                                 (lane & 3) * 16;
        (void)g_lane;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int k1 = 4 * g + r;
                const u4 b = {y[4 * g][r], y[4 * g + 1][r], y[4 * g + 2][r], y[4 * g + 3][r]};
                const u4 are = tab2[(2 * k1) * 64 + lane];
                const u4 aim = tab2[(2 * k1 + 1) * 64 + lane];
                const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
                const f4 dre = mma_f16(are, b, zero);
                const f4 dim = mma_f16(aim, b, zero);
                // both table factors carry 1/sqrt(N1): undo one (x 16, exact)
                const float2 tkf = cscale(twf[k1 * j], 16.0f);  // wave-uniform
                const uint32_t tk = h2_bits(tkf.x, tkf.y);
                // register r2 of lane (p, h) is grid row k1 + 16 (4 r2 + h), pair p
#pragma unroll
                for (int r2 = 0; r2 < 4; ++r2)
                    ring[(4 * r2 + h) * 16 + p] = cmul_h2(cmul_h2(h2_bits(dre[r2], dim[r2]), tk), tw_lane[r2]);
                wave_lds_fence();
                const u4 v = *reinterpret_cast<const u4*>(ring + lane * 4);
                const __amdgpu_buffer_rsrc_t rg =
                    sub_buffer(gdoc, grid_bytes, static_cast<int64_t>(k1) * m * (kPairsPerBlock * 4));
                __builtin_amdgcn_raw_buffer_store_b128(v, rg, static_cast<int>(st_lane), 0, 0);
                wave_lds_fence();  // the ring is rewritten for the next k1
            }
        }
        if constexpr (AMAX) {  // at the end, where few registers are live; every lane stores the same word
            uint32_t mx = amax_lane;
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) mx = max(mx, static_cast<uint32_t>(__shfl_xor(static_cast<int>(mx), o)));
            wave_amax = max(wave_amax, mx);
        }
    }
    if constexpr (AMAX) {  // one word per workgroup, so that the redo launch reduces a quarter as many
        __shared__ uint32_t wg_amax[4];
        wg_amax[wave] = wave_amax;  // every lane the same value
        __syncthreads();
        if (wave == 0)
            amax_out[blockIdx.x] =
                static_cast<uint16_t>(max(max(wg_amax[0], wg_amax[1]), max(wg_amax[2], wg_amax[3])));
    }
}

template <class TY>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void col_inv_mfma_kernel(const uint32_t* __restrict__ grid,
                                                           int64_t grid_pb_stride,
                                                           void* __restrict__ dst,
                                                           int64_t dst_row_stride, int D,
                                                           LaunchTables t, GridScale sc,
                                                           const u4* __restrict__ mt, int npb,
                                                           int ntasks) {
    constexpr int ES = std::is_same<TY, F32>::value ? 4 : 2;  // bytes per output channel
    __shared__ u4 tab2[kTab2];
    // per wave: one output group (16 tokens x 16 pairs) on its way to 16-byte stores
    __shared__ uint32_t ring_all[4][128 * ES];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    copy_to_lds(mt + kMtInv2, tab2, kTab2 / 64, wave, lane);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // the only workgroup barrier
    // columns in reverse order: the row stage before this pass wrote the last documents'
    // rows most recently, so part of them is still in the last-level cache (measured:
    // 5% faster than ascending order on the mid-length workload)
    const int task = (static_cast<int>(gridDim.x) - 1 - static_cast<int>(blockIdx.x)) * 4 + wave;
    if (task >= ntasks) return;
    const int col = task / npb, pb = task - col * npb;
    const Seg* sg = t.segs + t.col_seg[col];
    const int j = col - sg->col0, m = sg->m, len = sg->len;
    const int p = lane & 15, h = lane >> 4;
    uint32_t* ring = ring_all[wave];

    // stage 1 per k1: conjugate twiddle on the input, DFT over k2 -> n2.  All grid
    // loads are issued first; w_P^(u j) = w_P^(k1 j) * w_P^(16 k2 j) with k2 = 4i + h.
    const __amdgpu_buffer_rsrc_t rt = doc_buffer(t.tw + sg->twf_off, static_cast<uint32_t>(sg->P) * 8);
    const uint32_t* gdoc = grid + pb * grid_pb_stride + sg->grid_off * kPairsPerBlock;
    const int64_t grid_bytes = static_cast<int64_t>(sg->P) * kPairsPerBlock * 4;
    const uint32_t g_lane = (static_cast<uint32_t>(j) * kPairsPerBlock + p) * 4;
    uint32_t ld_lane[4];  // grid row u = k1 + 16 k2, k2 = 4 i + h: lane part of 16 k2
#pragma unroll
    for (int i = 0; i < 4; ++i)
        ld_lane[i] = static_cast<uint32_t>(16 * (4 * i + h)) * m * (kPairsPerBlock * 4) + g_lane;
    u4 yg[16];
#pragma unroll
    for (int k1 = 0; k1 < 16; ++k1) {
        const __amdgpu_buffer_rsrc_t rg =
            sub_buffer(gdoc, grid_bytes, static_cast<int64_t>(k1) * m * (kPairsPerBlock * 4));
#pragma unroll
        for (int i = 0; i < 4; ++i)
            yg[k1][i] = __builtin_amdgcn_raw_buffer_load_b32(rg, static_cast<int>(ld_lane[i]), 0, 0);
    }
    uint32_t tw_lane[4];  // complex fp16, conjugated
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const auto w = __builtin_amdgcn_raw_buffer_load_b64(
            rt, static_cast<int>(16u * (4 * i + h) * j * 8), 0, 0);
        tw_lane[i] = h2_bits(__uint_as_float(w[0]), -__uint_as_float(w[1]));
    }
    const u4 are1 = mt[kMtInv1 + lane];
    const u4 aim1 = mt[kMtInv1 + 64 + lane];
    const float2* twf = t.tw + sg->twf_off;
    // undoes the range scales of this lane's pair on the fp32 outputs
    const float out_mul = sc.pair[pb * kPairsPerBlock + p].y * sc.glob->y;
    __builtin_amdgcn_sched_barrier(0);

    uint32_t z[16][4];
#pragma unroll
    for (int k1 = 0; k1 < 16; ++k1) {
        const float2 tkf = cscale(cconj(twf[k1 * j]), 16.0f);  // wave-uniform
        const uint32_t tk = h2_bits(tkf.x, tkf.y);
        u4 b;
#pragma unroll
        for (int i = 0; i < 4; ++i) b[i] = cmul_h2(cmul_h2(yg[k1][i], tk), tw_lane[i]);
        const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
        const f4 dre = mma_f16(are1, b, zero);
        const f4 dim = mma_f16(aim1, b, zero);
#pragma unroll
        for (int r = 0; r < 4; ++r) z[k1][r] = pack_h2(dre[r], dim[r]);
    }
    // z[k1][r] = Z[k1][n2 = 4h + r]; regroup so that lane group h holds k1 = 4h + r'
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int rp = 0; rp < 4; ++rp)
            lanegroup_transpose(z[rp][r], z[4 + rp][r], z[8 + rp][r], z[12 + rp][r]);

    char* doc = static_cast<char*>(dst) + (static_cast<int64_t>(sg->row) * dst_row_stride +
                                           static_cast<int64_t>(sg->start) * D) * ES;
    const int64_t doc_bytes = static_cast<int64_t>(len) * D * ES;
    // 16-byte stores of the group of 16 tokens m (16 n1 + n2) + j, n1 < 16: lane l writes
    // token n1 = l / LPT (LPT lanes per token) at channel pair QPL (l % LPT) + ...
    constexpr int LPT = 4 * ES / 2;         // lanes per token: 64 B (bf16) or 128 B (fp32)
    constexpr int QPL = 16 / LPT;           // pairs per lane: 4 (bf16) or 2 (fp32)
    constexpr int ROUNDS = ES / 2;          // 16 tokens x 16 pairs take 1 or 2 instructions
    uint32_t st_lane[ROUNDS];
#pragma unroll
    for (int q = 0; q < ROUNDS; ++q) {
        const int n1 = (q * 64 + lane) / LPT;
        st_lane[q] = (static_cast<uint32_t>(m) * 16u * n1 * D +
                      2 * (pb * kPairsPerBlock + QPL * ((q * 64 + lane) % LPT))) * ES;
    }
    // fp32 outputs: the scales of the QPL = 2 pairs a lane stores (the same in both rounds)
    float st_mul[2] = {1.0f, 1.0f};
    if constexpr (std::is_same<TY, F32>::value) {
#pragma unroll
        for (int c = 0; c < 2; ++c)
            st_mul[c] = sc.pair[pb * kPairsPerBlock + QPL * (lane % LPT) + c].y * sc.glob->y;
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int n2 = 4 * g + r;
            const u4 b = {z[4 * g][r], z[4 * g + 1][r], z[4 * g + 2][r], z[4 * g + 3][r]};
            const u4 are = tab2[(2 * n2) * 64 + lane];
            const u4 aim = tab2[(2 * n2 + 1) * 64 + lane];
            const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
            const f4 dre = mma_f16(are, b, zero);
            const f4 dim = mma_f16(aim, b, zero);
            // register r2 of lane (p, h) is token n1 = 4 r2 + h of this n2, pair p
#pragma unroll
            for (int r2 = 0; r2 < 4; ++r2) {
                const int e = (4 * r2 + h) * 16 + p;  // [n1][pair]
                if constexpr (std::is_same<TY, F32>::value) {
                    // fp32 outputs go to LDS as the products left them; the scale is applied
                    // after the round trip (below): a multiply here, between the products and
                    // the LDS stores, gave 4-5% errors on this variant (see the design notes)
                    *reinterpret_cast<u2*>(ring + 2 * e) = u2{__float_as_uint(dre[r2]), __float_as_uint(dim[r2])};
                } else {
                    ring[e] = pack_bf2(dre[r2] * out_mul, dim[r2] * out_mul);
                }
            }
            wave_lds_fence();
            const __amdgpu_buffer_rsrc_t rs =
                sub_buffer(doc, doc_bytes, static_cast<int64_t>(m * n2 + j) * D * ES);
#pragma unroll
            for (int q = 0; q < ROUNDS; ++q) {
                u4 v = *reinterpret_cast<const u4*>(ring + (q * 64 + lane) * 4);
                if constexpr (std::is_same<TY, F32>::value) {
#pragma unroll
                    for (int c = 0; c < 4; ++c) v[c] = __float_as_uint(__uint_as_float(v[c]) * st_mul[c / 2]);
                }
                __builtin_amdgcn_raw_buffer_store_b128(v, rs, static_cast<int>(st_lane[q]), 0, 0);
            }
            wave_lds_fence();  // the ring is rewritten for the next n2
        }
    }
}

}  // namespace

hipError_t launch_col_fwd_mfma(int src_dtype, const void* src, int64_t src_row_stride, int D,
                               void* grid, int64_t grid_pb_stride, const LaunchTables& t,
                               GridScale sc, const void* mtab, int n_cols, int npb,
                               hipStream_t stream, uint16_t* amax_out, const uint16_t* amax_in,
                               float2* used, float first_scale, float* hint, float extra,
                               const float2* prev) {
    if (n_cols == 0) return hipSuccess;
    if ((amax_out != nullptr || amax_in != nullptr) && src_dtype != 1) return hipErrorInvalidValue;
    if (amax_out != nullptr && amax_in != nullptr) return hipErrorInvalidValue;
    if (amax_in != nullptr && (used == nullptr || (reinterpret_cast<uintptr_t>(amax_in) & 15) != 0))
        return hipErrorInvalidValue;
    const int ntasks = n_cols * npb;
    // the redo launch mostly does nothing: 1024 workgroups (four per CU) that loop over the
    // tasks start and leave faster than one workgroup per four tasks.  Its magnitudes are
    // those of the first launch, one per workgroup of that launch (wgs)
    const int wgs = (ntasks + 3) / 4;
    const dim3 g(amax_in != nullptr ? std::min(wgs, 1024) : wgs), b(256);
    const u4* mt = static_cast<const u4*>(mtab);
    uint32_t* gp = static_cast<uint32_t*>(grid);
    if (src_dtype == 1 && amax_out != nullptr)
        hipLaunchKernelGGL((col_fwd_mfma_kernel<kBf16In, true>), g, b, 0, stream, src, src_row_stride, D, gp,
                           grid_pb_stride, t, sc, mt, npb, ntasks, amax_out, amax_in, wgs, used, first_scale, hint,
                           extra, prev);
    else if (src_dtype == 1)
        hipLaunchKernelGGL((col_fwd_mfma_kernel<kBf16In, false>), g, b, 0, stream, src, src_row_stride, D, gp,
                           grid_pb_stride, t, sc, mt, npb, ntasks, amax_out, amax_in, wgs, used, first_scale, hint,
                           extra, prev);
    else
        hipLaunchKernelGGL((col_fwd_mfma_kernel<kF16In, false>), g, b, 0, stream, src, src_row_stride, D, gp,
                           grid_pb_stride, t, sc, mt, npb, ntasks, amax_out, amax_in, wgs, used, first_scale, hint,
                           extra, prev);
    return hipGetLastError();
}

hipError_t launch_col_inv_mfma(int y_dtype, const void* grid, int64_t grid_pb_stride, void* dst,
                               int64_t dst_row_stride, int D, const LaunchTables& t,
                               GridScale sc, const void* mtab, int n_cols, int npb,
                               hipStream_t stream) {
    if (n_cols == 0) return hipSuccess;
    const int ntasks = n_cols * npb;
    const dim3 g((ntasks + 3) / 4), b(256);
    const u4* mt = static_cast<const u4*>(mtab);
    const uint32_t* gp = static_cast<const uint32_t*>(grid);
    if (y_dtype == 1)
        hipLaunchKernelGGL(col_inv_mfma_kernel<BF16>, g, b, 0, stream, gp, grid_pb_stride, dst,
                           dst_row_stride, D, t, sc, mt, npb, ntasks);
    else
        hipLaunchKernelGGL(col_inv_mfma_kernel<F32>, g, b, 0, stream, gp, grid_pb_stride, dst,
                           dst_row_stride, D, t, sc, mt, npb, ntasks);
    return hipGetLastError();
}

}  // namespace rubiconv
