// row_dense.hip -- row pass on the matrix cores for complex fp16 grids, m <= 128.
//
// Algorithm 1's block-diagonal second DFT applies an m-point DFT to every grid
// row of a document.  For m <= 16 * NB this kernel applies it as one dense
// complex matrix product on v_mfma_f32_16x16x32_f16: NB x NB blocks of 16 x 16,
// each block the two real 16 x 32 operands [Re | -Im] and [Im | Re] against
// the row's 16 channel pairs (K interleaves real and imaginary parts).  The
// output layout of a product (lane group h holds rows 4h..4h+3 of a block) is
// the input layout of the next (lane group h holds K = 8h..8h+7, i.e. slots
// 4h..4h+3), so the forward transform, the spectral product and the inverse
// transform chain without any lane exchange.  Frequencies keep their natural
// order in the slots; time points are interleaved (slot 4h + t holds point
// 4t + h, folded into the operand tables) so that each load and store
// instruction covers four neighbouring grid points.
//
// One wave handles grid row u (0 <= u <= N1/2) of one document and its
// conjugate partner row ub = (N1 - u) mod N1, for one block of 16 pairs: the
// filter-class rows and the data rows of both are transformed, row ub's two
// spectra are brought to the lanes of the matching frequencies of row u (through
// LDS for rows of up to 32 points, by the transform itself for longer rows, see
// row_partner_kernel), and for each frequency f of row u the wave forms, from
// a = Z(f), b = Z(-f), A = F(f), Bf = F(-f) (Z data pair, F filter pair), the
// separated product of Algorithm 3 for both f and -f:
//   s = a + conj b, d = a - conj b, U = s - i d, V = s + i d,
//   4 W(f) = A U + conj(Bf) V,   4 W(-f) = conj(conj(Bf) U + A V),
// where W = X_d H_d + i X_(d+1) H_(d+1) is the spectrum of the output pair.  The
// frequency -f of f = u + N1 v sits in row ub at column (-v - [u > 0]) mod m.
// W(-f) feeds row ub's inverse transform; the inverse of both rows is written
// back over the grid rows.
//
// Scaling: the forward operands carry 1 / sqrt(m), so the product carries the
// 1 / m of the inverse row DFT; the inverse operands carry sqrt(N1) / 4 (the
// 1/4 of the two separations, and the sqrt(N1) that undoes the filter grid's
// 1 / sqrt(N1) column scaling), leaving the inverse column pass's 1 / sqrt(N1).
//
// Rows are read and written through buffer resources that cover exactly one
// row: the padded points of the last block read zeros and write nothing.  Row
// data is touched once, so it is loaded and stored non-temporally (cache policy
// nt).  The operand tables of a size class go to LDS once per workgroup, whose
// waves take consecutive rows of one document.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.hpp"
#include "pk_half.hpp"

namespace rubiconv {

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kPad = 16;    // LDS slots in front of a row: partner reads of padded points

__device__ __forceinline__ f4 mma(u4 a, u4 b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a),
                                                  __builtin_bit_cast(h8, b), c, 0, 0, 0);
}
__device__ __forceinline__ uint32_t pack_h2(float re, float im) {
    return __builtin_bit_cast(uint32_t, __float22half2_rn(make_float2(re, im)));
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_buffer(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes),
                                             0x00020000);
}

// Complex fp16 pairs (low half real, high half imaginary) on the packed-half ALU.
// op_sel picks the source halves of the low result, op_sel_hi those of the high
// result; neg_lo / neg_hi negate a source in the low / high result.
__device__ __forceinline__ uint32_t pk_add_conj(uint32_t a, uint32_t b) {  // a + conj b
    uint32_t r;
    asm("v_pk_add_f16 %0, %1, %2 neg_hi:[0,1]" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ uint32_t pk_swap_add_conj(uint32_t a, uint32_t b) {
    // (a.im + b.im, a.re - b.re)
    uint32_t r;
    asm("v_pk_add_f16 %0, %1, %2 op_sel:[1,1] op_sel_hi:[0,0] neg_hi:[0,1]" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ uint32_t pk_add_neg_hi(uint32_t a, uint32_t b) {  // (a.x + b.x, a.y - b.y)
    uint32_t r;
    asm("v_pk_add_f16 %0, %1, %2 neg_hi:[0,1]" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ uint32_t pk_add(uint32_t a, uint32_t b) {  // a + b
    uint32_t r;
    asm("v_pk_add_f16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}
__device__ __forceinline__ uint32_t pk_add_neg_lo(uint32_t a, uint32_t b) {  // (a.x - b.x, a.y + b.y)
    uint32_t r;
    asm("v_pk_add_f16 %0, %1, %2 neg_lo:[0,1]" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// 4 W(f) = A U + conj(Bf) V
__device__ __forceinline__ uint32_t w_pos(uint32_t A, uint32_t Bf, uint32_t U, uint32_t V) {
    uint32_t t;
    asm("v_pk_mul_f16 %0, %1, %2 op_sel_hi:[0,1]" : "=v"(t) : "v"(A), "v"(U));
    asm("v_pk_fma_f16 %0, %1, %2, %0 op_sel:[1,1,0] op_sel_hi:[1,0,1] neg_lo:[1,0,0]"
        : "+v"(t) : "v"(A), "v"(U));
    asm("v_pk_fma_f16 %0, %1, %2, %0 op_sel_hi:[0,1,1]" : "+v"(t) : "v"(Bf), "v"(V));
    asm("v_pk_fma_f16 %0, %1, %2, %0 op_sel:[1,1,0] op_sel_hi:[1,0,1] neg_hi:[1,0,0]"
        : "+v"(t) : "v"(Bf), "v"(V));
    return t;
}
// 4 W(-f) = conj(conj(Bf) U + A V)
__device__ __forceinline__ uint32_t w_neg(uint32_t A, uint32_t Bf, uint32_t U, uint32_t V) {
    uint32_t t;
    asm("v_pk_mul_f16 %0, %1, %2 op_sel_hi:[0,1] neg_hi:[1,0]" : "=v"(t) : "v"(Bf), "v"(U));
    asm("v_pk_fma_f16 %0, %1, %2, %0 op_sel:[1,1,0] op_sel_hi:[1,0,1]" : "+v"(t) : "v"(Bf), "v"(U));
    asm("v_pk_fma_f16 %0, %1, %2, %0 op_sel_hi:[0,1,1] neg_hi:[1,0,0]" : "+v"(t) : "v"(A), "v"(V));
    asm("v_pk_fma_f16 %0, %1, %2, %0 op_sel:[1,1,0] op_sel_hi:[1,0,1] neg_lo:[1,0,0] neg_hi:[1,0,0]"
        : "+v"(t) : "v"(A), "v"(V));
    return t;
}

// ---------------------------------------------------------------------------
// Variant for short rows (m <= 32): every memory access is 16 bytes per lane.
// The time and frequency layouts, the products and the LDS exchange are those of
// row_dense_kernel; what differs is how data reaches the matrix cores:
//   - a workgroup's waves take consecutive rows u of one document, so the class's
//     operand tables are copied into LDS once per workgroup;
//   - the four input rows are copied straight into LDS (buffer loads with the lds
//     modifier, 16 bytes per lane) and read from there in the operand layout;
//   - the two output rows are staged in LDS and written with 16-byte stores.
// The vector memory instructions per row pair drop from 16 NB + 8 NB (+ table
// fragments) to 6 NB, which is what bounds the short-row launches.
constexpr int kLdsWaves = 8;  // rows u of one document per workgroup

template <int NB>
struct RowInputs {  // one pair block's four rows in MFMA input layout
    u4 fu[NB], fb[NB], xu[NB], xb[NB];
};

struct RowBuffers {  // buffer resources of one pair block's rows u and ub
    __amdgpu_buffer_rsrc_t du, db, fu, fb;
};

__device__ __forceinline__ RowBuffers row_buffers(uint32_t* grid, int64_t grid_pb_stride,
                                                  const uint32_t* fgrid, int64_t fgrid_pb_stride,
                                                  const Seg* sg, int pb, int u, int ub) {
    const int m = sg->m;
    const uint32_t row_bytes = static_cast<uint32_t>(m) * 64;
    uint32_t* drow = grid + pb * grid_pb_stride + sg->grid_off * 16;
    const uint32_t* frow = fgrid + pb * fgrid_pb_stride + static_cast<int64_t>(sg->spec_off) * 16;
    return {row_buffer(drow + static_cast<int64_t>(u) * m * 16, row_bytes),
            row_buffer(drow + static_cast<int64_t>(ub) * m * 16, row_bytes),
            row_buffer(frow + static_cast<int64_t>(u) * m * 16, row_bytes),
            row_buffer(frow + static_cast<int64_t>(ub) * m * 16, row_bytes)};
}

__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// s_waitcnt immediate that waits until at most n vector memory operations are
// outstanding and leaves the other counters alone (vmcnt in bits 3:0 and 15:14)
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// 16 bytes per lane from buffer offset voffset (lane part) to LDS at lds + 16 * lane
__device__ __forceinline__ void lds_copy16(__amdgpu_buffer_rsrc_t rs, int voffset, void* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(lds), 16,
                                             voffset, 0, 0, 0);
}

template <int NB, bool SUM>
__global__ __launch_bounds__(64 * kLdsWaves) void row_lds_kernel(uint32_t* __restrict__ grid,
                                                               int64_t grid_pb_stride,
                                                               const uint32_t* __restrict__ fgrid,
                                                               int64_t fgrid_pb_stride,
                                                               const Seg* __restrict__ segs,
                                                               const int32_t* __restrict__ docs,
                                                               const int2* __restrict__ groups,
                                                               const u4* __restrict__ tabs, int n1,
                                                               int corr, float dscale, int out2) {
    constexpr int S = 16 * NB;                     // points per row, padded to whole blocks
    constexpr int kTabU4 = 4 * NB * NB * 64;       // forward then inverse fragments
    constexpr int kStage = 4 * S * 16;             // u32 per wave: four rows [point][16 pairs]
    static_assert(kStage >= 2 * (kPad + S) * 16, "the exchange rows reuse the staging area");
    __shared__ u4 tab[kTabU4];
    __shared__ uint32_t stage_all[kLdsWaves][kStage];

    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    const int p = lane & 15, h = lane >> 4;
    const int nu = n1 / 2 + 1;
    const int ug = (nu + kLdsWaves - 1) / kLdsWaves;
    // a group: documents of one size class, sharing the filter rows of the first
    const int2 grp = groups[blockIdx.x / ug];
    const Seg* sg = segs + docs[grp.x];
    const int u = (blockIdx.x % ug) * kLdsWaves + wave;
    const bool active = u < nu;  // wave-uniform
    const int m = sg->m;
    const int pb = blockIdx.y;
    uint32_t* stage = stage_all[wave];
    const bool pad = (NB - 1) * 16 * 64 + lane * 16 >= m * 64;  // this lane's copy was out of range

    // the class's operand tables, 1 KB per wave instruction
    {
        const __amdgpu_buffer_rsrc_t rt = row_buffer(tabs + sg->dense_off, kTabU4 * 16);
        for (int c = wave; c < kTabU4 / 64; c += kLdsWaves) lds_copy16(rt, c * 1024 + lane * 16, &tab[c * 64]);
    }
    const int ub = u == 0 ? 0 : n1 - u;  // n1 need not be a power of two (sub-row documents)
    RowBuffers rb = row_buffers(grid, grid_pb_stride, fgrid, fgrid_pb_stride, sg, pb, u, ub);
    // the four rows [fu, fb, xu, xb] as [point][16 pairs], 16 points per instruction
    if (active) {
#pragma unroll
        for (int jb = 0; jb < NB; ++jb) {
            const int off = jb * 1024 + lane * 16;
            lds_copy16(rb.fu, off, stage + 0 * S * 16 + jb * 256);
            lds_copy16(rb.fb, off, stage + 1 * S * 16 + jb * 256);
            lds_copy16(rb.du, off, stage + 2 * S * 16 + jb * 256);
            lds_copy16(rb.db, off, stage + 3 * S * 16 + jb * 256);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);  // the copies above have landed in LDS
    if (active && pad) {
        // the copy of points >= m was out of range: make the padding zero
#pragma unroll
        for (int r = 0; r < 4; ++r)
            *reinterpret_cast<u4*>(stage + r * S * 16 + (NB - 1) * 256 + lane * 4) = u4{0u, 0u, 0u, 0u};
    }
    __syncthreads();  // tables visible to every wave; the only workgroup barrier
    if (!active) return;

    // operand layout: register t of lane (p, h) holds point 16 jb + 4 t + h of pair p
    RowInputs<NB> in;
#pragma unroll
    for (int jb = 0; jb < NB; ++jb)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int e = (16 * jb + 4 * t + h) * 16 + p;
            in.fu[jb][t] = stage[0 * S * 16 + e];
            in.fb[jb][t] = stage[1 * S * 16 + e];
            in.xu[jb][t] = stage[2 * S * 16 + e];
            in.xb[jb][t] = stage[3 * S * 16 + e];
        }
    wave_lds_fence();

    // the staging area now holds the two exchange rows (row ub's spectra)
    const int shift = u == 0 ? 1 : 0;
    uint32_t* xlds = stage + kPad * 16 + p;
    uint32_t* flds = stage + (2 * kPad + S) * 16 + p;
    const u4* fwd = tab;
    const u4* inv = tab + 2 * NB * NB * 64;
    const int rbase = m - 1 - 4 * h;

    // forward DFT of rows u and ub: own[kb][r] = frequency 16 kb + 4 h + r of row u;
    // row ub's spectrum to the exchange row dst (slot 16 kb + 4 h + r - shift), and
    // its frequency 0 returned for row 0's wrap
    auto forward = [&](const u4* in_u, const u4* in_b, uint32_t(*own)[4], uint32_t* dst, float sc) {
#pragma unroll
        for (int i = 0; i < kPad / 4; ++i) dst[16 * (4 * i + h - kPad)] = 0u;
        uint32_t keep = 0u;
#pragma unroll
        for (int kb = 0; kb < NB; ++kb) {
            f4 acc[2][2];
#pragma unroll
            for (int i = 0; i < 2; ++i) acc[i][0] = acc[i][1] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int jb = 0; jb < NB; ++jb) {
                const u4 are = fwd[((kb * NB + jb) * 2) * 64 + lane];
                const u4 aim = fwd[((kb * NB + jb) * 2 + 1) * 64 + lane];
                acc[0][0] = mma(are, in_u[jb], acc[0][0]);
                acc[0][1] = mma(aim, in_u[jb], acc[0][1]);
                acc[1][0] = mma(are, in_b[jb], acc[1][0]);
                acc[1][1] = mma(aim, in_b[jb], acc[1][1]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                own[kb][r] = pack_h2(sc * acc[0][0][r], sc * acc[0][1][r]);
                const uint32_t bv = pack_h2(sc * acc[1][0][r], sc * acc[1][1][r]);
                dst[16 * (16 * kb + 4 * h + r - shift)] = bv;
                if (kb == 0 && r == 0) keep = bv;
            }
        }
        if (shift && h == 0) dst[16 * (m - 1)] = keep;  // row 0: point 0 is also slot m - 1
        wave_lds_fence();
    };

    // separated products of one document against its second rows' spectra fa (own) and
    // fl (partner values): W(f) of row u into wu, W(-f) of row ub into the exchange row
    auto products = [&](const uint32_t(*fa)[4], const uint32_t(*fl)[4], const uint32_t(*au)[4],
                        uint32_t(*wu)[4]) {
#pragma unroll
        for (int kb = 0; kb < NB; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int slot = rbase - 16 * kb - r;  // >= -15: inside the zeroed front slots
                const uint32_t b = xlds[16 * slot];
                const uint32_t a = au[kb][r];
                // correlation: the filter spectrum read at -f (its conjugate for real taps)
                const uint32_t A = corr ? fl[kb][r] : fa[kb][r];
                const uint32_t bf = corr ? fa[kb][r] : fl[kb][r];
                const uint32_t e1 = pk_add_conj(a, b);
                const uint32_t e2 = pk_swap_add_conj(a, b);
                const uint32_t U = pk_add_neg_hi(e1, e2);
                const uint32_t V = pk_add_neg_lo(e1, e2);
                wu[kb][r] = w_pos(A, bf, U, V);
                xlds[16 * slot] = w_neg(A, bf, U, V);
            }
        if (shift && h == 0) xlds[-16] = xlds[16 * (m - 1)];
        wave_lds_fence();
    };
    // inverse DFT of rows u (from wu) and ub (from wb) into LDS rows 0 and 1 as
    // [row][point][16 pairs], then 16-byte stores to the rows of rs
    auto inverse_store = [&](const uint32_t(*wu)[4], const u4* wb, const RowBuffers& rs) {
        uint32_t* out = stage;
#pragma unroll
        for (int kb = 0; kb < NB; ++kb) {
            f4 acc[2][2];
#pragma unroll
            for (int i = 0; i < 2; ++i) acc[i][0] = acc[i][1] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int jb = 0; jb < NB; ++jb) {
                const u4 are = inv[((kb * NB + jb) * 2) * 64 + lane];
                const u4 aim = inv[((kb * NB + jb) * 2 + 1) * 64 + lane];
                const u4 win = {wu[jb][0], wu[jb][1], wu[jb][2], wu[jb][3]};
                acc[0][0] = mma(are, win, acc[0][0]);
                acc[0][1] = mma(aim, win, acc[0][1]);
                acc[1][0] = mma(are, wb[jb], acc[1][0]);
                acc[1][1] = mma(aim, wb[jb], acc[1][1]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {  // output register r: time point 16 kb + 4 r + h
                const int e = (16 * kb + 4 * r + h) * 16 + p;
                out[e] = pack_h2(acc[0][0][r], acc[0][1][r]);
                out[S * 16 + e] = pack_h2(acc[1][0][r], acc[1][1][r]);
            }
        }
        wave_lds_fence();
#pragma unroll
        for (int jb = 0; jb < NB; ++jb) {
            const int off = jb * 1024 + lane * 16;
            const u4 vu = *reinterpret_cast<const u4*>(out + jb * 256 + lane * 4);
            const u4 vb = *reinterpret_cast<const u4*>(out + S * 16 + jb * 256 + lane * 4);
            __builtin_amdgcn_raw_buffer_store_b128(vu, rs.du, off, 0, 2);
            __builtin_amdgcn_raw_buffer_store_b128(vb, rs.db, off, 0, 2);
        }
    };

    if constexpr (SUM) {
        // every document brings its own second rows: both spectra per document (the data
        // rows' times dscale), the products added up (packed fp16), one inverse for the
        // group into its first document's rows (rb; with out2, its second rows)
        uint32_t su[NB][4];
        u4 sb[NB];
        for (int k = 0;;) {
            uint32_t fa[NB][4], fl[NB][4];
            forward(in.fu, in.fb, fa, flds, 1.0f);
#pragma unroll
            for (int kb = 0; kb < NB; ++kb)
#pragma unroll
                for (int r = 0; r < 4; ++r) fl[kb][r] = flds[16 * (rbase - 16 * kb - r)];
            wave_lds_fence();  // the second exchange row is free from here on
            uint32_t au[NB][4], wu[NB][4];
            forward(in.xu, in.xb, au, xlds, dscale);
            products(fa, fl, au, wu);
#pragma unroll
            for (int jb = 0; jb < NB; ++jb)
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const uint32_t wbv = xlds[16 * (16 * jb + 4 * h + t - shift)];
                    su[jb][t] = k == 0 ? wu[jb][t] : pk_add(su[jb][t], wu[jb][t]);
                    sb[jb][t] = k == 0 ? wbv : pk_add(sb[jb][t], wbv);
                }
            wave_lds_fence();  // the staging area is free for the next document's rows
            if (++k == grp.y) break;
            const RowBuffers rk = row_buffers(grid, grid_pb_stride, fgrid, fgrid_pb_stride,
                                              segs + docs[grp.x + k], pb, u, ub);
#pragma unroll
            for (int jb = 0; jb < NB; ++jb) {
                const int off = jb * 1024 + lane * 16;
                lds_copy16(rk.fu, off, stage + 0 * S * 16 + jb * 256);
                lds_copy16(rk.fb, off, stage + 1 * S * 16 + jb * 256);
                lds_copy16(rk.du, off, stage + 2 * S * 16 + jb * 256);
                lds_copy16(rk.db, off, stage + 3 * S * 16 + jb * 256);
            }
            __builtin_amdgcn_s_waitcnt(0);  // the copies have landed in LDS
            if (pad) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    *reinterpret_cast<u4*>(stage + r * S * 16 + (NB - 1) * 256 + lane * 4) = u4{0u, 0u, 0u, 0u};
            }
            wave_lds_fence();
#pragma unroll
            for (int jb = 0; jb < NB; ++jb)
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int e = (16 * jb + 4 * t + h) * 16 + p;
                    in.fu[jb][t] = stage[0 * S * 16 + e];
                    in.fb[jb][t] = stage[1 * S * 16 + e];
                    in.xu[jb][t] = stage[2 * S * 16 + e];
                    in.xb[jb][t] = stage[3 * S * 16 + e];
                }
            wave_lds_fence();
        }
        inverse_store(su, sb, out2 ? RowBuffers{rb.fu, rb.fb, rb.fu, rb.fb} : rb);
        return;
    }

    // the filter rows, once per group: own spectrum in registers, and the partner
    // values at the slots the product reads gathered from the exchange row
    uint32_t fa[NB][4], fl[NB][4];
    forward(in.fu, in.fb, fa, flds, 1.0f);
#pragma unroll
    for (int kb = 0; kb < NB; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) fl[kb][r] = flds[16 * (rbase - 16 * kb - r)];
    wave_lds_fence();  // the filter exchange row is free from here on

    for (int k = 0;;) {
        // the group's next document (if any): its two rows into LDS rows 2 and 3, which
        // nothing else uses from here on, while this one is computed
        {
            const bool more = k + 1 < grp.y;
            const RowBuffers nb_rb = row_buffers(grid, grid_pb_stride, fgrid, fgrid_pb_stride,
                                                 segs + docs[grp.x + (more ? k + 1 : k)], pb, u, ub);
            const __amdgpu_buffer_rsrc_t ndu = more ? nb_rb.du : row_buffer(nullptr, 0);
            const __amdgpu_buffer_rsrc_t ndb = more ? nb_rb.db : row_buffer(nullptr, 0);
#pragma unroll
            for (int jb = 0; jb < NB; ++jb) {
                const int off = jb * 1024 + lane * 16;
                lds_copy16(ndu, off, stage + 2 * S * 16 + jb * 256);
                lds_copy16(ndb, off, stage + 3 * S * 16 + jb * 256);
            }
            if (pad) {
#pragma unroll
                for (int r = 2; r < 4; ++r)
                    *reinterpret_cast<u4*>(stage + r * S * 16 + (NB - 1) * 256 + lane * 4) = u4{0u, 0u, 0u, 0u};
            }
            __builtin_amdgcn_sched_barrier(0);  // the copies stay ahead of this document's stores
        }
        uint32_t au[NB][4];
        forward(in.xu, in.xb, au, xlds, 1.0f);

        uint32_t wu[NB][4];
        products(fa, fl, au, wu);

        u4 wb[NB];
#pragma unroll
        for (int jb = 0; jb < NB; ++jb)
#pragma unroll
            for (int t = 0; t < 4; ++t) wb[jb][t] = xlds[16 * (16 * jb + 4 * h + t - shift)];
        wave_lds_fence();

        inverse_store(wu, wb, rb);
        if (++k == grp.y) break;

        // the next document's rows: the copies were issued before this document's 2 NB
        // stores, and the memory counter completes in order
        rb = row_buffers(grid, grid_pb_stride, fgrid, fgrid_pb_stride, segs + docs[grp.x + k], pb, u, ub);
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * NB));
        wave_lds_fence();
#pragma unroll
        for (int jb = 0; jb < NB; ++jb)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int e = (16 * jb + 4 * t + h) * 16 + p;
                in.xu[jb][t] = stage[2 * S * 16 + e];
                in.xb[jb][t] = stage[3 * S * 16 + e];
            }
        wave_lds_fence();
    }
}

// ---------------------------------------------------------------------------
// Rows of 33..128 points (3 to 8 blocks).  Their operand tables are too large to
// stream from the vector cache for every row, and the two LDS exchange rows of the
// short-row kernels would leave room for few waves beside the tables.  So this
// kernel keeps one real operand per block in LDS and produces the partner row's
// spectra directly in the order the separated product needs them:
//   - the imaginary output part comes from the same operand, its halves swapped and
//     one negated (A_re = [Re | -Im] becomes [Im | Re]), halving the tables;
//   - frequencies are interleaved in the slots like the time points, so that each
//     block of the DFT matrix is symmetric and the inverse transform, kappa times the
//     conjugate of the forward one, runs on the same operands: half the tables again;
//   - with w = exp(-2 pi i / m) and T the forward table, row ub's spectrum at the
//     partner column of v is Z(m - 1 - v) = conj(T conj(z(j) w^(-j)))(v) for u > 0,
//     and Z((m - v) mod m) = conj(T conj(z))(v) for row 0, so it lands in the
//     registers of frequency v of row u;
//   - W(-f) of row ub then sits at the slot of v, frequency m - 1 - v, and the row's
//     inverse is y(j) = w^j conj(T_inv conj(G))(j) = kappa w^j (T G)(j) with
//     G(v) = W(m - 1 - v).
// The products and inverses need no lane exchange, so the only LDS is the tables
// and the kernel runs as many waves as its registers allow.  Rows 0 and N1/2 are
// their own partners: their partner spectra come from their own data and only the
// row itself is transformed back and stored.
constexpr int kPartnerWaves = 4;  // rows u of one document per workgroup

// waves per SIMD the registers must allow (the summing variant keeps four loaded rows
// live across its blocks), and at most: rows of 5 or 6 blocks keep their filter spectra,
// a block of both data spectra and the products live at once (164-198 registers), and
// left free to aim at the occupancy their LDS would allow, the compiler's schedule
// spills instead
template <int NB, bool SUM>
constexpr int kPartnerMinWaves = NB <= (SUM ? 2 : 3) ? 4 : NB <= 4 ? 3 : NB <= 6 ? 2 : 1;
template <int NB, bool SUM>
constexpr int kPartnerMaxWaves = (!SUM && NB >= 5 && NB <= 6) ? 2 : 8;

// The operand that gives the imaginary output part from the input itself: an entry v
// held as (Re v, -Im v) becomes (Im v, Re v), so that the product with z sums
// Im v Re z + Re v Im z = Im(v z), as the operand itself does against -i z
__device__ __forceinline__ uint32_t imag_operand(uint32_t a) {
    return __builtin_amdgcn_alignbit(a, a, 16) ^ 0x00008000u;
}
__device__ __forceinline__ u4 imag_operand4(u4 a) {
    return u4{imag_operand(a[0]), imag_operand(a[1]), imag_operand(a[2]), imag_operand(a[3])};
}

template <int NB, bool SUM>
__global__ __launch_bounds__(64 * kPartnerWaves) __attribute__((amdgpu_waves_per_eu(kPartnerMinWaves<NB, SUM>, kPartnerMaxWaves<NB, SUM>)))
void row_partner_kernel(uint32_t* __restrict__ grid, int64_t grid_pb_stride,
                        const uint32_t* __restrict__ fgrid, int64_t fgrid_pb_stride,
                        const Seg* __restrict__ segs, const int32_t* __restrict__ docs,
                        const int2* __restrict__ groups, const u4* __restrict__ tabs, int n1,
                        int corr, float dscale, int out2) {
    constexpr int S = 16 * NB;
    constexpr int kFrag = NB * NB * 64;            // u4 of DFT operands
    constexpr int kTab = partner_tab_u4(NB);
    constexpr bool kPrefetch = NB <= 4;            // first data rows loaded with the filter rows
    __shared__ u4 tab[kTab];

    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    const int p = lane & 15, h = lane >> 4;
    const int nu = n1 / 2 + 1;
    const int ug = (nu + kPartnerWaves - 1) / kPartnerWaves;
    // a group: documents of one size class, sharing the filter rows of the first
    const int2 grp = groups[blockIdx.x / ug];
    const Seg* sg = segs + docs[grp.x];
    const int u = (blockIdx.x % ug) * kPartnerWaves + wave;
    const bool active = u < nu;                    // wave-uniform
    const bool self = u == 0 || 2 * u == n1;       // its own partner row
    const int ub = self ? u : n1 - u;
    const int pb = blockIdx.y;
    RowBuffers rb = row_buffers(grid, grid_pb_stride, fgrid, fgrid_pb_stride, sg, pb, u, ub);

    // register t of lane (p, h) holds point 16 jb + 4 t + h of pair p: one load covers
    // four neighbouring points, 256 contiguous bytes
    const int lane_off = (h * 16 + p) * 4;
    u4 fu[NB], fb[NB], xu[NB], xb[NB];
    auto load_rows = [&](__amdgpu_buffer_rsrc_t ru, __amdgpu_buffer_rsrc_t rbb, u4* du, u4* db) {
#pragma unroll
        for (int jb = 0; jb < NB; ++jb)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int off = lane_off + (16 * jb + 4 * t) * 64;
                du[jb][t] = __builtin_amdgcn_raw_buffer_load_b32(ru, off, 0, 2);
                db[jb][t] = __builtin_amdgcn_raw_buffer_load_b32(rbb, off, 0, 2);
            }
    };
    if (active) {
        load_rows(rb.fu, rb.fb, fu, fb);
        if constexpr (kPrefetch) load_rows(rb.du, rb.db, xu, xb);
    }
    {  // the class's tables, 1 KB per wave instruction
        const __amdgpu_buffer_rsrc_t rt = row_buffer(tabs + sg->dense_off, kTab * 16);
        for (int c = wave; c < kTab / 64; c += kPartnerWaves) lds_copy16(rt, c * 1024 + lane * 16, &tab[c * 64]);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // tables visible to every wave; the only workgroup barrier
    if (!active) return;

    const uint32_t* tw_pre = reinterpret_cast<const uint32_t*>(tab + kFrag);  // w^(-j), fp16
    const float2* tw_post = reinterpret_cast<const float2*>(tab + kFrag + S / 4);  // kappa w^j
    const float kappa = reinterpret_cast<const float*>(tab + kFrag + 3 * S / 4)[0];
    // rows u > 0 pair v with m - 1 - v and take the twiddle, row 0 pairs v with (m - v) mod m
    const int pre_mask = u != 0 ? -1 : 0;

    // forward DFT of rows u and ub: own[kb][r] and par[kb][r] hold frequency
    // v = 16 kb + 4 h + r of row u and the partner value of row ub
    // lk: the lane index through an empty asm statement, so that table reads indexed by
    // it are issued where they are used rather than hoisted out of the document loop
    // (which would hold every operand fragment in registers across the loop)
    auto forward = [&](u4* in_u, u4* in_b, uint32_t(*own)[4], uint32_t(*par)[4], int lk) {
        // partner input conj(z(j) w^(-j)); row 0 reads entry 0, w^0 = 1, for every j
#pragma unroll
        for (int jb = 0; jb < NB; ++jb)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const uint32_t tw = tw_pre[(16 * jb + 4 * t + (lk >> 4)) & pre_mask];
                in_b[jb][t] = cmul_h2(in_b[jb][t], tw) ^ 0x80000000u;
            }
#pragma unroll
        for (int kb = 0; kb < NB; ++kb) {
            f4 acc[4];  // own re, own im, partner re, partner im
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int jb = 0; jb < NB; ++jb) {
                const u4 a = tab[(kb * NB + jb) * 64 + lk];
                const u4 ai = imag_operand4(a);
                acc[0] = mma(a, in_u[jb], acc[0]);
                acc[1] = mma(ai, in_u[jb], acc[1]);
                acc[2] = mma(a, in_b[jb], acc[2]);
                acc[3] = mma(ai, in_b[jb], acc[3]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                own[kb][r] = pack_h2(acc[0][r], acc[1][r]);
                par[kb][r] = pack_h2(acc[2][r], -acc[3][r]);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    // separated products of one block of four frequencies: conj W(f) for row u into wu,
    // W(-f) for row ub at the slot of f into wp (G, see inverse_store)
    auto products_block = [&](const uint32_t* fa, const uint32_t* fp, const uint32_t* au,
                              const uint32_t* ap, uint32_t* wu, uint32_t* wp) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t a = au[r], b = ap[r];
            // correlation: the filter spectrum read at -f (its conjugate for real taps)
            const uint32_t A = corr ? fp[r] : fa[r];
            const uint32_t Bf = corr ? fa[r] : fp[r];
            const uint32_t e1 = pk_add_conj(a, b);       // s
            const uint32_t e2 = pk_swap_add_conj(a, b);  // (Im d, Re d)
            const uint32_t U = pk_add_neg_hi(e1, e2);    // s - i d
            const uint32_t V = pk_add_neg_lo(e1, e2);    // s + i d
            wu[r] = w_pos(A, Bf, U, V) ^ 0x80000000u;
            wp[r] = w_neg(A, Bf, U, V);
        }
    };
    // forward DFT of the data rows u and ub, block by block, each block's products
    // with the filter spectra fa / fp formed before the next block
    auto forward_products = [&](const u4* in_u, u4* in_b, const uint32_t(*fa)[4], const uint32_t(*fp)[4],
                                uint32_t(*wu)[4], uint32_t(*wp)[4], int lk) {
#pragma unroll
        for (int jb = 0; jb < NB; ++jb)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const uint32_t tw = tw_pre[(16 * jb + 4 * t + (lk >> 4)) & pre_mask];
                in_b[jb][t] = cmul_h2(in_b[jb][t], tw) ^ 0x80000000u;
            }
#pragma unroll
        for (int kb = 0; kb < NB; ++kb) {
            f4 acc[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int jb = 0; jb < NB; ++jb) {
                const u4 a = tab[(kb * NB + jb) * 64 + lk];
                const u4 ai = imag_operand4(a);
                acc[0] = mma(a, in_u[jb], acc[0]);
                acc[1] = mma(ai, in_u[jb], acc[1]);
                acc[2] = mma(a, in_b[jb], acc[2]);
                acc[3] = mma(ai, in_b[jb], acc[3]);
            }
            uint32_t au[4], ap[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                au[r] = pack_h2(acc[0][r], acc[1][r]);
                ap[r] = pack_h2(acc[2][r], -acc[3][r]);
            }
            products_block(fa[kb], fp[kb], au, ap, wu[kb], wp[kb]);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    // inverse DFT of row u and of row ub into the rows of rs, through the forward
    // operands: the inverse matrix is kappa conj(T), so row u's output is
    // kappa conj(T conj W) (wu holds conj W) and row ub's is kappa w^j (T G)(j), the
    // partner form of the forward section above.  A row that is its own partner stores
    // only the first: the second goes through a buffer resource of no bytes.  The code
    // has no branch between the matrix products and the reads of their results, so the
    // compiler's wait states after the products hold on every path.
    auto inverse_store = [&](const uint32_t(*wu)[4], const uint32_t(*wp)[4], const RowBuffers& rs, int lk) {
        // the operands are those of the forward transform: the lane index passes through
        // an empty asm statement again so that the compiler does not keep the forward
        // fragments live for reuse here
        asm volatile("" : "+v"(lk));
        const __amdgpu_buffer_rsrc_t rdb = self ? row_buffer(nullptr, 0) : rs.db;
#pragma unroll
        for (int kb = 0; kb < NB; ++kb) {
            f4 acc[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int jb = 0; jb < NB; ++jb) {
                const u4 a = tab[(kb * NB + jb) * 64 + lk];
                const u4 ai = imag_operand4(a);
                const u4 bu = {wu[jb][0], wu[jb][1], wu[jb][2], wu[jb][3]};
                const u4 bp = {wp[jb][0], wp[jb][1], wp[jb][2], wp[jb][3]};
                acc[0] = mma(a, bu, acc[0]);
                acc[1] = mma(ai, bu, acc[1]);
                acc[2] = mma(a, bp, acc[2]);
                acc[3] = mma(ai, bp, acc[3]);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {  // output register r: time point j = 16 kb + 4 r + h
                const int off = lane_off + (16 * kb + 4 * r) * 64;
                __builtin_amdgcn_raw_buffer_store_b32(pack_h2(kappa * acc[0][r], -kappa * acc[1][r]), rs.du,
                                                      off, 0, 2);
                // kappa w^j (R + i I) with kappa w^j = (c, s): (R c - I s, R s + I c)
                const float2 w = tw_post[16 * kb + 4 * r + (lk >> 4)];
                const float re = acc[2][r] * w.x - acc[3][r] * w.y;
                const float im = acc[2][r] * w.y + acc[3][r] * w.x;
                __builtin_amdgcn_raw_buffer_store_b32(pack_h2(re, im), rdb, off, 0, 2);
            }
        }
    };

    if constexpr (SUM) {
        // every document brings its own second rows: both spectra per document (the data
        // rows' times dscale), the products added up (packed fp16), one inverse for the
        // group into its first document's rows (with out2, its second rows).  Block kb of
        // all four spectra is formed and multiplied before the next, so that only the
        // loaded rows and the sums stay live across blocks.
        const RowBuffers r0 = rb;
        uint32_t su[NB][4], sp[NB][4];
        for (int k = 0;;) {
            if (!kPrefetch && k == 0) load_rows(rb.du, rb.db, xu, xb);
            int lk = lane;
            asm volatile("" : "+v"(lk));
            // partner inputs conj(z(j) w^(-j)) of both row pairs (row 0: w^0 = 1)
#pragma unroll
            for (int jb = 0; jb < NB; ++jb)
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const uint32_t tw = tw_pre[(16 * jb + 4 * t + (lk >> 4)) & pre_mask];
                    fb[jb][t] = cmul_h2(fb[jb][t], tw) ^ 0x80000000u;
                    xb[jb][t] = cmul_h2(xb[jb][t], tw) ^ 0x80000000u;
                }
#pragma unroll
            for (int kb = 0; kb < NB; ++kb) {
                f4 acc[8];  // second rows: own re, im, partner re, im; then the data rows alike
#pragma unroll
                for (int i = 0; i < 8; ++i) acc[i] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int jb = 0; jb < NB; ++jb) {
                    // the imaginary parts through the rotated operand: no -i copies of the
                    // four loaded rows stay live across blocks
                    const u4 a = tab[(kb * NB + jb) * 64 + lk];
                    const u4 ai = imag_operand4(a);
                    acc[0] = mma(a, fu[jb], acc[0]);
                    acc[1] = mma(ai, fu[jb], acc[1]);
                    acc[2] = mma(a, fb[jb], acc[2]);
                    acc[3] = mma(ai, fb[jb], acc[3]);
                    acc[4] = mma(a, xu[jb], acc[4]);
                    acc[5] = mma(ai, xu[jb], acc[5]);
                    acc[6] = mma(a, xb[jb], acc[6]);
                    acc[7] = mma(ai, xb[jb], acc[7]);
                }
                uint32_t fa[1][4], fp[1][4], au[1][4], ap[1][4], wu[1][4], wp[1][4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    fa[0][r] = pack_h2(acc[0][r], acc[1][r]);
                    fp[0][r] = pack_h2(acc[2][r], -acc[3][r]);
                    au[0][r] = pack_h2(dscale * acc[4][r], dscale * acc[5][r]);
                    ap[0][r] = pack_h2(dscale * acc[6][r], -dscale * acc[7][r]);
                }
                products_block(fa[0], fp[0], au[0], ap[0], wu[0], wp[0]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    su[kb][r] = k == 0 ? wu[0][r] : pk_add(su[kb][r], wu[0][r]);
                    sp[kb][r] = k == 0 ? wp[0][r] : pk_add(sp[kb][r], wp[0][r]);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
            if (++k == grp.y) break;
            rb = row_buffers(grid, grid_pb_stride, fgrid, fgrid_pb_stride, segs + docs[grp.x + k], pb, u, ub);
            load_rows(rb.fu, rb.fb, fu, fb);
            load_rows(rb.du, rb.db, xu, xb);
        }
        int lk = lane;
        asm volatile("" : "+v"(lk));
        inverse_store(su, sp, out2 ? RowBuffers{r0.fu, r0.fb, r0.fu, r0.fb} : r0, lk);
        return;
    }

    // the filter rows, once per group
    uint32_t fa[NB][4], fp[NB][4];
    forward(fu, fb, fa, fp, lane);

    for (int k = 0;;) {
        if (!kPrefetch || k > 0) load_rows(rb.du, rb.db, xu, xb);
        int lk = lane;
        asm volatile("" : "+v"(lk));
        // the data rows' spectra block by block, each block's separated products formed
        // at once (conj W(f) for row u, W(-f) for row ub at the slot of f), so that only
        // one block of the two spectra is live
        uint32_t wu[NB][4], wp[NB][4];
        forward_products(xu, xb, fa, fp, wu, wp, lk);
        inverse_store(wu, wp, rb, lk);
        if (++k == grp.y) break;
        rb = row_buffers(grid, grid_pb_stride, fgrid, fgrid_pb_stride, segs + docs[grp.x + k], pb, u, ub);
    }
}

// ---------------------------------------------------------------------------
// Rows of at most kMaxBatchM points (one 16-point block): R = 16 / m documents of a
// group sit side by side in the block, document r at slots r m .. r m + m - 1 of both
// the time and the frequency axis, and block-diagonal tables transform them together;
// the per-row work of the short-row kernel is then shared by R documents.  Each lane
// register reads its point from the grids of its own document (4 bytes per lane: the
// 16 lanes of a lane group cover one 64-byte grid point) and writes it back the same
// way, and each document's second rows are its own (Seg::spec_off), so one group may
// mix second grids (the filter gradient).  Row 0, whose partner columns wrap inside
// the row, keeps one document per block and the plain tables; rows that are their own
// partners store one row.
constexpr int kBatchWaves = 8;

__global__ __launch_bounds__(64 * kBatchWaves) void row_batch_kernel(uint32_t* __restrict__ grid,
                                                                    int64_t grid_pb_stride,
                                                                    const uint32_t* __restrict__ fgrid,
                                                                    int64_t fgrid_pb_stride,
                                                                    const Seg* __restrict__ segs,
                                                                    const int32_t* __restrict__ docs,
                                                                    const int2* __restrict__ groups,
                                                                    const u4* __restrict__ tabs, int n1,
                                                                    int corr) {
    constexpr int kTabU4 = 4 * 64;                   // one table set: forward then inverse
    constexpr uint32_t kNone = 0xffffffffu;          // an offset outside every buffer
    constexpr int kGroupCap = kMaxGroupDocs * 16;    // documents of a group (16 / m per block)
    __shared__ u4 tab[2 * kTabU4];                   // plain tables, then block-diagonal ones
    __shared__ uint32_t xch_all[kBatchWaves][2 * (kPad + 16) * 16];
    // the group's grid and second-grid offsets, read once per workgroup, so that a lane
    // finds its document's rows in LDS rather than through two dependent global loads
    __shared__ int64_t g_off[kGroupCap];
    __shared__ int32_t s_off[kGroupCap];

    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    const int p = lane & 15, h = lane >> 4;
    const int nu = n1 / 2 + 1;
    const int ug = (nu + kBatchWaves - 1) / kBatchWaves;
    const int2 grp = groups[blockIdx.x / ug];
    const int m = segs[docs[grp.x]].m;
    const int u = (blockIdx.x % ug) * kBatchWaves + wave;
    const bool active = u < nu;  // wave-uniform
    const int pb = blockIdx.y;
    {
        const __amdgpu_buffer_rsrc_t rt = row_buffer(tabs + segs[docs[grp.x]].dense_off, 2 * kTabU4 * 16);
        for (int c = wave; c < 2 * kTabU4 / 64; c += kBatchWaves) lds_copy16(rt, c * 1024 + lane * 16, &tab[c * 64]);
    }
    const int ndocs = min(grp.y, kGroupCap);  // the plan's groups hold at most kGroupCap
    for (int i = static_cast<int>(threadIdx.x); i < ndocs; i += 64 * kBatchWaves) {
        const Seg& sg = segs[docs[grp.x + i]];
        g_off[i] = sg.grid_off;
        s_off[i] = sg.spec_off;
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // tables and offsets visible to every wave; the only workgroup barrier
    if (!active) return;

    const int ub = u == 0 ? 0 : n1 - u;  // n1 need not be a power of two (sub-row documents)
    const bool self = ub == u;
    const int shift = u == 0 ? 1 : 0;
    const int R = u == 0 ? 1 : 16 / m;  // documents per block
    const u4* fwd = tab + (u == 0 ? 0 : kTabU4);
    const u4* inv = fwd + 2 * 64;
    const __amdgpu_buffer_rsrc_t rg =
        row_buffer(grid + pb * grid_pb_stride, static_cast<uint32_t>(grid_pb_stride * 4));
    const __amdgpu_buffer_rsrc_t rf =
        row_buffer(fgrid + pb * fgrid_pb_stride, static_cast<uint32_t>(fgrid_pb_stride * 4));
    uint32_t* stage = xch_all[wave];
    uint32_t* xlds = stage + kPad * 16 + p;
    uint32_t* flds = stage + (2 * kPad + 16) * 16 + p;

    // forward DFT of rows u and ub: own[r] = frequency slot 4 h + r of row u; row ub's
    // spectrum to the exchange row dst at slot 4 h + r - shift (row 0: its frequency 0
    // also at slot m - 1)
    auto forward = [&](u4 in_u, u4 in_b, uint32_t* own, uint32_t* dst) {
#pragma unroll
        for (int i = 0; i < kPad / 4; ++i) dst[16 * (4 * i + h - kPad)] = 0u;
        f4 acc[2][2];
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[i][0] = acc[i][1] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        const u4 are = fwd[lane], aim = fwd[64 + lane];
        acc[0][0] = mma(are, in_u, acc[0][0]);
        acc[0][1] = mma(aim, in_u, acc[0][1]);
        acc[1][0] = mma(are, in_b, acc[1][0]);
        acc[1][1] = mma(aim, in_b, acc[1][1]);
        uint32_t keep = 0u;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            own[r] = pack_h2(acc[0][0][r], acc[0][1][r]);
            const uint32_t bv = pack_h2(acc[1][0][r], acc[1][1][r]);
            dst[16 * (4 * h + r - shift)] = bv;
            if (r == 0) keep = bv;
        }
        if (shift && h == 0) dst[16 * (m - 1)] = keep;
        wave_lds_fence();
    };

    // frequency slot 4 h + r reads its partner at slot (2 q + 1) m - 1 - v, q its
    // document (row 0: m - 1 - v, through the shifted exchange row).  Slots past the
    // block's documents read the first front slot, which holds zero: their own slot may
    // hold a stale value (row 0 leaves slot 15 unwritten), and a non-finite one would
    // reach every output through the zero entries of the inverse table (0 * inf)
    int pslot[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int v = 4 * h + r, q = v / m;
        pslot[r] = q < R ? (2 * q + 1) * m - 1 - v : -kPad;
    }

    for (int k0 = 0; k0 < ndocs; k0 += R) {
        const int nr = min(R, ndocs - k0);  // documents in this block
        // register t holds time slot 4 t + h: point j of document q
        uint32_t o_du[4], o_db[4], o_fu[4], o_fb[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int v = 4 * t + h, q = v / m, j = v - q * m;
            o_du[t] = o_db[t] = o_fu[t] = o_fb[t] = kNone;
            if (q < nr) {
                const int64_t goff = g_off[k0 + q], soff = s_off[k0 + q];
                const uint32_t pbyte = static_cast<uint32_t>(p) * 4;
                o_du[t] = static_cast<uint32_t>((goff + static_cast<int64_t>(u) * m + j) * 64) + pbyte;
                o_db[t] = static_cast<uint32_t>((goff + static_cast<int64_t>(ub) * m + j) * 64) + pbyte;
                o_fu[t] = static_cast<uint32_t>((soff + static_cast<int64_t>(u) * m + j) * 64) + pbyte;
                o_fb[t] = static_cast<uint32_t>((soff + static_cast<int64_t>(ub) * m + j) * 64) + pbyte;
            }
        }
        u4 fu, fb, xu, xb;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            fu[t] = __builtin_amdgcn_raw_buffer_load_b32(rf, static_cast<int>(o_fu[t]), 0, 2);
            fb[t] = __builtin_amdgcn_raw_buffer_load_b32(rf, static_cast<int>(o_fb[t]), 0, 2);
            xu[t] = __builtin_amdgcn_raw_buffer_load_b32(rg, static_cast<int>(o_du[t]), 0, 2);
            xb[t] = __builtin_amdgcn_raw_buffer_load_b32(rg, static_cast<int>(o_db[t]), 0, 2);
        }

        uint32_t fa[4], fl[4], au[4], wu[4];
        forward(fu, fb, fa, flds);
#pragma unroll
        for (int r = 0; r < 4; ++r) fl[r] = flds[16 * pslot[r]];
        forward(xu, xb, au, xlds);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t b = xlds[16 * pslot[r]];
            const uint32_t a = au[r];
            // correlation: the filter spectrum read at -f (its conjugate for real taps)
            const uint32_t A = corr ? fl[r] : fa[r];
            const uint32_t bf = corr ? fa[r] : fl[r];
            const uint32_t e1 = pk_add_conj(a, b);
            const uint32_t e2 = pk_swap_add_conj(a, b);
            const uint32_t U = pk_add_neg_hi(e1, e2);
            const uint32_t V = pk_add_neg_lo(e1, e2);
            wu[r] = w_pos(A, bf, U, V);
            xlds[16 * pslot[r]] = w_neg(A, bf, U, V);
        }
        if (shift && h == 0) xlds[-16] = xlds[16 * (m - 1)];
        wave_lds_fence();
        u4 wb;
#pragma unroll
        for (int t = 0; t < 4; ++t) wb[t] = xlds[16 * (4 * h + t - shift)];
        wave_lds_fence();

        // inverse of both rows: output register r is time slot 4 r + h, the slot that
        // input register r came from
        f4 acc[2][2];
#pragma unroll
        for (int i = 0; i < 2; ++i) acc[i][0] = acc[i][1] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        const u4 are = inv[lane], aim = inv[64 + lane];
        const u4 win = {wu[0], wu[1], wu[2], wu[3]};
        acc[0][0] = mma(are, win, acc[0][0]);
        acc[0][1] = mma(aim, win, acc[0][1]);
        acc[1][0] = mma(are, wb, acc[1][0]);
        acc[1][1] = mma(aim, wb, acc[1][1]);
        uint32_t ou[4], ob[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            ou[r] = pack_h2(acc[0][0][r], acc[0][1][r]);
            ob[r] = pack_h2(acc[1][0][r], acc[1][1][r]);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            __builtin_amdgcn_raw_buffer_store_b32(ou[r], rg, static_cast<int>(o_du[r]), 0, 2);
            __builtin_amdgcn_raw_buffer_store_b32(ob[r], rg, static_cast<int>(self ? kNone : o_db[r]), 0, 2);
        }
    }
}

template <int NB>
hipError_t launch_lds_nb(void* grid, int64_t gs, const void* fgrid, int64_t fs, const Seg* segs,
                         const int32_t* docs, const int32_t* groups, int ngroups, const void* tabs,
                         int n1, int npb, int corr, hipStream_t stream, bool sum, float dscale,
                         bool out2) {
    const int ug = (n1 / 2 + 1 + kLdsWaves - 1) / kLdsWaves;
    const dim3 g(ngroups * ug, npb), b(64 * kLdsWaves);
    if (sum)
        hipLaunchKernelGGL((row_lds_kernel<NB, true>), g, b, 0, stream, static_cast<uint32_t*>(grid), gs,
                           static_cast<const uint32_t*>(fgrid), fs, segs, docs,
                           reinterpret_cast<const int2*>(groups), static_cast<const u4*>(tabs), n1, corr,
                           dscale, out2 ? 1 : 0);
    else
        hipLaunchKernelGGL((row_lds_kernel<NB, false>), g, b, 0, stream, static_cast<uint32_t*>(grid), gs,
                           static_cast<const uint32_t*>(fgrid), fs, segs, docs,
                           reinterpret_cast<const int2*>(groups), static_cast<const u4*>(tabs), n1, corr,
                           dscale, out2 ? 1 : 0);
    return hipGetLastError();
}

template <int NB>
hipError_t launch_partner_nb(void* grid, int64_t gs, const void* fgrid, int64_t fs, const Seg* segs,
                             const int32_t* docs, const int32_t* groups, int ngroups,
                             const void* tabs, int n1, int npb, int corr, hipStream_t stream, bool sum,
                             float dscale, bool out2) {
    const int ug = (n1 / 2 + 1 + kPartnerWaves - 1) / kPartnerWaves;
    const dim3 g(ngroups * ug, npb), b(64 * kPartnerWaves);
    if (sum)
        hipLaunchKernelGGL((row_partner_kernel<NB, true>), g, b, 0, stream, static_cast<uint32_t*>(grid), gs,
                           static_cast<const uint32_t*>(fgrid), fs, segs, docs,
                           reinterpret_cast<const int2*>(groups), static_cast<const u4*>(tabs), n1, corr,
                           dscale, out2 ? 1 : 0);
    else
        hipLaunchKernelGGL((row_partner_kernel<NB, false>), g, b, 0, stream, static_cast<uint32_t*>(grid), gs,
                           static_cast<const uint32_t*>(fgrid), fs, segs, docs,
                           reinterpret_cast<const int2*>(groups), static_cast<const u4*>(tabs), n1, corr,
                           dscale, out2 ? 1 : 0);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_row_batch(void* grid, int64_t grid_pb_stride, const void* fgrid,
                            int64_t fgrid_pb_stride, const Seg* segs, const int32_t* docs,
                            const int32_t* groups, int ngroups, const void* tabs, int n1, int npb,
                            int corr, hipStream_t stream) {
    if (ngroups == 0) return hipSuccess;
    const int ug = (n1 / 2 + 1 + kBatchWaves - 1) / kBatchWaves;
    const dim3 g(ngroups * ug, npb), b(64 * kBatchWaves);
    hipLaunchKernelGGL(row_batch_kernel, g, b, 0, stream, static_cast<uint32_t*>(grid), grid_pb_stride,
                       static_cast<const uint32_t*>(fgrid), fgrid_pb_stride, segs, docs,
                       reinterpret_cast<const int2*>(groups), static_cast<const u4*>(tabs), n1, corr);
    return hipGetLastError();
}

hipError_t launch_row_dense(int nb, void* grid, int64_t grid_pb_stride, const void* fgrid,
                            int64_t fgrid_pb_stride, const Seg* segs, const int32_t* docs,
                            const int32_t* groups, int ngroups, const void* tabs, int n1, int npb,
                            int corr, hipStream_t stream, bool sum, float dscale, bool out2) {
    if (ngroups == 0) return hipSuccess;
    if (!sum && (dscale != 1.0f || out2)) return hipErrorInvalidValue;
#define RUBICONV_ARGS grid, grid_pb_stride, fgrid, fgrid_pb_stride, segs, docs, groups, ngroups, tabs, n1, npb, corr, stream, sum, dscale, out2
    switch (nb) {
        case 1: return launch_lds_nb<1>(RUBICONV_ARGS);
        case 2: return launch_lds_nb<2>(RUBICONV_ARGS);
        case 3: return launch_partner_nb<3>(RUBICONV_ARGS);
        case 4: return launch_partner_nb<4>(RUBICONV_ARGS);
        case 5: return launch_partner_nb<5>(RUBICONV_ARGS);
        case 6: return launch_partner_nb<6>(RUBICONV_ARGS);
        case 7: return launch_partner_nb<7>(RUBICONV_ARGS);
        case 8: return launch_partner_nb<8>(RUBICONV_ARGS);
        default: return hipErrorInvalidValue;
    }
#undef RUBICONV_ARGS
}

}  // namespace rubiconv
