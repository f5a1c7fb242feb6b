/*
 * rubiconv_ct.h -- C ABI of the masked Cooley-Tukey variant of the packed
 * causal long convolution (RubiConv-CooleyTukey, Section 3.1, Algorithm 2),
 * a comparison path beside the four-step method of rubiconv.h.
 *
 * It computes exactly the convolution defined at the top of rubiconv.h, by a
 * different transform: every document is zero-padded to the power-of-two size
 * P_i, the smallest power of two >= L_i + min(L_i, L) - 1 (the causal padding
 * of Algorithm 1 with the power-of-two length Algorithm 2 needs), and the
 * iterative radix-2 FFT runs over the packed array with every butterfly stage
 * masked per element: at stage s an element whose document holds fewer than
 * 2^s points keeps its value (identity factors), every other element takes the
 * standard butterfly at its position inside its own document.  The product with
 * the filter's spectrum and the inverse transform (the same masked stages with
 * conjugate twiddles) follow, and each document keeps its first L_i outputs.
 * Two real channels share one complex transform and are separated by conjugate
 * symmetry (Appendix, "Optimizing dual real FFTs").
 *
 * The conventions of rubiconv.h apply: device pointers are HIP device memory,
 * the caller owns every buffer, stream calls only enqueue work and never
 * allocate, synchronise or print, and every call returns a status.
 *
 * Limits: D must be even, and no document may need a transform larger than
 * 2^19 points (L_i + min(L_i, L) - 1 <= 524288); other requests return
 * RUBICONV_ERR_UNSUPPORTED.  Documents above 2^15 points take one more pass over
 * their transform grid in each direction (the stages between the tile and the
 * column pass).
 */
#ifndef RUBICONV_CT_H_
#define RUBICONV_CT_H_

#include "rubiconv.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rubiconv_ct_plan_s* rubiconv_ct_plan_t; /* opaque, library-owned */

/*
 * Build a plan of the masked Cooley-Tukey variant from the document boundaries.
 * Arguments as for rubiconv_plan (without n1): B, N, D, L >= 1, max_docs >= 1,
 * cu_seqlens_host host int32 [B][max_docs + 1] with c[0] = 0, non-decreasing,
 * c[max_docs] = N (empty documents ignored), x_dtype and y_dtype the element
 * types of x and y.  The plan copies what it needs and uploads its tables
 * synchronously.
 * Errors: RUBICONV_ERR_ARG, RUBICONV_ERR_SEQLENS, RUBICONV_ERR_UNSUPPORTED (odd
 * D, or a document beyond the size limit above), RUBICONV_ERR_ALLOC,
 * RUBICONV_ERR_HIP.
 */
rubiconv_status_t rubiconv_ct_plan(rubiconv_ct_plan_t* out, int B, int N, int D, int L,
                                   int max_docs, const int32_t* cu_seqlens_host,
                                   rubiconv_dtype_t x_dtype, rubiconv_dtype_t y_dtype);

/* Release a plan (null is ignored); work using it must have finished. */
void rubiconv_ct_plan_destroy(rubiconv_ct_plan_t plan);

/* Bytes of the filter spectrum buffer: per power-of-two size present, the
 * non-negative half of the spectrum of every channel pair (complex fp16 for
 * bf16 x, complex fp32 otherwise). */
size_t rubiconv_ct_spectrum_bytes(rubiconv_ct_plan_t plan);

/* Bytes of device scratch rubiconv_ct_filter_spectrum and rubiconv_ct_packed_conv
 * need (one buffer serves both, not at the same time): the partly transformed
 * documents longer than 512 points, complex fp16 for bf16 x, complex fp32
 * otherwise. */
size_t rubiconv_ct_workspace_bytes(rubiconv_ct_plan_t plan);

/*
 * Transform the filters for every power-of-two size P of the plan: the first
 * min(L, floor((P + 1) / 2)) taps of each channel (every lag a document of that
 * size uses, and no tap that could wrap onto one of its outputs), zero-padded to
 * P, through the masked transform.
 *
 *   filters    device float32 [D][L], row-major.
 *   spectrum   device buffer of rubiconv_ct_spectrum_bytes(plan), 256-byte
 *              aligned, written completely; its layout is private to the library.
 *   workspace  device buffer of rubiconv_ct_workspace_bytes(plan), 256-byte aligned.
 *   stream     HIP stream the work is enqueued on.
 * Errors: RUBICONV_ERR_ARG (null or misaligned pointer), RUBICONV_ERR_HIP.
 */
rubiconv_status_t rubiconv_ct_filter_spectrum(rubiconv_ct_plan_t plan, const float* filters,
                                              void* spectrum, void* workspace, hipStream_t stream);

/*
 * The packed convolution (definition at the top of rubiconv.h) through the
 * masked Cooley-Tukey transform.
 *
 *   x          device [B][N][D] of the plan's x_dtype, channels last; 8-byte
 *              aligned for float32.
 *   spectrum   written by rubiconv_ct_filter_spectrum with this plan.
 *   y          device [B][N][D] of the plan's y_dtype, every element written; it
 *              must not overlap x, spectrum or workspace.  8-byte aligned for
 *              float32, 4-byte for bf16.
 *   workspace  device buffer of rubiconv_ct_workspace_bytes(plan), 256-byte aligned.
 *   stream     HIP stream the work is enqueued on.
 * Errors: RUBICONV_ERR_ARG, RUBICONV_ERR_HIP.
 */
rubiconv_status_t rubiconv_ct_packed_conv(rubiconv_ct_plan_t plan, const void* x,
                                          const void* spectrum, void* y, void* workspace,
                                          hipStream_t stream);

/*
 * The plan's document table in row order: out is host int32 [cap][6] receiving
 * (row, index of the document in its row, start, length, P_i, offset of the
 * document in the packed transform array) per non-empty document; *n_docs
 * receives the count (rows beyond cap are not written).  Used by tests to check
 * the segment indexing and the padding rule exactly.
 * Errors: RUBICONV_ERR_ARG.
 */
rubiconv_status_t rubiconv_ct_plan_doc_table(rubiconv_ct_plan_t plan, int32_t* out, int cap,
                                             int* n_docs);

#ifdef __cplusplus
}
#endif

#endif /* RUBICONV_CT_H_ */
