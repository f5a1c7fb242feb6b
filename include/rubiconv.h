/*
 * rubiconv.h -- C ABI of the MI355X (gfx950) boundary-respecting causal long
 * convolution over packed sequences (RubiConv, arXiv 2605.08451).
 *
 * The operation (problem statement, Section 1; depthwise causal convolution of
 * Section 4.1, "Benchmarking protocol"; block-diagonal Toeplitz form of
 * Section 3.2): every row b of x[B][N][D] is a concatenation of documents given
 * by cu_seqlens.  For each document [s0, s1) of row b and each channel d,
 *
 *     y[b][t][d] = sum_{tau = 0}^{min(t - s0, L - 1)} k[d][tau] * x[b][t - tau][d],
 *                  s0 <= t < s1,
 *
 * so no output mixes values across a document boundary and nothing wraps from
 * the end of a row to its start.  Lags tau >= L contribute nothing.
 *
 * How it is computed (Algorithm 1, Theorem 2.1, Appendix "Implementation
 * details"): every document i gets its own transform size P_i = N1 * m_i with
 * P_i >= L_i + min(L_i, L) - 1 (the causal zero padding of Algorithm 1; m_i is
 * rounded up to a 2^a 3^b 5^c size, which gives the identical exact result).
 * The document is laid out as an N1 x m_i grid in row-major order (time
 * t = m_i*a + j), transformed by N1-point column DFTs, the per-document twiddle
 * omega_{P_i}^{u*j}, and m_i-point row DFTs (the block-diagonal second DFT).
 * Two real channels share one complex transform and are separated by conjugate
 * symmetry (Appendix, "Optimizing dual real FFTs", Algorithm 3); the product
 * with the filter spectrum is taken on the 2-D frequency grid; the inverse runs
 * the same steps in reverse order, then the output is cut back to L_i.
 *
 * Conventions shared by every call:
 *   - All device pointers are HIP device memory on the current device; host
 *     pointers are ordinary process memory.  The caller owns every buffer it
 *     passes; the library owns only the plan, the plan's device tables and 1 KB of
 *     pinned host memory per plan (its range-scale guesses).
 *   - Calls taking a stream enqueue work on it and return without waiting.
 *     They never synchronise the device, never allocate device memory and
 *     never print.  The plan may be used from several streams and host threads
 *     at once as long as each call has its own workspace (and output).
 *     rubiconv_packed_conv forks independent launches onto side streams owned
 *     by the plan and joins them back into the caller's stream with events, so
 *     the call remains ordered on the caller's stream (and capturable).
 *   - Every call returns a status; nothing is thrown across the ABI.  Argument
 *     errors are detected on the host before anything is enqueued.
 *
 * Value range of bf16 inputs.  bf16 x runs on complex fp16 grids (fp16 spectra,
 * twiddle and separation products; fp32 accumulation in the matrix products), whose
 * range (6e-8 .. 65504) is far narrower than bf16's.  Two exact power-of-two scales
 * keep the grids inside it, and are undone in fp32 before the output is rounded:
 *   - rubiconv_filter_spectrum scales each channel pair's taps so that the larger
 *     of the two channels' sums of |k| (a bound on every spectrum value) is 2^8;
 *   - rubiconv_packed_conv scales x by 2^(3 - e), 2^e the power of two at or above
 *     the largest |x| of the call, and the gradient calls scale dy (and x) the same
 *     way.  On the matrix-core path (N1 = 256, D a multiple of 32) each call finds
 *     those scales inside its column passes: a pass runs at the scale the plan's
 *     previous call of the same kind on the same input buffer found (1 for the first
 *     call; 64 slots per kind, hashed from the buffer's address), and a second column
 *     pass runs only when the call's own scale differs.  The result does not depend on
 *     that guess (bit for bit); the plan keeps its guesses in pinned host memory that
 *     its kernels write.  Elsewhere the tensor is read once more for its largest
 *     magnitude.
 * Within that, results meet the 2e-2 relative L2 bar for finite bf16 inputs whose
 * outputs are finite in bf16, except for a document whose values lie far below the
 * call's largest |x| (the x scale is one per call): below about 1e-6 of it its grid
 * values fall into fp16's subnormal range and lose relative precision.  Setting RUBICONV_PRESCALE=0 in the environment when a plan is
 * created drops the forward's x scale: x is then taken as it is, which keeps the
 * range the tests cover (a constant 5 plus unit noise under an all-ones filter, whose
 * outputs reach 8e4, and rms(x) from 1e-4 to 300); coherent inputs of a few tens and
 * more can then overflow a grid.  fp32 inputs run on fp32 grids and have no such limit.
 */
#ifndef RUBICONV_H_
#define RUBICONV_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rubiconv_plan_s* rubiconv_plan_t; /* opaque, library-owned */

typedef enum {
    RUBICONV_F32 = 0,  /* IEEE float32 */
    RUBICONV_BF16 = 1  /* bfloat16 (upper half of a float32); outputs rounded to nearest even */
} rubiconv_dtype_t;

typedef enum {
    RUBICONV_OK = 0,
    RUBICONV_ERR_ARG = 1,         /* null pointer, non-positive size, unknown dtype */
    RUBICONV_ERR_SEQLENS = 2,     /* cu_seqlens row not 0 = c0 <= c1 <= ... <= c_max_docs = N */
    RUBICONV_ERR_UNSUPPORTED = 3, /* valid request the library does not implement */
    RUBICONV_ERR_ALLOC = 4,       /* host or device allocation for the plan failed */
    RUBICONV_ERR_HIP = 5          /* a HIP call or kernel launch failed */
} rubiconv_status_t;

/*
 * Build a plan from the document boundaries (Algorithm 1, the data-processing
 * step, which depends only on the segment ids and is shared by every layer of a
 * model; Appendix, "Precomputation of adaptive structures").
 *
 *   out             receives the plan handle (host pointer, not null).
 *   B, N, D, L      rows, tokens per row, channels, filter taps (all >= 1).
 *   max_docs        documents per row in cu_seqlens_host (>= 1).
 *   cu_seqlens_host host int32 [B][max_docs + 1]: per row the prefix sums of the
 *                   document lengths, c[0] = 0, non-decreasing, c[max_docs] = N.
 *                   Equal neighbours are empty documents and are ignored, which
 *                   lets rows with fewer documents be padded with N.
 *   x_dtype,y_dtype element types of x and y for packed_conv.
 *   n1              column size N1 of the grid (the paper's k): 0 picks the
 *                   default (256); otherwise 64 or 256.
 *
 * Documents of at most 64 tokens (512 with bf16 x and y and D a multiple of 32)
 * take the direct path when together they would fill at least 1/16 of the
 * transform grid: they skip the transforms, and their outputs are the defining sums
 * of the block-diagonal Toeplitz form (Section 3.2) evaluated directly, which avoids
 * padding a short document to a whole N1-point column grid.  With bf16 x and y and D
 * a multiple of 32 those sums run on the matrix cores as blocked Toeplitz products
 * (fp32 accumulation), and every x, y, dy and dx buffer passed with the plan must be
 * 16-byte aligned (RUBICONV_ERR_ARG otherwise); RUBICONV_DIRECT_MFMA = 0, read when the
 * plan is made, keeps them on the 64-token VALU kernel.  RUBICONV_DIRECT_MAX = 0..128
 * (0..512 on the matrix cores), read when the plan is made, sets the length limit and
 * drops the share condition (0 turns the path off).
 * Documents whose smallest transform sizes differ little may share one size class:
 * a document then takes a larger transform than its own minimum (any transform
 * holding the causal padding gives the same exact result, Theorem 2.1), when that
 * removes a filter spectrum and moves fewer bytes overall.  The environment
 * variable RUBICONV_CLASS_MERGE = 0 (read when the plan is made) keeps every
 * document at its own smallest size; 1 or unset merges.
 * Rows of at most 8 points (bf16 inputs) are transformed 16 / m documents at a time
 * when such rows hold at least a quarter of the grid; RUBICONV_ROW_BATCH = 0 turns
 * this off and 1..8 sets the largest batched row size regardless of the share.
 * Rows longer than 256 points (bf16 inputs) are split once more, m = m1 m2, into m1
 * sub-rows of at most 64 (else 128) points each, transformed by the same matrix-core
 * row kernels as short rows (Algorithm 1's four-step factorisation applied to
 * the row DFT); RUBICONV_LONG_ROWS = 0 (read when the plan is made) keeps such rows
 * whole in the generic row kernel instead.
 * A row size m_i is the smallest 2^a 3^b 5^c number of a fixed list (above it, any
 * 2^a 3^b 5^c number) whose N1 m_i holds the causal padding.  RUBICONV_EXACT_ROWS = 1
 * (read when the plan is made) gives rows of at most 128 points on the matrix cores
 * (bf16 inputs) the smallest integer m_i instead, as Algorithm 1 allows: the same
 * exact result on fewer grid points.
 *   stream          HIP stream the upload of the plan's device tables is enqueued on
 *                   (hipMemcpyAsync from a host copy the plan keeps): work that uses
 *                   the plan on this stream is ordered after it; other streams must
 *                   wait for it (or the device be synchronised) before using the plan.
 * The plan copies what it needs; cu_seqlens_host may be freed on return.  Plan
 * creation allocates the plan's device memory and pinned host words and creates its
 * side streams and events (hipMalloc, hipHostMalloc, hipStreamCreate, which HIP may
 * order with other device work);
 * it does not wait for the upload.
 * Errors: RUBICONV_ERR_ARG (also for a malformed RUBICONV_DIRECT_MAX,
 * RUBICONV_DIRECT_MFMA, RUBICONV_CLASS_MERGE or RUBICONV_PRESCALE),
 * RUBICONV_ERR_SEQLENS, RUBICONV_ERR_UNSUPPORTED (n1 not supported, a document
 * so long that its row DFT would exceed the largest supported size, or a shape whose
 * kernels would need buffer offsets of 32 bits or more: a document's or size
 * class's P * D * 4 bytes above 2^30, or a pair block's grid at 2^31 bytes or more),
 * RUBICONV_ERR_ALLOC, RUBICONV_ERR_HIP.
 */
rubiconv_status_t rubiconv_plan(rubiconv_plan_t* out, int B, int N, int D, int L, int max_docs,
                                const int32_t* cu_seqlens_host, rubiconv_dtype_t x_dtype,
                                rubiconv_dtype_t y_dtype, int n1, hipStream_t stream);

/* Release a plan and its device tables (null is ignored).  Work already
 * enqueued that uses the plan must have finished. */
void rubiconv_plan_destroy(rubiconv_plan_t plan);

/* Bytes of the device buffer that holds the transformed filters of a plan (one
 * grid per distinct transform size of the plan). 0 for a null plan. */
size_t rubiconv_spectrum_bytes(rubiconv_plan_t plan);

/* Bytes of device scratch that filter_spectrum and packed_conv need.  A single
 * buffer of this size serves both calls (not at the same time).  Grids are
 * complex fp32 for fp32 inputs and complex fp16 for bf16 inputs. */
size_t rubiconv_workspace_bytes(rubiconv_plan_t plan);

/*
 * Transform the filters for the plan's size classes (the filter side of
 * Algorithm 3).  For every distinct transform size P = N1 * m of the plan, the
 * first min(L, floor((P+1)/2)) taps of each channel (enough for every document
 * of that size) are padded to P and taken through the column DFTs and the
 * per-size twiddle, two channels per complex value.  rubiconv_packed_conv
 * applies the row DFTs and the conjugate-symmetry separation together with the
 * data's, so the buffer holds the filters' half-transformed grids.
 *
 *   filters    device float32 [D][L], row-major (channel d's taps contiguous).
 *   spectrum   device buffer of rubiconv_spectrum_bytes(plan), 256-byte aligned,
 *              written completely; its layout is private to the library.
 *   workspace  device buffer of rubiconv_workspace_bytes(plan), 256-byte aligned.
 *   stream     HIP stream the work is enqueued on.
 * Errors: RUBICONV_ERR_ARG (null plan or pointer, misaligned buffer),
 * RUBICONV_ERR_HIP (launch failure).
 */
rubiconv_status_t rubiconv_filter_spectrum(rubiconv_plan_t plan, const float* filters,
                                           void* spectrum, void* workspace, hipStream_t stream);

/*
 * The packed convolution y = conv(x, k) defined at the top of this file.
 *
 * Unlike a call that takes cu_seqlens and the filters directly, this one takes the
 * plan (which consumed the segment ids once: the data-processing step depends only on
 * them and is shared by every layer, Appendix, "Precomputation of adaptive
 * structures") and the filter spectrum (rubiconv_filter_spectrum, the filter side of
 * Algorithm 3, once per filter bank).  A step of the convolution is the two calls.
 *
 *   x          device [B][N][D] of the plan's x_dtype, channels last, row-major.
 *   spectrum   device spectra written by rubiconv_filter_spectrum with this plan.
 *   y          device [B][N][D] of the plan's y_dtype; every element is written.
 *              y must not overlap x, spectrum or workspace.
 *   workspace  device buffer of rubiconv_workspace_bytes(plan), 256-byte aligned.
 *   stream     HIP stream the work is enqueued on.
 * Errors: RUBICONV_ERR_ARG, RUBICONV_ERR_HIP.
 */
rubiconv_status_t rubiconv_packed_conv(rubiconv_plan_t plan, const void* x, const void* spectrum,
                                       void* y, void* workspace, hipStream_t stream);

/*
 * The packed convolution for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  It is
 * rubiconv_packed_conv with the workspace taken from a scratch array that the library
 * holds in device memory: RUBICONV_NOALLOC_SCRATCH_BYTES on every device that loads
 * the library, kept until the process ends.  The call itself allocates nothing.
 *
 *   x, spectrum, y, stream   as for rubiconv_packed_conv (the caller still owns them).
 * The scratch array of a device is shared by every call on that device and keeps the
 * last call's contents; nothing in it needs to start at zero.  Calls that overlap in
 * time on one device (other streams, other threads) race on it: order them.
 * Errors: RUBICONV_ERR_ARG (null plan or pointer, misaligned buffer),
 * RUBICONV_ERR_UNSUPPORTED (rubiconv_workspace_bytes(plan) exceeds
 * RUBICONV_NOALLOC_SCRATCH_BYTES), RUBICONV_ERR_HIP.
 */
#define RUBICONV_NOALLOC_SCRATCH_BYTES ((size_t)320 << 20)
rubiconv_status_t rubiconv_packed_conv_noalloc(rubiconv_plan_t plan, const void* x, const void* spectrum,
                                               void* y, hipStream_t stream);

/*
 * Gradients for training (the method targets training pipelines, Section 1).
 * The convolution is linear in x and in k, so for an upstream gradient dy of y
 * the gradients are the adjoints of the two maps:
 *
 *     dx[b][s][d] = sum_{tau = 0}^{min(s1 - 1 - s, L - 1)} k[d][tau] * dy[b][s + tau][d],
 *                   s0 <= s < s1   (anti-causal correlation inside the document);
 *     dk[d][tau]  = sum over every document [s0, s1) of every row of
 *                   sum_{t = s0 + tau}^{s1 - 1} dy[b][t][d] * x[b][t - tau][d],   tau < L.
 *
 * Both run the convolution's four-step passes on the same plan.  For dx the
 * product takes the filter spectrum at -f, i.e. its conjugate for real taps
 * (Appendix, conjugate symmetry of real transforms).  For dk each document's
 * product is dy's spectrum times the conjugate of x's spectrum on the
 * document's own grid, the inverse leaves the document's cross-correlation at
 * lags 0..len-1, and the documents' correlations are summed per channel and lag.
 * The inverse transforms are linear and the same for all documents of one size
 * class, so on the matrix-core row pass (bf16 inputs, rows of at most 128 points)
 * the products of up to eight documents of a class are added first, longest
 * document first, and transformed back once, onto the longest one's positions:
 * the class's transform size keeps the causal padding of its longest document,
 * so no document's correlation wraps onto a lag below that document's length.
 */

/*
 * dx for an upstream gradient dy.
 *
 *   dy         device [B][N][D] of the plan's y_dtype, channels last.
 *   spectrum   device spectra written by rubiconv_filter_spectrum with this plan
 *              (the same buffer the forward call uses).
 *   dx         device [B][N][D] of the plan's x_dtype; every element is written.
 *              dx must not overlap dy, spectrum or workspace.
 *   workspace  device buffer of rubiconv_workspace_bytes(plan), 256-byte aligned.
 *   stream     HIP stream the work is enqueued on.
 * Errors: RUBICONV_ERR_ARG, RUBICONV_ERR_HIP.
 */
rubiconv_status_t rubiconv_packed_conv_dx(rubiconv_plan_t plan, const void* dy, const void* spectrum,
                                          void* dx, void* workspace, hipStream_t stream);

/* Bytes of device scratch rubiconv_packed_conv_dk and rubiconv_packed_conv_backward
 * need: two document grids and a float32 [B][N][D] buffer (at least
 * rubiconv_workspace_bytes).  0 for a null plan. */
size_t rubiconv_dk_workspace_bytes(rubiconv_plan_t plan);

/*
 * dk for an upstream gradient dy and the forward input x.
 *
 *   x          device [B][N][D] of the plan's x_dtype (the forward call's input).
 *   dy         device [B][N][D] of the plan's y_dtype.
 *   dk         device float32 [D][L], row-major; every element is written (lags
 *              no document reaches are 0).
 *   workspace  device buffer of rubiconv_dk_workspace_bytes(plan), 256-byte
 *              aligned; dk must not overlap it.
 *   stream     HIP stream the work is enqueued on.
 * The sums over documents run in a fixed order (within a size class's group and
 * then over the groups' and other documents' correlations, longest first, ties in
 * table order), so results are deterministic.
 * Errors: RUBICONV_ERR_ARG, RUBICONV_ERR_UNSUPPORTED (a plan of 2^31 grid points
 * or more), RUBICONV_ERR_HIP.
 */
rubiconv_status_t rubiconv_packed_conv_dk(rubiconv_plan_t plan, const void* x, const void* dy,
                                          float* dk, void* workspace, hipStream_t stream);

/*
 * dx and dk of one backward pass in one call: the same results as
 * rubiconv_packed_conv_dx followed by rubiconv_packed_conv_dk, with dy's column
 * DFTs (Algorithm 1's first transform step) computed once for both.  dk's row
 * stage writes its class sums over x's grid in the workspace, so dy's grid stays
 * for dx's correlation with the filter (the same products as for dx alone).
 * Taken when every transform document runs on the matrix-core passes (bf16 x and
 * dy, rows of at most 128 points, no split rows); otherwise the two calls run in
 * sequence.  dx is bit-identical to rubiconv_packed_conv_dx's; dk's products are
 * formed from dy's grid at dx's range scale times the filter gradient's split
 * (exact powers of two), so it can differ from rubiconv_packed_conv_dk's in the
 * last bits of fp16 rounding.
 *
 *   x, dy, spectrum, dx, dk as for the two calls above; dx and dk must not
 *              overlap each other, the inputs or workspace.
 *   workspace  device buffer of rubiconv_dk_workspace_bytes(plan), 256-byte aligned.
 *   stream     HIP stream the work is enqueued on.
 * Errors: RUBICONV_ERR_ARG, RUBICONV_ERR_UNSUPPORTED (as for dk), RUBICONV_ERR_HIP.
 */
rubiconv_status_t rubiconv_packed_conv_backward(rubiconv_plan_t plan, const void* x, const void* dy,
                                                const void* spectrum, void* dx, float* dk, void* workspace,
                                                hipStream_t stream);

/* Summary of a plan (host call, no device work). */
typedef struct {
    int B, N, D, L;
    int n1;             /* column size N1 of the grid */
    int n_docs;         /* non-empty documents */
    int n_classes;      /* distinct transform sizes P = N1 * m */
    int n_pair_blocks;  /* channel pairs are processed in blocks of 16 */
    int64_t grid_points;    /* sum over documents of P_i */
    int64_t class_points;   /* sum over classes of P */
    int64_t tokens;         /* sum over documents of L_i (= B * N) */
    int direct_max;         /* documents of at most this many tokens take the direct path */
    int n_direct;           /* documents on the direct path */
} rubiconv_plan_info_t;

rubiconv_status_t rubiconv_plan_info(rubiconv_plan_t plan, rubiconv_plan_info_t* info);

/*
 * The plan's document table, in row order: out is host int32 [cap][6] receiving
 * (row, index of the document in its row, start, length, m_i, P_i) for each
 * non-empty document; *n_docs receives the count (rows beyond cap are not
 * written).  m_i = P_i = 0 marks a document of the direct path.  Used by tests to
 * check the segment indexing exactly.
 */
rubiconv_status_t rubiconv_plan_doc_table(rubiconv_plan_t plan, int32_t* out, int cap,
                                          int* n_docs);

/*
 * Stage timing (tracing; not for production loops).  After
 * rubiconv_profile_start(plan, max_calls), each of the next max_calls calls of
 * rubiconv_filter_spectrum / rubiconv_packed_conv / rubiconv_packed_conv_dx /
 * rubiconv_packed_conv_dk / rubiconv_packed_conv_backward with this plan records a
 * HIP event on its stream before its first kernel and after every stage (a stage is
 * one kernel, or the launches of the row stage across the plan's side streams up to
 * their join), at most 16 per call.  rubiconv_profile_read waits for the recorded
 * events and returns, per stage name, the number of calls that recorded it and
 * their total milliseconds (host array of cap entries; *n receives the number of
 * distinct stages).  The plan keeps the events it creates for this until it is
 * destroyed.  Profiling state belongs to the plan: use one stream and one thread
 * while it is active.  max_calls = 0 stops profiling.
 * Errors: RUBICONV_ERR_ARG, RUBICONV_ERR_ALLOC (event creation), RUBICONV_ERR_HIP.
 */
typedef struct {
    char name[32];   /* stage name, e.g. "col_fwd" */
    int launches;
    double total_ms;
} rubiconv_kernel_time_t;

rubiconv_status_t rubiconv_profile_start(rubiconv_plan_t plan, int max_calls);
rubiconv_status_t rubiconv_profile_read(rubiconv_plan_t plan, rubiconv_kernel_time_t* out, int cap,
                                        int* n);

/* Static, human-readable name of a status code. */
const char* rubiconv_status_string(rubiconv_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* RUBICONV_H_ */
