/*
 * rubiconv_oracle.c -- CPU oracle for the boundary-respecting causal long
 * convolution over packed sequences (RubiConv, arXiv 2605.08451).
 *
 * TEST INFRASTRUCTURE.  Only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark load this library.  It shares no code, header,
 * table or generator with the GPU library, and it never runs on the product
 * path.
 *
 * What it computes.  The problem statement (Section 1; Section 4.1,
 * "Benchmarking protocol") is a depthwise causal convolution of X in R^{N x D}
 * with per-channel filters of length L, applied inside every document of a
 * packed row and never across a document boundary or around the row end.
 * Written out for row b, document [s0, s1) and channel d:
 *
 *     y[b,t,d] = sum_{tau = 0}^{min(t - s0, L - 1)} k[d,tau] * x[b,t-tau,d],
 *                s0 <= t < s1.
 *
 * This is the block-diagonal Toeplitz product y = A x of Section 3.2 (one
 * Toeplitz block per document), evaluated entry by entry.  All arithmetic is
 * double precision; inputs are passed as doubles (bf16 and fp32 values convert
 * exactly).
 *
 * Two evaluations are provided:
 *   rco_conv_direct  -- the sum above, tau ascending.
 *   rco_conv_fft     -- per document and channel: zero-pad the document and
 *                       its first min(len, L) taps to the next power of two
 *                       >= len + min(len, L) - 1 (the causal padding rule of
 *                       Algorithm 1), radix-2 FFT both, multiply, inverse,
 *                       scale, keep the first len outputs.  Used where the
 *                       direct sum is too slow.
 * plus rco_conv_at (the sum at sampled (b, t, d) positions) and
 * rco_doc_table (the document table and minimal padded sizes of Algorithm 1).
 *
 * Layouts: x, y [B][N][D] (channels last); k [D][L]; cu_seqlens
 * [B][max_docs + 1] int32, each row 0 = c_0 <= c_1 <= ... <= c_max_docs = N.
 * Return value: 0 (or a count) on success, RCO_EBADSEQ / RCO_EBADARG on
 * invalid input.
 */
#include <complex.h>
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#define RCO_EBADARG (-1)
#define RCO_EBADSEQ (-2)
#define RCO_ENOMEM (-3)

/* ------------------------------------------------------------------ documents */
typedef struct {
    int b;      /* row */
    int k;      /* index of the document inside its row */
    int start;  /* first token */
    int len;    /* number of tokens (> 0) */
} rco_doc;

int rco_validate(int B, int N, int max_docs, const int32_t *cu) {
    if (B < 0 || N < 0 || max_docs < 1 || (B > 0 && !cu)) return RCO_EBADARG;
    for (int b = 0; b < B; ++b) {
        const int32_t *c = cu + (size_t)b * (max_docs + 1);
        if (c[0] != 0 || c[max_docs] != N) return RCO_EBADSEQ;
        for (int k = 0; k < max_docs; ++k)
            if (c[k + 1] < c[k]) return RCO_EBADSEQ;
    }
    return 0;
}

/* Non-empty documents in row order; returns their count or an error. */
static int collect_docs(int B, int N, int max_docs, const int32_t *cu, rco_doc **out) {
    int rc = rco_validate(B, N, max_docs, cu);
    if (rc) return rc;
    int n = 0;
    for (int b = 0; b < B; ++b)
        for (int k = 0; k < max_docs; ++k)
            n += cu[(size_t)b * (max_docs + 1) + k + 1] > cu[(size_t)b * (max_docs + 1) + k];
    rco_doc *d = (rco_doc *)malloc(sizeof(rco_doc) * (n ? n : 1));
    if (!d) return RCO_ENOMEM;
    int i = 0;
    for (int b = 0; b < B; ++b)
        for (int k = 0; k < max_docs; ++k) {
            int s0 = cu[(size_t)b * (max_docs + 1) + k];
            int s1 = cu[(size_t)b * (max_docs + 1) + k + 1];
            if (s1 > s0) {
                d[i].b = b; d[i].k = k; d[i].start = s0; d[i].len = s1 - s0;
                ++i;
            }
        }
    *out = d;
    return n;
}

/*
 * Document table of Algorithm 1 (pre-processing): for each non-empty document
 * (row, index, start, len) and the minimal padded length
 *     L_i' = k * ceil((len + min(len, L) - 1) / k):
 * min(len, L) - 1 causal zeros appended to the document, then the total
 * rounded up to a multiple of the column size k.  out is [cap][5].
 */
int rco_doc_table(int B, int N, int max_docs, const int32_t *cu, int L, int k,
                  int32_t *out, int cap) {
    if (L < 1 || k < 1) return RCO_EBADARG;
    rco_doc *docs = NULL;
    int n = collect_docs(B, N, max_docs, cu, &docs);
    if (n < 0) return n;
    for (int i = 0; i < n && i < cap; ++i) {
        long need = (long)docs[i].len + (docs[i].len < L ? docs[i].len : L) - 1;
        long padded = ((need + k - 1) / k) * (long)k;
        int32_t *o = out + (size_t)i * 5;
        o[0] = docs[i].b; o[1] = docs[i].k; o[2] = docs[i].start; o[3] = docs[i].len;
        o[4] = (int32_t)padded;
    }
    free(docs);
    return n;
}

/* ------------------------------------------------------------------ threads */
typedef struct {
    long n_items;
    long next;               /* shared counter, atomically incremented */
    void (*fn)(void *ctx, long item, void *scratch);
    void *ctx;
    size_t scratch_bytes;
    int failed;
} rco_pool;

static void *worker(void *arg) {
    rco_pool *p = (rco_pool *)arg;
    void *scratch = p->scratch_bytes ? malloc(p->scratch_bytes) : NULL;
    if (p->scratch_bytes && !scratch) {
        __atomic_store_n(&p->failed, 1, __ATOMIC_SEQ_CST);
        return NULL;
    }
    for (;;) {
        long i = __atomic_fetch_add(&p->next, 1, __ATOMIC_SEQ_CST);
        if (i >= p->n_items) break;
        p->fn(p->ctx, i, scratch);
    }
    free(scratch);
    return NULL;
}

static int run_parallel(long n_items, int nthreads, size_t scratch_bytes,
                        void (*fn)(void *, long, void *), void *ctx) {
    if (nthreads <= 0) nthreads = (int)sysconf(_SC_NPROCESSORS_ONLN);
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    rco_pool pool = {n_items, 0, fn, ctx, scratch_bytes, 0};
    pthread_t th[256];
    int started = 0;
    for (int t = 0; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, worker, &pool) != 0) break;
        ++started;
    }
    if (started == 0) worker(&pool);
    for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
    return pool.failed ? RCO_ENOMEM : 0;
}

int rco_default_threads(void) { return (int)sysconf(_SC_NPROCESSORS_ONLN); }

/* ------------------------------------------------------------------ direct form */
typedef struct {
    const rco_doc *docs;
    int N, D, L;
    const double *x, *k;
    double *y;
} conv_ctx;

/* One (document, channel): the defining sum, lags ascending. */
static void direct_item(void *vctx, long item, void *scratch) {
    const conv_ctx *c = (const conv_ctx *)vctx;
    const rco_doc *doc = &c->docs[item / c->D];
    int d = (int)(item % c->D);
    double *col = (double *)scratch;                 /* the document's channel-d values */
    const double *xrow = c->x + ((size_t)doc->b * c->N + doc->start) * c->D + d;
    for (int t = 0; t < doc->len; ++t) col[t] = xrow[(size_t)t * c->D];
    const double *kd = c->k + (size_t)d * c->L;
    double *yrow = c->y + ((size_t)doc->b * c->N + doc->start) * c->D + d;
    for (int t = 0; t < doc->len; ++t) {
        int last = t < c->L - 1 ? t : c->L - 1;      /* k[d, tau] = 0 for tau >= L */
        double acc = 0.0;
        for (int tau = 0; tau <= last; ++tau) acc += kd[tau] * col[t - tau];
        yrow[(size_t)t * c->D] = acc;
    }
}

static int max_len(const rco_doc *docs, int n) {
    int m = 1;
    for (int i = 0; i < n; ++i) if (docs[i].len > m) m = docs[i].len;
    return m;
}

/* Tokens not covered by any document do not exist (cu covers [0, N) exactly),
 * so every output entry is written by exactly one (document, channel) item. */
int rco_conv_direct(int B, int N, int D, int L, int max_docs, const int32_t *cu,
                    const double *x, const double *k, double *y, int nthreads) {
    if (D < 1 || L < 1 || !x || !k || !y) return RCO_EBADARG;
    rco_doc *docs = NULL;
    int n = collect_docs(B, N, max_docs, cu, &docs);
    if (n < 0) return n;
    conv_ctx ctx = {docs, N, D, L, x, k, y};
    int rc = run_parallel((long)n * D, nthreads, sizeof(double) * (size_t)max_len(docs, n),
                          direct_item, &ctx);
    free(docs);
    return rc;
}

/* ------------------------------------------------------------------ FFT variant */
static int next_pow2(long v) {
    int p = 1;
    while (p < v) p <<= 1;
    return p;
}

/* In-place iterative radix-2 decimation-in-time DFT of length n (a power of two):
 * a[f] <- sum_t a[t] exp(sign * 2 pi i f t / n).  Bit-reversal permutation first,
 * then log2(n) butterfly stages; each twiddle is taken from cos/sin directly. */
static void fft_radix2(double complex *a, int n, int sign) {
    for (int i = 1, j = 0; i < n; ++i) {
        int bit = n >> 1;
        for (; j & bit; bit >>= 1) j ^= bit;
        j ^= bit;
        if (i < j) { double complex t = a[i]; a[i] = a[j]; a[j] = t; }
    }
    for (int len = 2; len <= n; len <<= 1) {
        int half = len >> 1;
        for (int j = 0; j < half; ++j) {
            double ang = sign * 2.0 * M_PI * (double)j / (double)len;
            double complex w = cos(ang) + I * sin(ang);
            for (int s = 0; s < n; s += len) {
                double complex u = a[s + j];
                double complex v = a[s + j + half] * w;
                a[s + j] = u + v;
                a[s + j + half] = u - v;
            }
        }
    }
}

static void fft_item(void *vctx, long item, void *scratch) {
    const conv_ctx *c = (const conv_ctx *)vctx;
    const rco_doc *doc = &c->docs[item / c->D];
    int d = (int)(item % c->D);
    int taps = doc->len < c->L ? doc->len : c->L;    /* lags that can occur */
    int P = next_pow2((long)doc->len + taps - 1);    /* causal zero padding */
    double complex *a = (double complex *)scratch;
    double complex *h = a + P;
    const double *xrow = c->x + ((size_t)doc->b * c->N + doc->start) * c->D + d;
    const double *kd = c->k + (size_t)d * c->L;
    for (int t = 0; t < P; ++t) {
        a[t] = t < doc->len ? xrow[(size_t)t * c->D] : 0.0;
        h[t] = t < taps ? kd[t] : 0.0;
    }
    fft_radix2(a, P, -1);
    fft_radix2(h, P, -1);
    for (int f = 0; f < P; ++f) a[f] *= h[f];
    fft_radix2(a, P, +1);
    double *yrow = c->y + ((size_t)doc->b * c->N + doc->start) * c->D + d;
    for (int t = 0; t < doc->len; ++t) yrow[(size_t)t * c->D] = creal(a[t]) / (double)P;
}

int rco_conv_fft(int B, int N, int D, int L, int max_docs, const int32_t *cu,
                 const double *x, const double *k, double *y, int nthreads) {
    if (D < 1 || L < 1 || !x || !k || !y) return RCO_EBADARG;
    rco_doc *docs = NULL;
    int n = collect_docs(B, N, max_docs, cu, &docs);
    if (n < 0) return n;
    int ml = max_len(docs, n);
    int P = next_pow2((long)ml + (ml < L ? ml : L) - 1);
    conv_ctx ctx = {docs, N, D, L, x, k, y};
    int rc = run_parallel((long)n * D, nthreads, 2 * sizeof(double complex) * (size_t)P,
                          fft_item, &ctx);
    free(docs);
    return rc;
}

/* ------------------------------------------------------------------ sampled */
typedef struct {
    int N, D, L, max_docs;
    const int32_t *cu;
    const double *x, *k;
    const int64_t *btd;
    double *out;
} at_ctx;

static void at_item(void *vctx, long i, void *scratch) {
    (void)scratch;
    const at_ctx *c = (const at_ctx *)vctx;
    int64_t b = c->btd[3 * i], t = c->btd[3 * i + 1], d = c->btd[3 * i + 2];
    const int32_t *row = c->cu + (size_t)b * (c->max_docs + 1);
    int64_t s0 = 0;
    for (int j = 0; j < c->max_docs; ++j)            /* the document holding t */
        if (row[j] <= t && t < row[j + 1]) { s0 = row[j]; break; }
    int64_t last = t - s0 < c->L - 1 ? t - s0 : c->L - 1;
    double acc = 0.0;
    for (int64_t tau = 0; tau <= last; ++tau)
        acc += c->k[d * c->L + tau] * c->x[((size_t)b * c->N + (t - tau)) * c->D + d];
    c->out[i] = acc;
}

/* y at n sampled positions btd[n][3] = (b, t, d). */
int rco_conv_at(int B, int N, int D, int L, int max_docs, const int32_t *cu,
                const double *x, const double *k, long n, const int64_t *btd,
                double *out, int nthreads) {
    if (D < 1 || L < 1 || !x || !k || (n > 0 && (!btd || !out))) return RCO_EBADARG;
    int rc = rco_validate(B, N, max_docs, cu);
    if (rc) return rc;
    for (long i = 0; i < n; ++i)
        if (btd[3 * i] < 0 || btd[3 * i] >= B || btd[3 * i + 1] < 0 || btd[3 * i + 1] >= N ||
            btd[3 * i + 2] < 0 || btd[3 * i + 2] >= D)
            return RCO_EBADARG;
    at_ctx ctx = {N, D, L, max_docs, cu, x, k, btd, out};
    return run_parallel(n, nthreads, 0, at_item, &ctx);
}

/* ------------------------------------------------------------------ gradients
 * The convolution is linear in x and in k, so its gradients are the adjoints of
 * the two linear maps (the transpose of the block-diagonal Toeplitz matrix of
 * Section 3.2, and of the map k -> y).  For an upstream gradient dy:
 *
 *     dx[b,s,d] = sum_{tau = 0}^{min(s1 - 1 - s, L - 1)} k[d,tau] * dy[b,s+tau,d],
 *                 s0 <= s < s1   (anti-causal correlation inside the document);
 *     dk[d,tau] = sum over documents [s0, s1) of every row of
 *                 sum_{t = s0 + tau}^{s1 - 1} dy[b,t,d] * x[b,t-tau,d],   tau < L.
 */
typedef struct {
    const rco_doc *docs;
    int n_docs, N, D, L;
    const double *x, *k, *dy;
    double *dx, *dk;
} grad_ctx;

/* dx for one (document, channel), lags ascending. */
static void grad_x_item(void *vctx, long item, void *scratch) {
    (void)scratch;
    const grad_ctx *c = (const grad_ctx *)vctx;
    const rco_doc *doc = &c->docs[item / c->D];
    int d = (int)(item % c->D);
    const double *kd = c->k + (size_t)d * c->L;
    const double *dyrow = c->dy + ((size_t)doc->b * c->N + doc->start) * c->D + d;
    double *dxrow = c->dx + ((size_t)doc->b * c->N + doc->start) * c->D + d;
    for (int s = 0; s < doc->len; ++s) {
        int last = doc->len - 1 - s < c->L - 1 ? doc->len - 1 - s : c->L - 1;
        double acc = 0.0;
        for (int tau = 0; tau <= last; ++tau) acc += kd[tau] * dyrow[(size_t)(s + tau) * c->D];
        dxrow[(size_t)s * c->D] = acc;
    }
}

int rco_conv_grad_x(int B, int N, int D, int L, int max_docs, const int32_t *cu,
                    const double *k, const double *dy, double *dx, int nthreads) {
    if (D < 1 || L < 1 || !k || !dy || !dx) return RCO_EBADARG;
    rco_doc *docs = NULL;
    int n = collect_docs(B, N, max_docs, cu, &docs);
    if (n < 0) return n;
    grad_ctx ctx = {docs, n, N, D, L, NULL, k, dy, dx, NULL};
    int rc = run_parallel((long)n * D, nthreads, 0, grad_x_item, &ctx);
    free(docs);
    return rc;
}

/* dk for one channel: every document of every row, lags ascending, tokens ascending. */
static void grad_k_item(void *vctx, long d, void *scratch) {
    (void)scratch;
    const grad_ctx *c = (const grad_ctx *)vctx;
    double *dkd = c->dk + (size_t)d * c->L;
    for (int tau = 0; tau < c->L; ++tau) dkd[tau] = 0.0;
    for (int i = 0; i < c->n_docs; ++i) {
        const rco_doc *doc = &c->docs[i];
        const double *xrow = c->x + ((size_t)doc->b * c->N + doc->start) * c->D + d;
        const double *dyrow = c->dy + ((size_t)doc->b * c->N + doc->start) * c->D + d;
        int lags = doc->len < c->L ? doc->len : c->L;
        for (int tau = 0; tau < lags; ++tau) {
            double acc = 0.0;
            for (int t = tau; t < doc->len; ++t)
                acc += dyrow[(size_t)t * c->D] * xrow[(size_t)(t - tau) * c->D];
            dkd[tau] += acc;
        }
    }
}

int rco_conv_grad_k(int B, int N, int D, int L, int max_docs, const int32_t *cu,
                    const double *x, const double *dy, double *dk, int nthreads) {
    if (D < 1 || L < 1 || !x || !dy || !dk) return RCO_EBADARG;
    rco_doc *docs = NULL;
    int n = collect_docs(B, N, max_docs, cu, &docs);
    if (n < 0) return n;
    grad_ctx ctx = {docs, n, N, D, L, x, NULL, dy, NULL, dk};
    int rc = run_parallel(D, nthreads, 0, grad_k_item, &ctx);
    free(docs);
    return rc;
}

/* dk at n sampled entries dt[n][2] = (d, tau). */
typedef struct {
    grad_ctx g;
    const int64_t *dt;
    double *out;
} grad_k_at_ctx;

static void grad_k_at_item(void *vctx, long i, void *scratch) {
    (void)scratch;
    const grad_k_at_ctx *c = (const grad_k_at_ctx *)vctx;
    int64_t d = c->dt[2 * i], tau = c->dt[2 * i + 1];
    double acc = 0.0;
    for (int j = 0; j < c->g.n_docs; ++j) {
        const rco_doc *doc = &c->g.docs[j];
        const double *xrow = c->g.x + ((size_t)doc->b * c->g.N + doc->start) * c->g.D + d;
        const double *dyrow = c->g.dy + ((size_t)doc->b * c->g.N + doc->start) * c->g.D + d;
        for (int64_t t = tau; t < doc->len; ++t)
            acc += dyrow[(size_t)t * c->g.D] * xrow[(size_t)(t - tau) * c->g.D];
    }
    c->out[i] = acc;
}

int rco_conv_grad_k_at(int B, int N, int D, int L, int max_docs, const int32_t *cu,
                       const double *x, const double *dy, long n, const int64_t *dt,
                       double *out, int nthreads) {
    if (D < 1 || L < 1 || !x || !dy || (n > 0 && (!dt || !out))) return RCO_EBADARG;
    for (long i = 0; i < n; ++i)
        if (dt[2 * i] < 0 || dt[2 * i] >= D || dt[2 * i + 1] < 0 || dt[2 * i + 1] >= L)
            return RCO_EBADARG;
    rco_doc *docs = NULL;
    int nd = collect_docs(B, N, max_docs, cu, &docs);
    if (nd < 0) return nd;
    grad_k_at_ctx ctx = {{docs, nd, N, D, L, x, NULL, dy, NULL, NULL}, dt, out};
    int rc = run_parallel(n, nthreads, 0, grad_k_at_item, &ctx);
    free(docs);
    return rc;
}

/* dx at n sampled positions bsd[n][3] = (b, s, d). */
typedef struct {
    int N, D, L, max_docs;
    const int32_t *cu;
    const double *k, *dy;
    const int64_t *bsd;
    double *out;
} grad_x_at_ctx;

static void grad_x_at_item(void *vctx, long i, void *scratch) {
    (void)scratch;
    const grad_x_at_ctx *c = (const grad_x_at_ctx *)vctx;
    int64_t b = c->bsd[3 * i], s = c->bsd[3 * i + 1], d = c->bsd[3 * i + 2];
    const int32_t *row = c->cu + (size_t)b * (c->max_docs + 1);
    int64_t s1 = c->N;
    for (int j = 0; j < c->max_docs; ++j)            /* the document holding s */
        if (row[j] <= s && s < row[j + 1]) { s1 = row[j + 1]; break; }
    int64_t last = s1 - 1 - s < c->L - 1 ? s1 - 1 - s : c->L - 1;
    double acc = 0.0;
    for (int64_t tau = 0; tau <= last; ++tau)
        acc += c->k[d * c->L + tau] * c->dy[((size_t)b * c->N + (s + tau)) * c->D + d];
    c->out[i] = acc;
}

int rco_conv_grad_x_at(int B, int N, int D, int L, int max_docs, const int32_t *cu,
                       const double *k, const double *dy, long n, const int64_t *bsd,
                       double *out, int nthreads) {
    if (D < 1 || L < 1 || !k || !dy || (n > 0 && (!bsd || !out))) return RCO_EBADARG;
    int rc = rco_validate(B, N, max_docs, cu);
    if (rc) return rc;
    for (long i = 0; i < n; ++i)
        if (bsd[3 * i] < 0 || bsd[3 * i] >= B || bsd[3 * i + 1] < 0 || bsd[3 * i + 1] >= N ||
            bsd[3 * i + 2] < 0 || bsd[3 * i + 2] >= D)
            return RCO_EBADARG;
    grad_x_at_ctx ctx = {N, D, L, max_docs, cu, k, dy, bsd, out};
    return run_parallel(n, nthreads, 0, grad_x_at_item, &ctx);
}
