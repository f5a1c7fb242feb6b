// plan_build.cpp -- the data-processing step of Algorithm 1 as host tables.
//
// For every document i of length L_i the causal padding rule of Algorithm 1
// asks for a transform of at least L_i + min(L_i, L) - 1 points that N1
// divides.  The row DFT size m_i is the smallest size of row_sizes.hpp's list
// (longer rows: the smallest 2^a 3^b 5^c number) with
// N1 * m_i >= L_i + min(L_i, L) - 1.  With RUBICONV_EXACT_ROWS = 1, rows of at most
// 16 * kMaxDenseBlocks points on complex fp16 grids (the matrix-core row kernels, whose
// dense blocks apply an m-point DFT of any m) take the smallest integer m_i instead:
// fewer grid points, but as many 16-point blocks per row, and measured no faster.
// Any such size gives the same exact
// convolution on [0, L_i) because the circular wrap of the padded product lands
// only on positions >= L_i.  Documents with equal m_i share a size class and
// one filter spectrum; that spectrum keeps Lh = min(L, floor((P + 1) / 2)) taps,
// which covers every lag min(L_i, L) - 1 a document of the class can use and
// still cannot wrap onto an output position < L_i (both follow from
// P >= L_i + min(L_i, L) - 1).
#include "plan_build.hpp"

#include "row_sizes.hpp"

#include <algorithm>
#include <cmath>
#include <complex>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>

namespace rubiconv {

int smooth_ceil(int v) {
    if (v < 1) v = 1;
    for (int n = v;; ++n) {
        int k = n;
        while (k % 2 == 0) k /= 2;
        while (k % 3 == 0) k /= 3;
        while (k % 5 == 0) k /= 5;
        if (k == 1) return n;
    }
}

namespace {

// Radices of m in the order the row DFT applies them: 4s, then 2, 3s, 5s.
int factorize(int m, int8_t* fac) {
    int n = 0;
    while (m % 4 == 0) { fac[n++] = 4; m /= 4; }
    while (m % 2 == 0) { fac[n++] = 2; m /= 2; }
    while (m % 3 == 0) { fac[n++] = 3; m /= 3; }
    while (m % 5 == 0) { fac[n++] = 5; m /= 5; }
    return m == 1 ? n : -1;
}

// Pairs per row task of the generic row kernel: three LDS buffers of two rows of
// m * spb complex values of esz bytes (the grid's element) must fit its LDS budget.
int pairs_per_task(int m, int esz) {
    int spb = kPairsPerBlock;
    if (m <= kMaxFastM) return spb;  // register-resident kernel: 32 lines of m values in LDS
    while (spb > 1 && 6 * m * spb * esz > kRowLdsBytes) spb /= 2;
    return spb;
}

// z[r] = exp(-2 pi i r / period), r < period.  Only the first eighth of the circle is
// evaluated (cos and sin of 2 pi r / period); the rest follows from the exact
// symmetries of the circle, so the table costs period / 8 evaluations.
std::vector<std::complex<double>> unit_circle(int64_t period) {
    std::vector<std::complex<double>> z(static_cast<size_t>(period));
    const double two_pi = 6.283185307179586476925286766559;
    auto direct = [&](int64_t r) {
        const double a = two_pi * static_cast<double>(r) / static_cast<double>(period);
        return std::complex<double>(std::cos(a), -std::sin(a));
    };
    if (period % 8 != 0) {
        for (int64_t r = 0; r < period; ++r) z[r] = direct(r);
        return z;
    }
    const int64_t q = period / 4, e = period / 8;
    std::vector<double> c(q + 1), sn(q + 1);  // cos, sin of 2 pi r / period, r <= period / 4
    for (int64_t r = 0; r <= e; ++r) {
        const double a = two_pi * static_cast<double>(r) / static_cast<double>(period);
        c[r] = std::cos(a);
        sn[r] = std::sin(a);
    }
    for (int64_t r = e + 1; r <= q; ++r) {  // cos(pi/2 - x) = sin x
        c[r] = sn[q - r];
        sn[r] = c[q - r];
    }
    for (int64_t r = 0; r < period; ++r) {
        const int64_t quad = r / q, t = r % q;
        double cr, sr;  // cos, sin of 2 pi r / period
        switch (quad) {
            case 0: cr = c[t]; sr = sn[t]; break;
            case 1: cr = -sn[t]; sr = c[t]; break;
            case 2: cr = -c[t]; sr = -sn[t]; break;
            default: cr = sn[t]; sr = -c[t]; break;
        }
        z[r] = std::complex<double>(cr, -sr);
    }
    return z;
}

void push_twiddles(std::vector<float>& tw, int64_t count, int64_t period, double scale = 1.0) {
    // forward roots w_period^r = exp(-2 pi i r / period)
    const std::vector<std::complex<double>> z = unit_circle(period);
    const size_t base = tw.size();
    tw.resize(base + 2 * static_cast<size_t>(count));
    float* out = tw.data() + base;
    for (int64_t r = 0; r < count; ++r) {
        const std::complex<double>& w = z[r % period];
        out[2 * r] = static_cast<float>(scale * w.real());
        out[2 * r + 1] = static_cast<float>(scale * w.imag());
    }
}

uint16_t to_f16_bits(double v) {
    const _Float16 h = static_cast<_Float16>(static_cast<float>(v));  // round to nearest even
    uint16_t b;
    std::memcpy(&b, &h, 2);
    return b;
}

uint16_t to_bf16_bits(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    u += 0x7fffu + ((u >> 16) & 1u);  // finite inputs only
    return static_cast<uint16_t>(u >> 16);
}

float bf16_value(uint16_t b) {
    const uint32_t u = static_cast<uint32_t>(b) << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// One 16 x 16 complex matrix M (row = output, column = input) as the two real
// 16 x 32 MFMA A-operands A_re = [Re M | -Im M], A_im = [Im M | Re M] with the
// K index interleaving (re, im) of each input; lane l holds row l % 16 and
// K = 8 (l / 16) .. + 7.  kind: 0 = fp16, 1 = bf16 high part, 2 = bf16 low part.
template <class F>
void push_operands(std::vector<uint32_t>* out, F entry, int kind) {
    for (int part = 0; part < 2; ++part) {  // 0: output real part, 1: output imaginary part
        for (int lane = 0; lane < 64; ++lane) {
            uint16_t hv[8];
            for (int i = 0; i < 8; ++i) {
                const int row = lane % 16, kk = 8 * (lane / 16) + i, n = kk / 2, c = kk % 2;
                const std::complex<double> mv = entry(row, n);
                double v = part == 0 ? (c == 0 ? mv.real() : -mv.imag())
                                     : (c == 0 ? mv.imag() : mv.real());
                if (kind == 0) {
                    hv[i] = to_f16_bits(v);
                } else {
                    const uint16_t hi = to_bf16_bits(static_cast<float>(v));
                    hv[i] = kind == 1 ? hi : to_bf16_bits(static_cast<float>(v - bf16_value(hi)));
                }
            }
            for (int w = 0; w < 4; ++w) out->push_back(hv[2 * w] | (static_cast<uint32_t>(hv[2 * w + 1]) << 16));
        }
    }
}

// Index assigned to operand slot s = 4h + i (lane group h, slot i): 4i + h, so
// that the four lane groups of one load or store instruction touch neighbouring
// grid rows (an involution).
int interleave(int s) { return 4 * (s % 4) + s / 4; }

// exp(2 pi i e / 256) for any integer e (the column stages' roots, all 256th roots of
// unity), from one table
std::complex<double> root256(int64_t e) {
    static const std::vector<std::complex<double>> z = unit_circle(256);  // exp(-2 pi i r / 256)
    return std::conj(z[static_cast<size_t>(((e % 256) + 256) % 256)]);
}

}  // namespace

namespace {
void make_mfma_tables(std::vector<uint32_t>* out) {
    // stage 1 contracts over the interleaved input slot; stage 2 produces the
    // interleaved output slot (kernels address rows accordingly)
    auto fwd1 = [](int k1, int s) { return root256(-16 * k1 * interleave(s)); };
    // forward stage 1 in bf16 hi/lo: (re_hi, re_lo, im_hi, im_lo)
    std::vector<uint32_t> hi, lo;
    push_operands(&hi, fwd1, 1);
    push_operands(&lo, fwd1, 2);
    out->insert(out->end(), hi.begin(), hi.begin() + 256);          // re_hi
    out->insert(out->end(), lo.begin(), lo.begin() + 256);          // re_lo
    out->insert(out->end(), hi.begin() + 256, hi.end());            // im_hi
    out->insert(out->end(), lo.begin() + 256, lo.end());            // im_lo
    push_operands(out, fwd1, 0);                                    // forward stage 1, fp16
    for (int k1 = 0; k1 < 16; ++k1)                                 // stage 2, twiddle folded
        push_operands(out, [k1](int s, int n2) {
            const int k2 = interleave(s);
            return root256(-16 * n2 * k2 - n2 * k1);
        }, 0);
    push_operands(out, [](int n2, int s) { return root256(16 * n2 * interleave(s)); }, 0);
    for (int n2 = 0; n2 < 16; ++n2)
        push_operands(out, [n2](int s, int k1) {
            const int n1 = interleave(s);
            return root256(16 * n1 * k1 + n2 * k1);
        }, 0);
}

// batch > 1 (m <= 8, one block): the block-diagonal form for `batch` rows side by side,
// row r at slots r m .. r m + m - 1 in both time and frequency, zero elsewhere.
void make_dense_tables(int m, int n1, std::vector<uint32_t>* out, int batch = 1) {
    const int nb = (m + 15) / 16;
    const double fwd_scale = 1.0 / std::sqrt(static_cast<double>(m));
    const double inv_scale = std::sqrt(static_cast<double>(n1)) / 4.0;
    const std::vector<std::complex<double>> z = unit_circle(m);  // exp(-2 pi i e / m)
    // time-domain points are interleaved within a block (slot s <-> point interleave(s)),
    // so that one load or store instruction covers four neighbouring points; frequencies
    // keep their natural order
    for (int dir = 0; dir < 2; ++dir)
        for (int kb = 0; kb < nb; ++kb)
            for (int jb = 0; jb < nb; ++jb)
                push_operands(out, [=](int row, int n) {
                    int k = dir == 0 ? 16 * kb + row : 16 * jb + n;              // frequency
                    int j = dir == 0 ? 16 * jb + interleave(n) : 16 * kb + interleave(row);  // time
                    if (batch > 1) {  // row k / m of the batch, and the same row for j
                        if (k / m != j / m || k / m >= batch) return std::complex<double>(0.0, 0.0);
                        k %= m;
                        j %= m;
                    }
                    if (k >= m || j >= m) return std::complex<double>(0.0, 0.0);
                    const std::complex<double> w = z[(static_cast<int64_t>(k) * j) % m];
                    return dir == 0 ? w * fwd_scale : std::conj(w) * inv_scale;
                }, 0);
}

void make_partner_tables(int m, int n1, std::vector<uint32_t>* out) {
    const int nb = (m + 15) / 16, S = 16 * nb;
    const double fwd_scale = 1.0 / std::sqrt(static_cast<double>(m));
    const double inv_scale = std::sqrt(static_cast<double>(n1)) / 4.0;
    // the inverse operands are kappa times the conjugates of the forward ones
    const double kappa = inv_scale / fwd_scale;
    const std::vector<std::complex<double>> z = unit_circle(m);  // exp(-2 pi i e / m)
    const size_t start = out->size();
    // one real operand per 16 x 16 block: lane (row, q) holds entries (row, 4 q + c) as
    // (Re, -Im) pairs, c = 0..3; the imaginary output part comes from the same operand
    // applied to -i times the input.  Frequencies are interleaved like the time points,
    // so that block (kb, jb) is symmetric in its two axes and its conjugate is block
    // (kb, jb) of the inverse transform
    for (int kb = 0; kb < nb; ++kb)
        for (int jb = 0; jb < nb; ++jb)
            for (int lane = 0; lane < 64; ++lane)
                for (int c = 0; c < 4; ++c) {
                    const int k = 16 * kb + interleave(lane % 16);            // frequency
                    const int j = 16 * jb + interleave(4 * (lane / 16) + c);  // time
                    std::complex<double> v(0.0, 0.0);
                    if (k < m && j < m) v = z[(static_cast<int64_t>(k) * j) % m] * fwd_scale;
                    out->push_back(to_f16_bits(v.real()) |
                                   (static_cast<uint32_t>(to_f16_bits(-v.imag())) << 16));
                }
    // partner-row twiddles: exp(+2 pi i j / m) as complex fp16, then kappa exp(-2 pi i j / m)
    // as complex fp32, for time points j < S (zero past m), then kappa itself (fp32)
    for (int j = 0; j < S; ++j) {
        const std::complex<double> w = j < m ? std::conj(z[j]) : std::complex<double>(0.0, 0.0);
        out->push_back(to_f16_bits(w.real()) | (static_cast<uint32_t>(to_f16_bits(w.imag())) << 16));
    }
    auto push_f32 = [out](double v) {
        const float f = static_cast<float>(v);
        uint32_t b;
        std::memcpy(&b, &f, 4);
        out->push_back(b);
    };
    for (int j = 0; j < S; ++j) {
        const std::complex<double> w = j < m ? z[j] * kappa : std::complex<double>(0.0, 0.0);
        push_f32(w.real());
        push_f32(w.imag());
    }
    push_f32(kappa);
    // whole 1 KB chunks, as the kernel copies them
    while ((out->size() - start) % 256) out->push_back(0u);
}

// Operand tables depend only on (kind, m, N1): each is computed once per process and
// copied into every plan that needs it.
const std::vector<uint32_t>& cached_tables(int kind, int m, int n1) {
    static std::mutex mu;
    static std::map<std::tuple<int, int, int>, std::vector<uint32_t>> cache;
    std::lock_guard<std::mutex> lock(mu);
    auto it = cache.find({kind, m, n1});
    if (it == cache.end()) {
        std::vector<uint32_t> t;
        if (kind == 0) make_mfma_tables(&t);
        else if (kind == 1) make_dense_tables(m, n1, &t);
        else if (kind == 2) make_partner_tables(m, n1, &t);
        else make_dense_tables(m, n1, &t, 16 / m);
        it = cache.emplace(std::make_tuple(kind, m, n1), std::move(t)).first;
    }
    return it->second;
}
}  // namespace

void build_mfma_tables(std::vector<uint32_t>* out) { *out = cached_tables(0, 0, 0); }

void build_dense_tables(int m, int n1, std::vector<uint32_t>* out) {
    const std::vector<uint32_t>& t = cached_tables(1, m, n1);
    out->insert(out->end(), t.begin(), t.end());
}

void build_partner_tables(int m, int n1, std::vector<uint32_t>* out) {
    const std::vector<uint32_t>& t = cached_tables(2, m, n1);
    out->insert(out->end(), t.begin(), t.end());
}

void build_batch_tables(int m, int n1, std::vector<uint32_t>* out) {
    const std::vector<uint32_t>& t = cached_tables(3, m, n1);
    out->insert(out->end(), t.begin(), t.end());
}

std::vector<int> merge_size_classes(const std::vector<int>& m0, int max_merge_m) {
    std::map<int, int64_t> count;
    for (int m : m0) ++count[m];
    std::vector<int> u;
    std::vector<int64_t> c;
    for (const auto& kv : count) {
        u.push_back(kv.first);
        c.push_back(kv.second);
    }
    const int k = static_cast<int>(u.size());
    // best[j]: cheapest cost of sizes u_0 .. u_{j-1}; first[j]: first size of the last group
    std::vector<int64_t> best(k + 1, 0);
    std::vector<int> first(k + 1, 0);
    for (int j = 1; j <= k; ++j) {
        const int64_t s = u[j - 1];
        int64_t docs = 0;
        best[j] = -1;
        for (int i = j; i >= 1; --i) {
            docs += c[i - 1];
            if (i < j && s > max_merge_m) break;
            const int64_t cost = best[i - 1] + kClassPointCost * s + kDocPointCost * s * docs;
            if (best[j] < 0 || cost < best[j]) {
                best[j] = cost;
                first[j] = i;
            }
        }
    }
    std::map<int, int> to;
    for (int j = k; j >= 1; j = first[j] - 1)
        for (int i = first[j]; i <= j; ++i) to[u[i - 1]] = u[j - 1];
    std::vector<int> out;
    out.reserve(m0.size());
    for (int m : m0) out.push_back(to[m]);
    return out;
}

BuildError build_host_plan(HostPlan* out, int B, int N, int D, int L, int max_docs,
                           const int32_t* cu, int x_dtype, int y_dtype, int n1, int direct_max,
                           bool direct_by_share, bool merge_classes, bool direct_mfma) {
    if (!out || !cu || B < 1 || N < 1 || D < 1 || L < 1 || max_docs < 1) return BuildError::kArg;
    if (x_dtype < 0 || x_dtype > 1 || y_dtype < 0 || y_dtype > 1) return BuildError::kArg;
    if (n1 == 0) n1 = 256;
    int r = 0;
    if (n1 == 64) r = 8;
    else if (n1 == 256) r = 16;
    else return BuildError::kUnsupported;
    // Element offsets are 64-bit; per-row token indices are 32-bit.
    if (static_cast<int64_t>(N) * D > (int64_t(1) << 40)) return BuildError::kUnsupported;

    for (int b = 0; b < B; ++b) {
        const int32_t* c = cu + static_cast<int64_t>(b) * (max_docs + 1);
        if (c[0] != 0 || c[max_docs] != N) return BuildError::kSeqlens;
        for (int k = 0; k < max_docs; ++k)
            if (c[k + 1] < c[k] || c[k + 1] > N) return BuildError::kSeqlens;
    }

    // the matrix-core direct path: bf16 x and dy, channels in blocks of 32
    direct_mfma = direct_mfma && direct_mfma_possible(x_dtype, y_dtype, D);
    if (direct_max < 0 || direct_max > (direct_mfma ? kMaxDirectMfma : kMaxDirect)) return BuildError::kArg;
    if (direct_by_share && direct_max > 0) {
        // the direct path pays once its documents would hold a real share of the
        // transform grid (each at least one whole N1-point column grid); a handful of
        // short documents among long ones stays on the transform path
        int64_t all = 0, shortp = 0;
        for (int b = 0; b < B; ++b) {
            const int32_t* c = cu + static_cast<int64_t>(b) * (max_docs + 1);
            for (int k = 0; k < max_docs; ++k) {
                const int len = c[k + 1] - c[k];
                if (len == 0) continue;
                const int64_t mmin = (static_cast<int64_t>(len) + std::min(len, L) - 1 + n1 - 1) / n1;
                const int64_t P = n1 * mmin;
                all += P;
                if (len <= direct_max) shortp += P;
            }
        }
        if (shortp * kDirectMinShare < all) direct_max = 0;
    }
    HostPlan p;
    p.B = B; p.N = N; p.D = D; p.L = L; p.max_docs = max_docs; p.n1 = n1; p.r = r;
    p.direct_max = direct_max;
    p.x_dtype = x_dtype; p.y_dtype = y_dtype;
    p.grid_half = x_dtype == 1;  // bf16 inputs: complex fp16 grids and spectra
    p.npb = ((D + 1) / 2 + kPairsPerBlock - 1) / kPairsPerBlock;

    // documents and their row DFT sizes (RUBICONV_EXACT_ROWS = 1: matrix-core rows at their
    // own size)
    const char* exact_env = std::getenv("RUBICONV_EXACT_ROWS");
    const bool exact_rows = p.grid_half && exact_env && exact_env[0] == '1';
    std::map<int, int> class_of_m;
    for (int b = 0; b < B; ++b) {
        const int32_t* c = cu + static_cast<int64_t>(b) * (max_docs + 1);
        for (int k = 0; k < max_docs; ++k) {
            int len = c[k + 1] - c[k];
            if (len == 0) continue;
            if (len <= direct_max) {
                Seg s{};
                s.row = b; s.start = c[k]; s.len = len;
                p.direct_docs.push_back(s);
                p.direct_index.push_back(k);
                p.all_docs.push_back(s);
                p.all_index.push_back(k);
                continue;
            }
            int64_t need = static_cast<int64_t>(len) + std::min(len, L) - 1;
            int64_t mmin = (need + n1 - 1) / n1;
            if (mmin > kMaxM) return BuildError::kUnsupported;
            // column passes address a document with 32-bit buffer offsets
            if (static_cast<int64_t>(n1) * mmin * D * 4 > (int64_t(1) << 30)) return BuildError::kUnsupported;
            // matrix-core rows take their own size; listed sizes have register-resident
            // row kernels; longer rows are 5-smooth
            int m = exact_rows && mmin <= 16 * kMaxDenseBlocks ? static_cast<int>(mmin)
                                                                 : fast_row_size(static_cast<int>(mmin));
            if (m == 0) m = smooth_ceil(static_cast<int>(mmin));
            if (m > kMaxM) return BuildError::kUnsupported;
            Seg s{};
            s.row = b; s.start = c[k]; s.len = len; s.m = m; s.P = n1 * m;
            p.docs.push_back(s);
            p.doc_index.push_back(k);
            p.all_docs.push_back(s);
            p.all_index.push_back(k);
        }
    }
    if (merge_classes && p.docs.size() > 1) {
        std::vector<int> m0;
        for (const Seg& s : p.docs) m0.push_back(s.m);
        // the column passes address a document with 32-bit offsets (as checked above)
        const int max_merge_m = static_cast<int>(std::min<int64_t>(
            kMaxM, (int64_t(1) << 30) / (static_cast<int64_t>(n1) * D * 4)));
        const std::vector<int> m1 = merge_size_classes(m0, max_merge_m);
        for (size_t i = 0; i < p.docs.size(); ++i) {
            p.docs[i].m = m1[i];
            p.docs[i].P = n1 * m1[i];
        }
        for (size_t i = 0, k = 0; i < p.all_docs.size(); ++i)
            if (p.all_docs[i].P > 0) p.all_docs[i] = p.docs[k++];
    }
    for (const Seg& s : p.docs) class_of_m[s.m] = 0;

    if (!p.direct_docs.empty()) p.direct_taps = std::min(L, direct_max);
    p.direct_mfma = direct_mfma && !p.direct_docs.empty();
    // size classes, ascending m: twiddles, spectrum offsets, filter taps
    {
        size_t tw_floats = 0;
        for (const auto& kv : class_of_m) tw_floats += 2 * (static_cast<size_t>(kv.first) + static_cast<size_t>(n1) * kv.first);
        p.tw.reserve(tw_floats);
    }
    // long rows on fp16 grids: the first-level size m1 of each class (0: the generic row
    // kernel); sub-rows of at most 64 points if possible, else at most 128
    std::vector<int> lr_m1;
    const char* lr_env = std::getenv("RUBICONV_LONG_ROWS");
    const bool lr_on = p.grid_half && !(lr_env && lr_env[0] == '0');
    for (auto& kv : class_of_m) {
        int m = kv.first;
        int m1 = 0;
        for (int cap : {64, 128}) {
            if (!lr_on || m <= kMaxFastM || m1) break;
            for (int r1 : kLrRadices)
                if (m % r1 == 0 && m / r1 <= cap) { m1 = r1; break; }
        }
        lr_m1.push_back(m1);
        kv.second = static_cast<int>(p.classes.size());
        Seg s{};
        s.m = m; s.P = n1 * m; s.cls = kv.second;
        s.len = static_cast<int32_t>(std::min<int64_t>(L, (static_cast<int64_t>(s.P) + 1) / 2));
        s.tw_off = static_cast<int32_t>(p.tw.size() / 2);
        push_twiddles(p.tw, m, m);             // w_m^h, h < m (row DFTs)
        s.twf_off = static_cast<int32_t>(p.tw.size() / 2);
        // w_P^r / sqrt(N1), r < P: the per-document twiddle of the column passes, which
        // also scale by 1/sqrt(N1) (a power of two, exact)
        push_twiddles(p.tw, s.P, s.P, 1.0 / r);
        s.spb = pairs_per_task(m, p.grid_half ? 4 : 8);
        s.nfac = factorize(m, s.fac);
        p.taps_max = std::max(p.taps_max, s.len);
        p.classes.push_back(s);
    }

    // documents: class data, grid offsets, column and row-task tables
    for (auto& s : p.docs) {
        const Seg& c = p.classes[class_of_m[s.m]];
        s.cls = c.cls; s.tw_off = c.tw_off; s.twf_off = c.twf_off;
        s.spb = c.spb; s.nfac = c.nfac;
        std::copy(c.fac, c.fac + kMaxFactors, s.fac);
        s.grid_off = p.grid_points;
        p.grid_points += s.P;
        s.col0 = static_cast<int32_t>(p.doc_col_seg.size());
        s.task0 = static_cast<int32_t>(p.doc_task_seg.size());
        int idx = static_cast<int>(&s - p.docs.data());
        p.doc_col_seg.insert(p.doc_col_seg.end(), s.m, idx);
        if (s.m > kMaxFastM && lr_m1[s.cls] == 0) {
            p.doc_task_seg.insert(p.doc_task_seg.end(), (n1 / 2 + 1) * (kPairsPerBlock / s.spb), idx);
            p.row_lds_docs = std::max(p.row_lds_docs, 6 * s.m * s.spb * (p.grid_half ? 4 : 8));
        }
    }
    for (auto& s : p.classes) {
        s.grid_off = p.class_points;
        s.spec_off = static_cast<int32_t>(s.grid_off);  // a class's own filter grid
        p.class_points += s.P;
        s.col0 = static_cast<int32_t>(p.cls_col_seg.size());
        int idx = static_cast<int>(&s - p.classes.data());
        p.cls_col_seg.insert(p.cls_col_seg.end(), s.m, idx);
        // documents of this class, in document order
        s.list0 = static_cast<int32_t>(p.class_docs.size());
        for (size_t i = 0; i < p.docs.size(); ++i)
            if (p.docs[i].cls == s.cls) p.class_docs.push_back(static_cast<int32_t>(i));
        s.nlist = static_cast<int32_t>(p.class_docs.size()) - s.list0;
        p.class_ident.push_back(s.cls);
    }
    for (auto& s : p.docs) s.spec_off = p.classes[s.cls].spec_off;  // its class's filter grid
    if (p.class_points > (int64_t(1) << 31) - 1) return BuildError::kUnsupported;
    push_twiddles(p.tw_n1, n1, n1);
    // bf16 inputs, N1 = 256 and whole 32-channel blocks: column passes on the matrix cores
    p.col_mfma = p.grid_half && n1 == 256 && D % 32 == 0;
    if (p.col_mfma) build_mfma_tables(&p.mfma_tab);
    // complex fp16 grids: rows of up to 16 * kMaxDenseBlocks points on the matrix cores
    p.row_dense = p.grid_half;
    // the batched kernel addresses a pair block's grids with 32-bit byte offsets
    // (twice the grids: the sub-row regions of long rows, added below, are at most as large)
    int batch_m = 2 * p.grid_points * 64 < (int64_t(1) << 31) && 2 * p.class_points * 64 < (int64_t(1) << 31)
                      ? kMaxBatchM : 0;
    if (batch_m > 0) {
        // the batched kernel is one more launch: worth it once its rows hold a real share
        // of the grid (RUBICONV_ROW_BATCH = 0 turns it off, 1..8 sets the largest batched
        // row size and drops the share condition)
        const char* v = std::getenv("RUBICONV_ROW_BATCH");
        if (v) {
            batch_m = std::min(batch_m, std::max(0, std::atoi(v)));
        } else {
            int64_t pts = 0;
            for (const Seg& d : p.docs) pts += d.m <= batch_m ? d.P : 0;
            if (pts * kBatchMinShare < p.grid_points) batch_m = 0;
        }
    }
    if (p.row_dense) {
        for (auto& c : p.classes) {
            if (c.m > 16 * kMaxDenseBlocks) continue;
            c.dense_off = static_cast<int32_t>(p.dense_tab.size() / 4);
            if (c.m <= 32)
                build_dense_tables(c.m, n1, &p.dense_tab);
            else
                build_partner_tables(c.m, n1, &p.dense_tab);
            // rows of at most kMaxBatchM points: the block-diagonal tables follow the plain ones
            if (c.m <= batch_m) build_batch_tables(c.m, n1, &p.dense_tab);
        }
        for (auto& s : p.docs) s.dense_off = p.classes[s.cls].dense_off;
        for (int nb = 1; nb <= kMaxDenseBlocks; ++nb) {
            p.dense_list0[nb] = static_cast<int32_t>(p.dense_docs.size());
            for (int32_t d : p.class_docs)
                if ((p.docs[d].m + 15) / 16 == nb) p.dense_docs.push_back(d);
            p.dense_count[nb] = static_cast<int32_t>(p.dense_docs.size()) - p.dense_list0[nb];
        }
        // class groups: consecutive entries of one class (class_docs is in class order),
        // split into near-equal groups of at most `cap` documents.  Rows of at most
        // kMaxBatchM points go to the batched kernel (pass 1), the others to the kernel
        // of their block count (pass 0).
        auto class_groups = [&](int nb, bool batched) {
            const int e0 = p.dense_list0[nb], e1 = e0 + p.dense_count[nb];
            for (int a = e0; a < e1;) {
                int b = a;
                while (b < e1 && p.docs[p.dense_docs[b]].cls == p.docs[p.dense_docs[a]].cls) ++b;
                const int m = p.docs[p.dense_docs[a]].m;
                if ((m <= batch_m) == batched) {
                    const int cap = batched ? kMaxGroupDocs * (16 / m) : kMaxGroupDocs;
                    const int n = b - a, ng = (n + cap - 1) / cap;
                    for (int g = 0, first = a; g < ng; ++g) {
                        const int cnt = n / ng + (g < n % ng ? 1 : 0);
                        p.dense_groups.push_back(first);
                        p.dense_groups.push_back(cnt);
                        first += cnt;
                    }
                }
                a = b;
            }
        };
        for (int nb = 1; nb <= kMaxDenseBlocks; ++nb) {
            p.dense_grp0[nb] = static_cast<int32_t>(p.dense_groups.size() / 2);
            class_groups(nb, false);
            p.dense_grp_n[nb] = static_cast<int32_t>(p.dense_groups.size() / 2) - p.dense_grp0[nb];
        }
        // filter gradient: each class's documents longest first (ties in document order),
        // in near-equal groups of at most kMaxSumDocs
        for (int nb = 1; nb <= kMaxDenseBlocks; ++nb) {
            p.dense_sgrp0[nb] = static_cast<int32_t>(p.dense_sgroups.size() / 2);
            for (const Seg& c : p.classes) {
                if (c.m > 16 * kMaxDenseBlocks || (c.m + 15) / 16 != nb || c.nlist == 0) continue;
                std::vector<int32_t> mem(p.class_docs.begin() + c.list0, p.class_docs.begin() + c.list0 + c.nlist);
                std::stable_sort(mem.begin(), mem.end(),
                                 [&](int32_t a, int32_t b) { return p.docs[a].len > p.docs[b].len; });
                const int n = static_cast<int>(mem.size()), ng = (n + kMaxSumDocs - 1) / kMaxSumDocs;
                for (int g = 0, first = 0; g < ng; ++g) {
                    const int cnt = n / ng + (g < n % ng ? 1 : 0);
                    p.dense_sgroups.push_back(static_cast<int32_t>(p.dense_sdocs.size()));
                    p.dense_sgroups.push_back(cnt);
                    for (int q = 0; q < cnt; ++q) p.dense_sdocs.push_back(mem[first + q]);
                    first += cnt;
                }
            }
            p.dense_sgrp_n[nb] = static_cast<int32_t>(p.dense_sgroups.size() / 2) - p.dense_sgrp0[nb];
        }
        p.dense_bgrp0 = static_cast<int32_t>(p.dense_groups.size() / 2);
        class_groups(1, true);
        p.dense_bgrp_n = static_cast<int32_t>(p.dense_groups.size() / 2) - p.dense_bgrp0;
        for (int k = 0; k < p.dense_count[1]; ++k) {
            const Seg& d = p.docs[p.dense_docs[p.dense_list0[1] + k]];
            if (d.m <= batch_m) p.dense_bwork += d.m;
        }
    }
    // long rows: sub-row regions past the documents' and classes' grids, tables of m2
    for (size_t c = 0; c < p.classes.size(); ++c) {
        const int m1 = lr_m1[c];
        if (m1 == 0) continue;
        const Seg& cs = p.classes[c];
        const int m2 = cs.m / m1;
        const int64_t vcls = p.class_points + p.class_points_lr;
        p.class_points_lr += cs.P;
        const int32_t dense_off = static_cast<int32_t>(p.dense_tab.size() / 4);
        if (m2 <= 32)
            build_dense_tables(m2, n1, &p.dense_tab);
        else
            build_partner_tables(m2, n1, &p.dense_tab);
        p.lr_cls_items.push_back(LrItem{cs.grid_off, vcls, cs.m, m1, m2, cs.tw_off});
        HostPlan::LrLaunch L{m1, (m2 + 15) / 16, 0, 0, 0, 0, 0.0};
        const int first = static_cast<int>(p.lr_idx.size());
        for (const Seg& d : p.docs) {
            if (d.cls != cs.cls) continue;
            const int64_t vdoc = p.grid_points + p.grid_points_lr;
            p.grid_points_lr += d.P;
            p.lr_doc_items.push_back(LrItem{d.grid_off, vdoc, d.m, m1, m2, d.tw_off});
            Seg v = d;
            v.m = m2;
            v.grid_off = vdoc;
            v.spec_off = static_cast<int32_t>(vcls);
            v.dense_off = dense_off;
            p.lr_segs.push_back(v);
            v.spec_off = static_cast<int32_t>(vdoc);  // the filter gradient's own rows
            p.lr_gsegs.push_back(v);
            p.lr_idx.push_back(static_cast<int32_t>(p.lr_segs.size()) - 1);
            L.work += d.m;
        }
        const int n = static_cast<int>(p.lr_idx.size()) - first;
        const int ng = (n + kMaxGroupDocs - 1) / kMaxGroupDocs;
        L.grp0 = static_cast<int>(p.lr_groups.size() / 2);
        for (int g = 0, f = first; g < ng; ++g) {
            const int cnt = n / ng + (g < n % ng ? 1 : 0);
            p.lr_groups.push_back(f);
            p.lr_groups.push_back(cnt);
            f += cnt;
        }
        L.grp_n = ng;
        L.dgrp0 = static_cast<int>(p.lr_groups.size() / 2);
        for (int k = 0; k < n; ++k) {
            p.lr_groups.push_back(first + k);
            p.lr_groups.push_back(1);
        }
        L.dgrp_n = n;
        p.lr_launches.push_back(L);
    }
    if (p.class_points + p.class_points_lr > (int64_t(1) << 31) - 1 ||
        p.grid_points + p.grid_points_lr > (int64_t(1) << 31) - 1)
        return BuildError::kUnsupported;
    // 32-bit buffer offsets: the column passes address a document's tokens and grid
    // points (and a size class's taps) with offsets below P D 4 bytes, after the final
    // row sizes (rounding and class merging may have raised them); the row kernels
    // address a pair block's grid (and second grid) with offsets below its byte size
    const int64_t pb_point_bytes = p.grid_half ? 64 : 128;
    for (const Seg& d : p.docs)
        if (static_cast<int64_t>(d.P) * D * 4 > (int64_t(1) << 30)) return BuildError::kUnsupported;
    for (const Seg& c : p.classes)
        if (static_cast<int64_t>(c.P) * D * 4 > (int64_t(1) << 30)) return BuildError::kUnsupported;
    if ((p.grid_points + p.grid_points_lr) * pb_point_bytes >= (int64_t(1) << 31) ||
        (p.class_points + p.class_points_lr) * pb_point_bytes >= (int64_t(1) << 31))
        return BuildError::kUnsupported;
    // filter gradient outputs: every document but the sum groups' followers
    {
        std::vector<char> follower(p.docs.size(), 0);
        for (size_t g = 0; g + 1 < p.dense_sgroups.size(); g += 2)
            for (int q = 1; q < p.dense_sgroups[g + 1]; ++q) follower[p.dense_sdocs[p.dense_sgroups[g] + q]] = 1;
        int32_t col = 0;
        for (size_t i = 0, k = 0; i < p.all_docs.size(); ++i) {
            if (p.all_docs[i].P == 0) {  // a direct document: its sums go straight to the lag sum
                p.dk_sum_segs.push_back(p.all_docs[i]);
                continue;
            }
            const size_t d = k++;
            if (follower[d]) continue;
            Seg s = p.docs[d];
            s.spec_off = static_cast<int32_t>(s.grid_off);  // second rows: its own x grid
            s.col0 = col;
            p.dk_col_seg.insert(p.dk_col_seg.end(), s.m, static_cast<int32_t>(p.dk_segs.size()));
            col += s.m;
            p.dk_segs.push_back(s);
            p.dk_sum_segs.push_back(s);
        }
        std::stable_sort(p.dk_sum_segs.begin(), p.dk_sum_segs.end(),
                         [](const Seg& a, const Seg& b) { return a.len > b.len; });
    }
    *out = std::move(p);
    return BuildError::kOk;
}

}  // namespace rubiconv
