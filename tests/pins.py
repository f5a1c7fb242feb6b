"""Pins for the CPU oracle: checks fixed by the paper's definition and by mathematics.

Each ``pin_*`` takes ``conv(x, k, cu_seqlens) -> y`` (float64 arrays; x ``[B,N,D]``,
k ``[D,L]``, cu ``[B, max_docs+1]``) and raises ``AssertionError`` when the result
contradicts what the definition fixes.  None of them re-types the defining sum:
they compare against library routines (scipy/numpy), explicit matrices, closed
forms, exact special cases and invariants.

The definition (problem statement, Section 1; depthwise causal convolution,
Section 4.1; block-diagonal Toeplitz form, Section 3.2): inside every document
``[s0, s1)`` of a row and for every channel ``d``,
``y[t] = sum_{tau=0}^{min(t-s0, L-1)} k[d, tau] x[t - tau]``.
"""
import json
import os

import numpy as np
import scipy.linalg
import scipy.signal

import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "worked_examples.json")


def _rel(a, b):
    den = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (den if den > 0 else 1.0)


def _match(conv, y, ref, msg=""):
    """Exact for an evaluation that sums in the defining order (``conv.exact``
    true, the default); otherwise equal to within float64 rounding."""
    if getattr(conv, "exact", True):
        np.testing.assert_array_equal(y, ref, err_msg=msg)
    else:
        scale = max(np.abs(ref).max(), 1.0)
        np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12 * scale, err_msg=msg)


def docs_of(cu):
    """(row, start, end) of every non-empty document."""
    out = []
    for b, row in enumerate(np.asarray(cu)):
        for s0, s1 in zip(row[:-1], row[1:]):
            if s1 > s0:
                out.append((b, int(s0), int(s1)))
    return out


# ------------------------------------------------------------------ hand-worked
def pin_golden(conv):
    """Hand-derived outputs of tests/golden/worked_examples.json (exact integers)."""
    with open(GOLDEN) as f:
        g = json.load(f)
    for ex in g["conv"]:
        x = np.array(ex["x"], dtype=np.float64)
        k = np.array(ex["filters"], dtype=np.float64)
        cu = np.array(ex["cu_seqlens"], dtype=np.int32)
        y = conv(x, k, cu)
        np.testing.assert_allclose(y, np.array(ex["y"], dtype=np.float64), rtol=0, atol=1e-12,
                                   err_msg=ex["name"])


# ------------------------------------------------------------------ brute force
def pin_toeplitz(conv, seed=1, cases=6, N=48):
    """y = A x with A = blockdiag over documents of lower-triangular Toeplitz blocks
    built from each channel's first min(len, L) taps (Section 3.2)."""
    rng = np.random.default_rng(seed)
    for c in range(cases):
        B, D = 2, 3
        L = int(rng.choice([1, 3, 17, N + 5]))
        rows = wl.random_rows(rng, B, N, max_len=N // 2 + 3, p_short=0.4)
        cu = wl.cu_from_rows(rows, N)
        x = rng.standard_normal((B, N, D))
        k = rng.standard_normal((D, L))
        y = conv(x, k, cu)
        for b in range(B):
            for d in range(D):
                blocks = []
                for n in rows[b]:
                    col = np.zeros(n)
                    m = min(n, L)
                    col[:m] = k[d, :m]
                    blocks.append(scipy.linalg.toeplitz(col, np.r_[col[0], np.zeros(n - 1)]))
                A = scipy.linalg.block_diag(*blocks)
                ref = A @ x[b, :, d]
                assert _rel(y[b, :, d], ref) < 1e-12, (c, b, d, _rel(y[b, :, d], ref))


def pin_single_document_library(conv, N=257, D=2):
    """One document per row reduces to the plain causal convolution (no wrap at the row
    end): numpy.convolve, scipy.signal.lfilter and a zero-padded numpy FFT."""
    rng = np.random.default_rng(2)
    for L in (N, 40, 1):
        x = rng.standard_normal((1, N, D))
        k = rng.standard_normal((D, L))
        cu = np.array([[0, N]], dtype=np.int32)
        y = conv(x, k, cu)
        for d in range(D):
            r1 = np.convolve(x[0, :, d], k[d])[:N]
            r2 = scipy.signal.lfilter(k[d], [1.0], x[0, :, d])
            n = 1 << int(np.ceil(np.log2(N + L - 1)))
            r3 = np.fft.irfft(np.fft.rfft(x[0, :, d], n) * np.fft.rfft(k[d], n), n)[:N]
            for r in (r1, r2, r3):
                assert _rel(y[0, :, d], r) < 1e-12, (L, d)


# ------------------------------------------------------------------ exact special cases
def pin_delta_input(conv, seed=3):
    """x = unit impulse at (b, s_i + u, d): the document's channel-d output is the
    filter shifted by u, everything else is exactly 0."""
    rng = np.random.default_rng(seed)
    rows = [[5, 1, 9, 3], [2, 14, 2]]
    N, D, L = 18, 3, 7
    cu = wl.cu_from_rows(rows, N)
    k = rng.standard_normal((D, L))
    for (b, s0, s1) in docs_of(cu):
        for u in {0, (s1 - s0) // 2, s1 - s0 - 1}:
            for d in (0, D - 1):
                x = np.zeros((len(rows), N, D))
                x[b, s0 + u, d] = 1.0
                y = conv(x, k, cu)
                ref = np.zeros_like(x)
                n = min(s1 - s0 - u, L)
                ref[b, s0 + u:s0 + u + n, d] = k[d, :n]
                _match(conv, y, ref, f"{b},{s0},{u},{d}")


def pin_delta_filter(conv, seed=4):
    """k = e_0 gives y = x; k = e_j shifts each document by j with j leading zeros."""
    rng = np.random.default_rng(seed)
    rows = [[1, 6, 2, 8], [10, 7]]
    N, D = 17, 2
    cu = wl.cu_from_rows(rows, N)
    x = rng.standard_normal((2, N, D))
    for j, L in ((0, 1), (0, 5), (2, 3), (4, 9)):
        k = np.zeros((D, L))
        k[:, j] = 1.0
        y = conv(x, k, cu)
        ref = np.zeros_like(x)
        for (b, s0, s1) in docs_of(cu):
            ref[b, s0 + j:s1] = x[b, s0:s1 - j] if s1 - j > s0 else 0.0
        _match(conv, y, ref, f"j={j} L={L}")


def pin_bilinearity(conv, seed=5):
    rng = np.random.default_rng(seed)
    rows = wl.random_rows(rng, 2, 40, 15)
    cu = wl.cu_from_rows(rows, 40)
    D, L = 3, 11
    x1, x2 = rng.standard_normal((2, 2, 40, D))
    k1, k2 = rng.standard_normal((2, D, L))
    a, b = 0.7, -1.9
    lhs = conv(a * x1 + b * x2, k1, cu)
    rhs = a * conv(x1, k1, cu) + b * conv(x2, k1, cu)
    assert _rel(lhs, rhs) < 1e-12
    lhs = conv(x1, a * k1 + b * k2, cu)
    rhs = a * conv(x1, k1, cu) + b * conv(x1, k2, cu)
    assert _rel(lhs, rhs) < 1e-12


def pin_leakage(conv, seed=6, N=64):
    """An impulse in document j leaves every other document, and every other row,
    at exactly 0 -- with an undecayed filter as long as the row.  An impulse at a
    row's last token leaves all earlier documents at 0 (no wrap from the row end)."""
    rng = np.random.default_rng(seed)
    rows = [[7, 1, 20, 3, 33], [N]]
    cu = wl.cu_from_rows(rows, N)
    D = 2
    k = rng.standard_normal((D, N))                   # no decay: long lags are live
    for (b, s0, s1) in docs_of(cu) + [(0, N - 1, N)]:
        x = np.zeros((2, N, D))
        t = s0 + int(rng.integers(0, s1 - s0))
        x[b, t, :] = rng.standard_normal(D)
        y = conv(x, k, cu)
        doc = [(bb, a, e) for (bb, a, e) in docs_of(cu) if bb == b and a <= t < e][0]
        inside = np.zeros_like(y, dtype=bool)
        inside[b, doc[1]:doc[2], :] = True
        assert np.all(y[~inside] == 0.0), (b, s0, s1)
        assert np.all(y[b, t, :] != 0.0)


# ------------------------------------------------------------------ closed forms
def pin_prefix_sum(conv, seed=7):
    """k = 1 for every lag (L >= N): per-document prefix sums."""
    rng = np.random.default_rng(seed)
    rows = [[3, 1, 12, 16], [32]]
    N, D = 32, 2
    cu = wl.cu_from_rows(rows, N)
    x = rng.standard_normal((2, N, D))
    y = conv(x, np.ones((D, N + 3)), cu)
    ref = np.zeros_like(x)
    for (b, s0, s1) in docs_of(cu):
        ref[b, s0:s1] = np.cumsum(x[b, s0:s1], axis=0)
    assert _rel(y, ref) < 1e-13


def pin_geometric(conv, seed=8):
    """k[tau] = r^tau for tau < L: y[t] = r y[t-1] + x[t] - r^L x[t-L], with
    y and x taken as 0 before the document start (a state reset per document)."""
    rng = np.random.default_rng(seed)
    rows = [[9, 2, 30, 1, 22], [40, 24]]
    N, D = 64, 2
    cu = wl.cu_from_rows(rows, N)
    x = rng.standard_normal((2, N, D))
    for r, L in ((0.9, N), (-0.7, N), (0.95, 5), (1.0, 13)):
        k = np.tile(r ** np.arange(L, dtype=np.float64), (D, 1))
        y = conv(x, k, cu)
        ref = np.zeros_like(x)
        for (b, s0, s1) in docs_of(cu):
            prev = np.zeros(D)
            for t in range(s0, s1):
                cur = r * prev + x[b, t]
                if t - L >= s0:
                    cur = cur - r ** L * x[b, t - L]
                ref[b, t] = cur
                prev = cur
        assert _rel(y, ref) < 1e-12, (r, L)


# ------------------------------------------------------------------ invariants
def pin_permutation_and_packing(conv, seed=9):
    """Permuting documents inside a row permutes their outputs; a document's output
    is the same packed or alone in a row of its own length."""
    rng = np.random.default_rng(seed)
    lens = [4, 1, 13, 7, 2, 21]
    N, D, L = sum(lens), 2, 9
    k = rng.standard_normal((D, L))
    segs = [rng.standard_normal((n, D)) for n in lens]
    x = np.concatenate(segs)[None]
    y = conv(x, k, wl.cu_from_rows([lens], N))
    perm = rng.permutation(len(lens))
    xp = np.concatenate([segs[i] for i in perm])[None]
    yp = conv(xp, k, wl.cu_from_rows([[lens[i] for i in perm]], N))
    starts = np.r_[0, np.cumsum(lens)]
    pstarts = np.r_[0, np.cumsum([lens[i] for i in perm])]
    for j, i in enumerate(perm):
        a = y[0, starts[i]:starts[i + 1]]
        bb = yp[0, pstarts[j]:pstarts[j + 1]]
        _match(conv, a, bb, "permutation")
        alone = conv(segs[i][None], k, np.array([[0, lens[i]]], dtype=np.int32))[0]
        _match(conv, a, alone, "packed vs alone")


ALL_PINS = [pin_golden, pin_toeplitz, pin_single_document_library, pin_delta_input,
            pin_delta_filter, pin_bilinearity, pin_leakage, pin_prefix_sum, pin_geometric,
            pin_permutation_and_packing]
