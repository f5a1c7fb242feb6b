"""The masked Cooley-Tukey oracle (Algorithm 2) against its pins (no GPU).

Algorithm 2 claims the masked stages compute, for every document, exactly the
DFT of that document alone.  The transform is pinned to numpy.fft.fft per
document and to an explicit DFT matrix; the convolution built on it is pinned to
the direct oracle (itself pinned in tests/test_oracle.py).  A mutation test shows
that dropping the mask, the bit reversal or a twiddle sign fails the pins.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from oracle import masked_fft as mf


def _packed(rng, sizes, channels=3):
    n = sum(sizes)
    return rng.standard_normal((n, channels)) + 1j * rng.standard_normal((n, channels))


def _per_doc(y, sizes, fn):
    out, o = np.empty_like(y), 0
    for p in sizes:
        out[o:o + p] = fn(y[o:o + p], axis=0)
        o += p
    return out


@pytest.mark.parametrize("sizes", [
    [1], [2], [8], [1, 1, 1], [4, 1, 2, 8, 1], [16, 2, 2, 32, 1, 4, 64],
    [1, 128, 1, 2, 256],          # unsorted: short documents between long ones
])
def test_masked_fft_is_per_document_fft(sizes):
    rng = np.random.default_rng(len(sizes) * 31 + sum(sizes))
    y = _packed(rng, sizes)
    got = mf.masked_fft(y, sizes)
    ref = _per_doc(y, sizes, np.fft.fft)
    assert np.max(np.abs(got - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))
    inv = mf.masked_fft(got, sizes, inverse=True)
    assert np.max(np.abs(inv - y)) <= 1e-12 * np.max(np.abs(y))
    np.testing.assert_allclose(mf.masked_fft(y, sizes, inverse=True),
                               _per_doc(y, sizes, np.fft.ifft), rtol=0, atol=1e-12)


def test_masked_fft_against_dft_matrix():
    sizes = [4, 2, 1, 8]
    rng = np.random.default_rng(5)
    y = _packed(rng, sizes, channels=1)[:, 0]
    got = mf.masked_fft(y, sizes)
    o = 0
    for p in sizes:
        f = np.arange(p)
        F = np.exp(-2j * np.pi * np.outer(f, f) / p)   # X[f] = sum_t x[t] w_P^(f t)
        assert np.allclose(got[o:o + p], F @ y[o:o + p], rtol=0, atol=1e-12)
        o += p


def test_masked_fft_hand_example():
    # one document [1, 2, 3, 4] (P = 4) and one [5] (P = 1), worked by hand:
    # X = [10, -2+2i, -2, -2-2i]; a length-1 DFT is the identity
    got = mf.masked_fft(np.array([1, 2, 3, 4, 5], dtype=complex), [4, 1])
    assert np.allclose(got, [10, -2 + 2j, -2, -2 - 2j, 5], rtol=0, atol=1e-14)


def test_impulse_stays_in_its_document():
    sizes = [8, 2, 16, 1, 4]
    for doc in range(len(sizes)):
        o = sum(sizes[:doc])
        y = np.zeros(sum(sizes), dtype=complex)
        y[o + sizes[doc] - 1] = 1.0
        z = mf.masked_fft(y, sizes)
        outside = np.ones(len(y), bool)
        outside[o:o + sizes[doc]] = False
        assert np.all(z[outside] == 0)              # exactly: masked factors are 0 or 1


def test_padded_size_rule():
    for n in range(1, 300):
        for L in (1, 7, 64, 1000):
            p = mf.ct_padded_size(n, L)
            need = n + min(n, L) - 1
            assert p >= need and p & (p - 1) == 0 and (p == 1 or p // 2 < need)


@pytest.mark.parametrize("rows,D,L", [
    ([[5, 1, 9, 17]], 3, 32),
    ([[1] * 8, [3, 5]], 2, 4),
    ([[20, 12], [32]], 4, 7),       # L shorter than the documents
    ([[64]], 2, 200),               # L longer than N
])
def test_conv_matches_direct(rows, D, L):
    W = wl.make_case(rows, D, L, seed=sum(map(sum, rows)) + D)
    ref = oracle.conv_direct(W.x, W.filters, W.cu_seqlens)
    got = mf.conv_masked_fft(W.x, W.filters, W.cu_seqlens)
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_conv_matches_direct_tiny_config():
    W = wl.make_config(0)
    ref = oracle.conv_direct(W.x, W.filters, W.cu_seqlens)
    got = mf.conv_masked_fft(W.x, W.filters, W.cu_seqlens)
    assert np.max(np.abs(got - ref)) <= 1e-11 * np.max(np.abs(ref))


def test_conv_with_empty_documents():
    cu = np.array([[0, 0, 3, 3, 8]], dtype=np.int32)
    rng = np.random.default_rng(2)
    x = rng.standard_normal((1, 8, 2))
    k = rng.standard_normal((2, 5))
    np.testing.assert_allclose(mf.conv_masked_fft(x, k, cu), oracle.conv_direct(x, k, cu),
                               rtol=0, atol=1e-12)


# ----------------------------------------------------------------- mutations
def _mutant(kind):
    """A copy of masked_fft with one plausible mistake."""
    def run(y, sizes):
        sizes_, off = mf._layout(sizes)
        y = np.array(y, dtype=np.complex128)
        n = y.shape[0]
        doc_len = np.repeat(np.asarray(sizes_, dtype=np.int64), sizes_)
        local = np.arange(n) - np.repeat(off[:-1], sizes_)
        if kind != "no_bit_reversal":
            perm = np.empty(n, dtype=np.int64)
            for p, o in zip(sizes_, off[:-1]):
                bits = p.bit_length() - 1
                for j in range(p):
                    perm[o + j] = o + mf._bit_reverse(j, bits)
            y = y[perm]
        for s in range(1, max(p.bit_length() - 1 for p in sizes_) + 1):
            m, h = 1 << s, 1 << (s - 1)
            active = np.ones(n, bool) if kind == "no_mask" else doc_len >= m
            r = local % m
            top = r < h
            sign = 1.0 if kind == "twiddle_sign" else -1.0
            w = np.exp(sign * 2j * np.pi * np.where(top, r, r - h) / m)
            tw0 = np.where(active, np.where(top, 1.0, -w), 1.0)
            twf = np.where(active & ~top, 1.0, 0.0)
            twb = np.where(active & top, w, 0.0)
            y = y * tw0 + np.roll(y, h) * twf + np.roll(y, -h) * twb
        return y
    return run


@pytest.mark.parametrize("kind", ["no_mask", "no_bit_reversal", "twiddle_sign"])
def test_pins_catch_mutations(kind):
    sizes = [8, 2, 1, 4, 16]
    rng = np.random.default_rng(9)
    y = _packed(rng, sizes, channels=1)[:, 0]
    ref = _per_doc(y, sizes, np.fft.fft)
    assert np.allclose(_mutant("none")(y, sizes), ref, rtol=0, atol=1e-12)
    assert not np.allclose(_mutant(kind)(y, sizes), ref, rtol=0, atol=1e-6)
