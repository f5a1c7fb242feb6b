"""The CPU oracle against its pins (no GPU).

The oracle is trusted only because these checks pass: library routines,
explicit block-diagonal Toeplitz matrices, hand-worked examples, closed forms,
exact special cases and invariants (tests/pins.py).  The mutation test at the end
shows that plausible mistakes -- a dropped term, a missing reset at a document
boundary, a reversed lag, swapped channels, circular wrap inside a document, a
transposed operand -- each fail at least one pin.
"""
import json

import numpy as np
import pytest

import oracle
import workloads as wl
from tests import pins


def _direct(x, k, cu):
    return oracle.conv_direct(x, k, cu)


def _fft(x, k, cu):
    return oracle.conv_fft(x, k, cu)


_fft.exact = False


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_direct_form_pins(pin):
    pin(_direct)


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_fft_variant_pins(pin):
    pin(_fft)


# ------------------------------------------------------------------ direct vs FFT
def _rel(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


@pytest.mark.parametrize("case", ["c0", "c3-mini", "ragged", "L>N", "L<docs", "D odd"])
def test_direct_matches_fft(case):
    rng = np.random.default_rng(11)
    if case == "c0":
        W = wl.make_config(0)
    elif case == "c3-mini":   # the boundary-stress rows at a reduced size
        rows = [[512], wl.pack_rows(lambda: rng.integers(1, 65), 1, 512)[0],
                [1, 64] * 7 + [1, 56], wl.pack_rows(wl.lognormal_draw(rng, 60, 1.5, 1, 512), 1, 512)[0]]
        W = wl.make_case(rows, D=5, L=512, seed=3)
    elif case == "ragged":
        W = wl.make_case(wl.random_rows(rng, 3, 700, 300), D=4, L=700, seed=4)
    elif case == "L>N":
        W = wl.make_case(wl.random_rows(rng, 2, 300, 200), D=3, L=1000, seed=5)
    elif case == "L<docs":
        W = wl.make_case(wl.random_rows(rng, 2, 900, 600), D=3, L=37, seed=6)
    else:
        W = wl.make_case(wl.random_rows(rng, 2, 400, 250), D=7, L=400, seed=7)
    a = oracle.conv_direct(W.x, W.filters, W.cu_seqlens)
    b = oracle.conv_fft(W.x, W.filters, W.cu_seqlens)
    assert _rel(b, a) < 1e-12


def test_conv_at_matches_direct():
    W = wl.make_config(0)
    y = oracle.conv_direct(W.x, W.filters, W.cu_seqlens)
    rng = np.random.default_rng(0)
    idx = np.stack([rng.integers(0, W.B, 300), rng.integers(0, W.N, 300),
                    rng.integers(0, W.D, 300)], axis=1)
    v = oracle.conv_at(W.x, W.filters, W.cu_seqlens, idx)
    np.testing.assert_array_equal(v, y[idx[:, 0], idx[:, 1], idx[:, 2]])


def test_threads_do_not_change_result():
    W = wl.make_case([[100, 3, 200, 1]], D=6, L=150, seed=2)
    a = oracle.conv_direct(W.x, W.filters, W.cu_seqlens, threads=1)
    b = oracle.conv_direct(W.x, W.filters, W.cu_seqlens, threads=5)
    np.testing.assert_array_equal(a, b)


# ------------------------------------------------------------------ document table
def test_padding_rule_golden():
    """Algorithm 1: L_i' = k ceil((L_i + min(L_i, L) - 1) / k), hand-worked cases."""
    with open(pins.GOLDEN) as f:
        cases = json.load(f)["padding"]["cases"]
    for c in cases:
        cu = np.array([[0, c["len"]]], dtype=np.int32)
        t = oracle.doc_table(cu, c["len"], c["L"], c["k"])
        assert t.shape == (1, 5)
        assert t[0, 4] == c["padded"], c


def test_doc_table_segments():
    cu = np.array([[0, 3, 3, 10, 12, 12], [0, 12, 12, 12, 12, 12]], dtype=np.int32)
    t = oracle.doc_table(cu, 12, 5, 4)
    np.testing.assert_array_equal(t[:, :4], [[0, 0, 0, 3], [0, 2, 3, 7], [0, 3, 10, 2], [1, 0, 0, 12]])
    # padded sizes: 3+3-1=5->8, 7+5-1=11->12, 2+2-1=3->4, 12+5-1=16->16
    np.testing.assert_array_equal(t[:, 4], [8, 12, 4, 16])


@pytest.mark.parametrize("cu", [
    [[1, 5, 10]],          # does not start at 0
    [[0, 5, 9]],           # does not end at N
    [[0, 6, 5, 10]],       # decreasing
    [[0, 11, 10]],         # beyond N then back
])
def test_doc_table_rejects_bad_seqlens(cu):
    with pytest.raises(oracle.OracleError):
        oracle.doc_table(np.array(cu, dtype=np.int32), 10, 4, 4)
    assert not oracle.validate(np.array(cu, dtype=np.int32), 10)


# ------------------------------------------------------------------ mutation test
def _loop(x, k, cu, mutant=None):
    """A slow loop used only to host planted mistakes (never the oracle)."""
    B, N, D = x.shape
    L = k.shape[1]
    if mutant == "transposed-x":
        x = x.reshape(B, D, N).transpose(0, 2, 1)
    if mutant == "transposed-k":
        k = k.reshape(L, D).T
    y = np.zeros((B, N, D))
    for (b, s0, s1) in pins.docs_of(cu):
        n = s1 - s0
        for d in range(D):
            dk = D - 1 - d if mutant == "channel-swap" else d
            for t in range(s0, s1):
                acc = 0.0
                lo = 1 if mutant == "drop-current" else 0
                hi = min(t - s0, L - 1)
                if mutant == "drop-last-tap":
                    hi = min(t - s0, L - 2)
                if mutant == "no-reset":          # lags counted from the row start
                    hi = min(t, L - 1)
                if mutant == "circular":
                    hi = min(n - 1, L - 1)
                for tau in range(lo, hi + 1):
                    if mutant == "anticausal":
                        s = t + tau
                        if s >= s1:
                            continue
                    elif mutant == "circular":
                        s = s0 + (t - s0 - tau) % n
                    else:
                        s = t - tau
                    acc += k[dk, tau] * x[b, s, d]
                y[b, t, d] = acc
    return y


MUTANTS = ["drop-current", "drop-last-tap", "no-reset", "anticausal", "channel-swap",
           "circular", "transposed-x", "transposed-k"]


def test_loop_host_passes_pins():
    """The mutation host itself, with no mistake planted, passes every pin."""
    for pin in pins.ALL_PINS:
        pin(lambda x, k, cu: _loop(x, k, cu))


@pytest.mark.parametrize("mutant", MUTANTS)
def test_each_planted_mistake_fails_a_pin(mutant):
    def conv(x, k, cu):
        return _loop(x, k, cu, mutant)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(conv)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches mutant {mutant}"


# ------------------------------------------------------------------ workloads
def test_config_shapes_and_determinism():
    for i in range(5):
        cu = wl.config_cu_seqlens(i)
        B, N = {0: (1, 1024), 1: (8, 4096), 2: (4, 16384), 3: (4, 8192), 4: (1, 262144)}[i]
        assert cu.shape[0] == B and np.all(cu[:, 0] == 0) and np.all(cu[:, -1] == N)
        assert np.all(np.diff(cu, axis=1) >= 0)
        np.testing.assert_array_equal(cu, wl.config_cu_seqlens(i))
        assert oracle.validate(cu, N)
    rows = wl.rows_from_cu(wl.config_cu_seqlens(0))[0]
    assert len(rows) == 5 and min(rows) >= 8
    r3 = wl.rows_from_cu(wl.config_cu_seqlens(3))
    assert r3[0] == [8192] and max(r3[1]) <= 64
    assert r3[2][:4] == [1, wl.DEFAULT_N1, 1, wl.DEFAULT_N1]


def test_bf16_rounding_is_nearest_even():
    # bf16 keeps 7 mantissa bits: the spacing at 1 is 2^-7.
    v = np.array([1.0 + 2 ** -7, 1.0 + 3 * 2 ** -9, -2.5, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8],
                 dtype=np.float32)
    r = wl.round_to_bf16(v)
    # representable; rounds up; exact; tie -> even (1); tie -> even (1 + 2^-6)
    np.testing.assert_array_equal(r, np.array([1.0 + 2 ** -7, 1.0 + 2 ** -7, -2.5, 1.0,
                                               1.0 + 2 ** -6], dtype=np.float32))
