"""Pins of the oracle's gradients (CPU only).

The convolution is linear in x and in k, so its gradients are the adjoints of the two
linear maps.  They are pinned against things other than their own loops: the adjoint
identities against the (separately pinned) forward sum, the transposes of explicit
block-diagonal Toeplitz matrices (Section 3.2), delta filters, impulse inputs, and a
hand-worked example.
"""
import numpy as np
import pytest
import scipy.linalg

import oracle
import workloads as wl
from tests.pins import docs_of


def _cases(seed, n=6, N=40):
    rng = np.random.default_rng(seed)
    for c in range(n):
        B, D = 2, 3
        L = int(rng.choice([1, 3, 17, N + 5]))
        rows = wl.random_rows(rng, B, N, max_len=N // 2 + 3, p_short=0.4)
        cu = wl.cu_from_rows(rows, N)
        yield c, rows, cu, rng.standard_normal((B, N, D)), rng.standard_normal((D, L)), \
            rng.standard_normal((B, N, D))


def test_hand_worked_gradients():
    """Documents [0, 2) and [2, 5), k = (1, 2), x = 1..5, dy = (1, 1, 1, 2, 3), worked by
    hand: dx[s] = k0 dy[s] + k1 dy[s+1] inside the document, dk[tau] = sum dy[t] x[t-tau]."""
    cu = np.array([[0, 2, 5]], dtype=np.int32)
    k = np.array([[1.0, 2.0]])
    x = np.arange(1.0, 6.0).reshape(1, 5, 1)
    dy = np.array([1.0, 1.0, 1.0, 2.0, 3.0]).reshape(1, 5, 1)
    np.testing.assert_array_equal(oracle.grad_x(k, dy, cu)[0, :, 0], [3, 1, 5, 8, 3])
    np.testing.assert_array_equal(oracle.grad_k(x, dy, cu, 2)[0], [29, 19])


def test_adjoint_identities():
    """<y(x), dy> = <x, dx> and <y(k), dy> = <k, dk> with y the pinned forward sum."""
    for c, rows, cu, x, k, dy in _cases(21):
        y = oracle.conv_direct(x, k, cu)
        dx = oracle.grad_x(k, dy, cu)
        dk = oracle.grad_k(x, dy, cu, k.shape[1])
        lhs = float(np.sum(y * dy))
        scale = np.abs(y).sum() * np.abs(dy).max() + 1.0
        assert abs(lhs - float(np.sum(x * dx))) < 1e-12 * scale, c
        assert abs(lhs - float(np.sum(k * dk))) < 1e-12 * scale, c


def test_explicit_matrix_transposes():
    """dx = A^T dy with A the block-diagonal lower-triangular Toeplitz matrix of each
    channel; dk = X^T dy with X[t, tau] = x[t - tau] inside the document (the matrix of
    the map k -> y)."""
    for c, rows, cu, x, k, dy in _cases(22):
        B, N, D = x.shape
        L = k.shape[1]
        dx = oracle.grad_x(k, dy, cu)
        dk = oracle.grad_k(x, dy, cu, L)
        dk_ref = np.zeros_like(dk)
        for b in range(B):
            for d in range(D):
                blocks, xblocks = [], []
                s0 = 0
                for n in rows[b]:
                    col = np.zeros(n)
                    col[:min(n, L)] = k[d, :min(n, L)]
                    blocks.append(scipy.linalg.toeplitz(col, np.r_[col[0], np.zeros(n - 1)]))
                    seg = x[b, s0:s0 + n, d]
                    xb = scipy.linalg.toeplitz(seg, np.r_[seg[0], np.zeros(L - 1)])
                    xblocks.append(xb)
                    s0 += n
                A = scipy.linalg.block_diag(*blocks)
                X = np.vstack(xblocks)
                np.testing.assert_allclose(dx[b, :, d], A.T @ dy[b, :, d], rtol=0, atol=1e-12 * 50)
                dk_ref[d] += X.T @ dy[b, :, d]
        np.testing.assert_allclose(dk, dk_ref, rtol=0, atol=1e-11 * (1 + np.abs(dk_ref).max()))


def test_delta_filters_shift_dy_back():
    """k = e_j: dx[s] = dy[s + j] while s + j stays in the document, else 0 (exact)."""
    rng = np.random.default_rng(23)
    N, D = 50, 2
    rows = wl.random_rows(rng, 2, N, max_len=20, p_short=0.4)
    cu = wl.cu_from_rows(rows, N)
    dy = rng.standard_normal((2, N, D))
    for j in (0, 1, 4):
        k = np.zeros((D, j + 2))
        k[:, j] = 1.0
        dx = oracle.grad_x(k, dy, cu)
        ref = np.zeros_like(dy)
        for b, s0, s1 in docs_of(cu):
            ref[b, s0:s1 - j] = dy[b, s0 + j:s1] if s1 - j > s0 else 0.0
        np.testing.assert_array_equal(dx, ref)


def test_impulse_input_gives_dy_window():
    """x = impulse at (b, s0 + u, d): dk[d, tau] = dy[b, s0 + u + tau, d] for the lags
    that stay in the document and below L; every other channel is 0 (exact)."""
    rng = np.random.default_rng(24)
    N, D, L = 60, 3, 9
    rows = wl.random_rows(rng, 2, N, max_len=25, p_short=0.3)
    cu = wl.cu_from_rows(rows, N)
    dy = rng.standard_normal((2, N, D))
    for b, s0, s1 in docs_of(cu)[:6]:
        u = (s1 - s0) // 2
        x = np.zeros((2, N, D))
        x[b, s0 + u, 1] = 1.0
        dk = oracle.grad_k(x, dy, cu, L)
        ref = np.zeros((D, L))
        n = min(L, s1 - s0 - u)
        ref[1, :n] = dy[b, s0 + u:s0 + u + n, 1]
        np.testing.assert_array_equal(dk, ref)


def test_grad_k_at_matches_grad_k():
    for c, rows, cu, x, k, dy in _cases(25, n=3):
        L = k.shape[1]
        dk = oracle.grad_k(x, dy, cu, L)
        dt = np.array([(d, t) for d in range(dk.shape[0]) for t in range(L)])
        # the same sums, accumulated over documents in one running sum instead of per document
        np.testing.assert_allclose(oracle.grad_k_at(x, dy, cu, L, dt), dk.reshape(-1), rtol=0,
                                   atol=1e-12 * (1 + np.abs(dk).max()))


def test_grad_x_at_matches_grad_x():
    for c, rows, cu, x, k, dy in _cases(26, n=3):
        dx = oracle.grad_x(k, dy, cu)
        bsd = np.array([(b, s, d) for b in range(dx.shape[0]) for s in range(dx.shape[1])
                        for d in range(dx.shape[2])])
        np.testing.assert_array_equal(oracle.grad_x_at(k, dy, cu, bsd), dx.reshape(-1))


@pytest.mark.parametrize("bad", [np.array([[0, 3, 2]]), np.array([[1, 4]])])
def test_gradients_reject_bad_seqlens(bad):
    x = np.zeros((1, 4, 1))
    with pytest.raises(oracle.OracleError):
        oracle.grad_x(np.ones((1, 2)), x, bad.astype(np.int32))
    with pytest.raises(oracle.OracleError):
        oracle.grad_k(x, x, bad.astype(np.int32), 2)
