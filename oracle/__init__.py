"""CPU oracle for the packed causal long convolution (RubiConv, arXiv 2605.08451).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this package.  It shares no code with the
GPU library and the product path never calls it.

What it computes (problem statement, Section 1 and Section 4.1; the direct
block-diagonal Toeplitz form of Section 3.2): for every row, every document
``[s0, s1)`` given by ``cu_seqlens`` and every channel ``d``::

    y[b, t, d] = sum_{tau=0}^{min(t - s0, L - 1)} k[d, tau] * x[b, t - tau, d]

in float64.  ``conv_direct`` evaluates that sum; ``conv_fft`` evaluates the same
result through a per-document power-of-two radix-2 FFT with the causal zero
padding of Algorithm 1; ``conv_at`` evaluates the sum at sampled positions;
``doc_table`` returns the document table and the minimal padded sizes
``L_i' = k * ceil((L_i + min(L_i, L) - 1) / k)`` of Algorithm 1.

Gradients (the method targets training pipelines, Section 1): the map is linear in
x and in k, so for an upstream gradient ``dy`` the gradients are the adjoints of
the two maps.  ``grad_x`` is the anti-causal correlation inside every document,
``dx[s] = sum_{tau <= min(s1 - 1 - s, L - 1)} k[d, tau] dy[s + tau]``; ``grad_k``
sums ``dy[t] x[t - tau]`` over the tokens of every document of every row for each
lag ``tau < L``; ``grad_x_at`` and ``grad_k_at`` evaluate single entries.

``oracle.masked_fft`` holds the boundary-respecting Cooley-Tukey transform of
Algorithm 2 (masked radix-2 stages over the packed array) and the convolution
built on it, pinned separately (tests/test_oracle_ct.py).

Pins (tests/test_oracle.py, tests/golden/): brute-force block-diagonal Toeplitz
matrices, single documents against library convolutions (numpy.convolve,
scipy.signal.lfilter, numpy.fft), delta inputs and delta filters, bilinearity,
zero leakage across documents and row ends, closed forms (prefix sums,
geometric-filter recurrences with a reset at each document start), document
permutation and packing invariance, direct versus FFT agreement, and hand-worked
examples.  The gradients are pinned by the adjoint identities
``<y(x), dy> = <x, grad_x>`` and ``<y(k), dy> = <k, grad_k>`` against the pinned
forward sum, by the transposes of explicit block-diagonal Toeplitz matrices, and by
delta filters and impulse inputs.  No function here is "parity unpinned".
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None


class OracleError(RuntimeError):
    pass


def _lib():
    global _LIB
    if _LIB is None:
        path = _build.build(force=False)
        lib = ctypes.CDLL(path)
        i32p = ctypes.POINTER(ctypes.c_int32)
        f64p = ctypes.POINTER(ctypes.c_double)
        i64p = ctypes.POINTER(ctypes.c_int64)
        c_int, c_long = ctypes.c_int, ctypes.c_long
        lib.rco_validate.argtypes = [c_int, c_int, c_int, i32p]
        lib.rco_doc_table.argtypes = [c_int, c_int, c_int, i32p, c_int, c_int, i32p, c_int]
        for name in ("rco_conv_direct", "rco_conv_fft"):
            getattr(lib, name).argtypes = [c_int, c_int, c_int, c_int, c_int, i32p,
                                           f64p, f64p, f64p, c_int]
        lib.rco_conv_at.argtypes = [c_int, c_int, c_int, c_int, c_int, i32p, f64p, f64p,
                                    c_long, i64p, f64p, c_int]
        lib.rco_conv_grad_x.argtypes = [c_int, c_int, c_int, c_int, c_int, i32p, f64p, f64p,
                                        f64p, c_int]
        lib.rco_conv_grad_k.argtypes = [c_int, c_int, c_int, c_int, c_int, i32p, f64p, f64p,
                                        f64p, c_int]
        lib.rco_conv_grad_x_at.argtypes = [c_int, c_int, c_int, c_int, c_int, i32p, f64p, f64p,
                                           c_long, i64p, f64p, c_int]
        lib.rco_conv_grad_k_at.argtypes = [c_int, c_int, c_int, c_int, c_int, i32p, f64p, f64p,
                                           c_long, i64p, f64p, c_int]
        lib.rco_default_threads.argtypes = []
        _LIB = lib
    return _LIB


def _p(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _check(rc, what):
    if rc < 0:
        raise OracleError(f"{what}: error {rc} ({'bad cu_seqlens' if rc == -2 else 'bad argument'})")
    return rc


def _prep(x, k, cu):
    x = np.ascontiguousarray(x, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    cu = np.ascontiguousarray(cu, dtype=np.int32)
    if x.ndim != 3 or k.ndim != 2 or cu.ndim != 2:
        raise OracleError("expected x[B,N,D], k[D,L], cu_seqlens[B,max_docs+1]")
    B, N, D = x.shape
    if k.shape[0] != D or cu.shape[0] != B or cu.shape[1] < 2:
        raise OracleError("shape mismatch")
    return x, k, cu, B, N, D, k.shape[1], cu.shape[1] - 1


def default_threads() -> int:
    return int(_lib().rco_default_threads())


def conv_direct(x, k, cu_seqlens, threads: int = 0) -> np.ndarray:
    """The defining sum, float64 (y has x's shape)."""
    x, k, cu, B, N, D, L, nd = _prep(x, k, cu_seqlens)
    y = np.zeros_like(x)
    _check(_lib().rco_conv_direct(B, N, D, L, nd, _p(cu, ctypes.c_int32), _p(x, ctypes.c_double),
                                  _p(k, ctypes.c_double), _p(y, ctypes.c_double), threads),
           "conv_direct")
    return y


def conv_fft(x, k, cu_seqlens, threads: int = 0) -> np.ndarray:
    """Same result through per-document radix-2 FFTs, float64."""
    x, k, cu, B, N, D, L, nd = _prep(x, k, cu_seqlens)
    y = np.zeros_like(x)
    _check(_lib().rco_conv_fft(B, N, D, L, nd, _p(cu, ctypes.c_int32), _p(x, ctypes.c_double),
                               _p(k, ctypes.c_double), _p(y, ctypes.c_double), threads),
           "conv_fft")
    return y


def conv_at(x, k, cu_seqlens, btd, threads: int = 0) -> np.ndarray:
    """The defining sum at positions ``btd[n, 3] = (b, t, d)``."""
    x, k, cu, B, N, D, L, nd = _prep(x, k, cu_seqlens)
    btd = np.ascontiguousarray(btd, dtype=np.int64).reshape(-1, 3)
    out = np.zeros(btd.shape[0], dtype=np.float64)
    _check(_lib().rco_conv_at(B, N, D, L, nd, _p(cu, ctypes.c_int32), _p(x, ctypes.c_double),
                              _p(k, ctypes.c_double), btd.shape[0], _p(btd, ctypes.c_int64),
                              _p(out, ctypes.c_double), threads), "conv_at")
    return out


def grad_x(k, dy, cu_seqlens, threads: int = 0) -> np.ndarray:
    """Gradient of the convolution with respect to x for an upstream gradient dy:
    the anti-causal correlation of dy with k inside every document, float64."""
    dy, k, cu, B, N, D, L, nd = _prep(dy, k, cu_seqlens)
    dx = np.zeros_like(dy)
    _check(_lib().rco_conv_grad_x(B, N, D, L, nd, _p(cu, ctypes.c_int32), _p(k, ctypes.c_double),
                                  _p(dy, ctypes.c_double), _p(dx, ctypes.c_double), threads),
           "grad_x")
    return dx


def grad_x_at(k, dy, cu_seqlens, bsd, threads: int = 0) -> np.ndarray:
    """grad_x at positions ``bsd[n, 3] = (b, s, d)``."""
    dy, k, cu, B, N, D, L, nd = _prep(dy, k, cu_seqlens)
    bsd = np.ascontiguousarray(bsd, dtype=np.int64).reshape(-1, 3)
    out = np.zeros(bsd.shape[0], dtype=np.float64)
    _check(_lib().rco_conv_grad_x_at(B, N, D, L, nd, _p(cu, ctypes.c_int32), _p(k, ctypes.c_double),
                                     _p(dy, ctypes.c_double), bsd.shape[0], _p(bsd, ctypes.c_int64),
                                     _p(out, ctypes.c_double), threads), "grad_x_at")
    return out


def grad_k(x, dy, cu_seqlens, L: int, threads: int = 0) -> np.ndarray:
    """Gradient with respect to the filters, [D, L] float64: per channel and lag, the
    sum over all documents of dy[t] x[t - lag] inside the document."""
    kshape = np.zeros((np.shape(x)[2], L))
    x, _, cu, B, N, D, L, nd = _prep(x, kshape, cu_seqlens)
    dy = np.ascontiguousarray(dy, dtype=np.float64)
    if dy.shape != x.shape:
        raise OracleError("dy must have x's shape")
    dk = np.zeros((D, L), dtype=np.float64)
    _check(_lib().rco_conv_grad_k(B, N, D, L, nd, _p(cu, ctypes.c_int32), _p(x, ctypes.c_double),
                                  _p(dy, ctypes.c_double), _p(dk, ctypes.c_double), threads),
           "grad_k")
    return dk


def grad_k_at(x, dy, cu_seqlens, L: int, dt, threads: int = 0) -> np.ndarray:
    """grad_k at entries ``dt[n, 2] = (d, lag)``."""
    kshape = np.zeros((np.shape(x)[2], L))
    x, _, cu, B, N, D, L, nd = _prep(x, kshape, cu_seqlens)
    dy = np.ascontiguousarray(dy, dtype=np.float64)
    if dy.shape != x.shape:
        raise OracleError("dy must have x's shape")
    dt = np.ascontiguousarray(dt, dtype=np.int64).reshape(-1, 2)
    out = np.zeros(dt.shape[0], dtype=np.float64)
    _check(_lib().rco_conv_grad_k_at(B, N, D, L, nd, _p(cu, ctypes.c_int32), _p(x, ctypes.c_double),
                                     _p(dy, ctypes.c_double), dt.shape[0], _p(dt, ctypes.c_int64),
                                     _p(out, ctypes.c_double), threads), "grad_k_at")
    return out


def validate(cu_seqlens, N: int) -> bool:
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    return _lib().rco_validate(cu.shape[0], N, cu.shape[1] - 1, _p(cu, ctypes.c_int32)) == 0


def doc_table(cu_seqlens, N: int, L: int, k: int) -> np.ndarray:
    """int32 [n_docs, 5]: (row, index in row, start, length, minimal padded length)."""
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    B, nd = cu.shape[0], cu.shape[1] - 1
    cap = B * nd
    out = np.zeros((max(cap, 1), 5), dtype=np.int32)
    n = _check(_lib().rco_doc_table(B, N, nd, _p(cu, ctypes.c_int32), L, k,
                                    _p(out, ctypes.c_int32), cap), "doc_table")
    return out[:n].copy()
