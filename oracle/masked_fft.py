"""Boundary-respecting Cooley-Tukey FFT and convolution (Algorithm 2, Section 3.1).

TEST INFRASTRUCTURE: like the rest of ``oracle/``, only ``tests/``,
``__graft_entry__.smoke()`` and the CPU baseline leg of ``bench.py`` may use it,
and it shares no code with the GPU library.

The method keeps the iterative radix-2 FFT over the whole packed array and stops
data from crossing document boundaries by masking every butterfly stage:

* every document is zero-padded to a power-of-two length ``P_i``; for a causal
  convolution the padding must also hold the linear (not circular) result, so
  ``P_i`` is the smallest power of two ``>= L_i + min(L_i, L) - 1`` (the causal
  padding rule of Algorithm 1 with the power-of-two size Algorithm 2 needs);
* inside every document the elements are put in bit-reversed order;
* stage ``s = 1 .. max log2 P_i`` (butterfly size ``m = 2^s``) updates every
  element ``i`` at once as ``y*Tw0 + roll(y, m/2)*TwF + roll(y, -m/2)*TwB``,
  where an element whose document is shorter than ``m`` takes the identity
  factors ``(1, 0, 0)`` and every other element the factors of the standard
  stage at its position inside its own document.

With ``l`` the element's index inside its document, ``r = l mod m``,
``h = m/2`` and ``w = exp(-2 pi i / m)`` (forward transform), the standard
radix-2 decimation-in-time stage gives

* top of a butterfly (``r < h``):    ``y'[i] = y[i] + w^r y[i+h]``, so
  ``(Tw0, TwF, TwB) = (1, 0, w^r)``;
* bottom (``r >= h``):               ``y'[i] = y[i-h] - w^(r-h) y[i]``, so
  ``(Tw0, TwF, TwB) = (-w^(r-h), 1, 0)``.

``roll(y, h)[i] = y[i-h]`` and ``roll(y, -h)[i] = y[i+h]`` (numpy's convention).
The inverse transform is the forward transform of the complex conjugate,
conjugated and divided by ``P_i``.  Everything is float64 / complex128.

Pins (tests/test_oracle_ct.py): per-document ``numpy.fft.fft`` on packed arrays
in any document order (the library routine the masked stages must reproduce),
an explicit DFT matrix on tiny documents, exact zeros outside an impulse's
document, and the convolution against the pinned direct oracle.
"""
import numpy as np


def ct_padded_size(length: int, L: int) -> int:
    """Smallest power of two >= length + min(length, L) - 1 (1 for length 1)."""
    need = max(1, length + min(length, L) - 1)
    return 1 << (need - 1).bit_length()


def _bit_reverse(n: int, bits: int) -> int:
    r = 0
    for _ in range(bits):
        r = (r << 1) | (n & 1)
        n >>= 1
    return r


def _layout(sizes):
    sizes = [int(p) for p in sizes]
    for p in sizes:
        if p < 1 or p & (p - 1):
            raise ValueError("every document length must be a power of two")
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    return sizes, off


def masked_fft(y, sizes, inverse: bool = False) -> np.ndarray:
    """Per-document DFTs of the packed array ``y`` (axis 0) by Algorithm 2.

    ``sizes`` lists the power-of-two document lengths in packing order; they must
    sum to ``y.shape[0]``.  Extra axes (channels) are transformed independently.
    ``inverse`` gives the inverse DFT (with the 1/P_i factor).
    """
    sizes, off = _layout(sizes)
    y = np.array(y, dtype=np.complex128, copy=True)
    n = y.shape[0]
    if int(off[-1]) != n:
        raise ValueError("document lengths do not cover the array")
    if inverse:
        y = np.conj(y)
    # document of every element, its index inside it and its document's length
    doc_len = np.repeat(np.asarray(sizes, dtype=np.int64), sizes)
    local = np.arange(n, dtype=np.int64) - np.repeat(off[:-1], sizes)
    # per-document bit reversal
    perm = np.empty(n, dtype=np.int64)
    for p, o in zip(sizes, off[:-1]):
        bits = p.bit_length() - 1
        for j in range(p):
            perm[o + j] = o + _bit_reverse(j, bits)
    y = y[perm]
    max_log2 = max((p.bit_length() - 1 for p in sizes), default=0)
    shape = (n,) + (1,) * (y.ndim - 1)
    for s in range(1, max_log2 + 1):
        m = 1 << s
        h = m // 2
        active = doc_len >= m
        r = local % m
        top = r < h
        ang = -2.0 * np.pi * np.where(top, r, r - h) / m
        w = np.cos(ang) + 1j * np.sin(ang)
        tw0 = np.where(active, np.where(top, 1.0 + 0j, -w), 1.0 + 0j)
        twf = np.where(active & ~top, 1.0 + 0j, 0j)
        twb = np.where(active & top, w, 0j)
        y = (y * tw0.reshape(shape) + np.roll(y, h, axis=0) * twf.reshape(shape)
             + np.roll(y, -h, axis=0) * twb.reshape(shape))
    if inverse:
        y = np.conj(y) / doc_len.reshape(shape)
    return y


def conv_masked_fft(x, k, cu_seqlens) -> np.ndarray:
    """Packed causal convolution through Algorithm 2's transform.

    ``x`` is [B, N, D], ``k`` is [D, L], ``cu_seqlens`` is [B, docs + 1].  Row by
    row, every non-empty document's tokens and the first ``min(L_i, L)`` taps of
    every channel's filter are zero-padded to ``P_i`` and packed in document order;
    both packed arrays are transformed by ``masked_fft``, multiplied pointwise
    and transformed back, and each document keeps its first ``L_i`` outputs.
    """
    x = np.asarray(x, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    B, N, D = x.shape
    L = k.shape[1]
    y = np.zeros((B, N, D), dtype=np.float64)
    for b in range(B):
        docs = [(int(s0), int(s1)) for s0, s1 in zip(cu[b, :-1], cu[b, 1:]) if s1 > s0]
        if not docs:
            continue
        sizes = [ct_padded_size(s1 - s0, L) for s0, s1 in docs]
        total = sum(sizes)
        xp = np.zeros((total, D))
        kp = np.zeros((total, D))
        o = 0
        for (s0, s1), p in zip(docs, sizes):
            n = s1 - s0
            xp[o:o + n] = x[b, s0:s1]
            taps = min(n, L)
            kp[o:o + taps] = k[:, :taps].T
            o += p
        prod = masked_fft(xp, sizes) * masked_fft(kp, sizes)
        out = masked_fft(prod, sizes, inverse=True).real
        o = 0
        for (s0, s1), p in zip(docs, sizes):
            y[b, s0:s1] = out[o:o + s1 - s0]
            o += p
    return y
