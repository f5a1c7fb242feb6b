"""Seeded synthetic packed-sequence workloads.

This module is shared by the CPU oracle's tests, the GPU parity tests and the
benchmark.  It only draws inputs: document lengths (as ``cu_seqlens``), the
activations ``x`` and the per-channel causal filters.  It holds none of the
convolution's arithmetic.

The paper measures on document lengths sampled from a tokenised FineWeb-Edu
sample (Section 4.1, "Data").  That dataset is not available here; lognormal
and uniform length models of the same shape stand in for it.  Token values are
synthetic in the paper too.

Every workload follows one draw order from ``numpy.random.default_rng(seed)``:
document lengths row by row, then the filter decay rates ``alpha_d``, then the
filter noise ``g[d, t]``, then ``x``.

Layouts (all C-contiguous):
  * ``x``        float32 ``[B, N, D]``, channels last.  For bf16 workloads the
                 values are already rounded to bf16 (round to nearest even), so
                 ``x`` holds exactly what the GPU reads; ``x_bits`` holds the
                 raw bf16 bit patterns (uint16, same shape).
  * ``filters``  float32 ``[D, L]``: ``k_d[t] = g[d, t] * exp(-alpha_d * t / 1024)``.
  * ``cu_seqlens`` int32 ``[B, max_docs + 1]``: per row the prefix sums of the
                 document lengths, starting at 0 and padded with ``N``.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Callable, List, Optional, Sequence

import numpy as np

#: Column size of the four-step grid that the boundary-stress workload (config 3,
#: row 2) alternates with length-1 documents.  It is the library's default.
DEFAULT_N1 = 256


# --------------------------------------------------------------------------- bf16
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); return the bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    flat_u, flat_o = u.reshape(-1), out.reshape(-1)
    step = 1 << 22
    for s in range(0, flat_u.size, step):          # chunked: bounded temporaries
        c = flat_u[s:s + step]
        bias = ((c >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
        # finite inputs only (|x| < 2^128), so c + bias cannot wrap a uint32
        flat_o[s:s + step] = ((c + bias) >> np.uint32(16)).astype(np.uint16)
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(f32_to_bf16_bits(a))


# --------------------------------------------------------------------------- lengths
def pack_rows(draw: Callable[[], int], B: int, N: int) -> List[List[int]]:
    """Fill each of ``B`` rows greedily with drawn lengths; truncate the last to fill ``N``."""
    rows = []
    for _ in range(B):
        row, used = [], 0
        while used < N:
            n = int(draw())
            n = min(n, N - used)
            row.append(n)
            used += n
        rows.append(row)
    return rows


def lognormal_draw(rng: np.random.Generator, median: float, sigma: float, lo: int, hi: int):
    def draw():
        v = int(np.rint(np.exp(rng.normal(np.log(median), sigma))))
        return int(np.clip(v, lo, hi))
    return draw


def uniform_composition(rng: np.random.Generator, total: int, parts: int, minimum: int) -> List[int]:
    """A uniformly drawn composition of ``total`` into ``parts`` parts, each >= ``minimum``."""
    free = total - parts * (minimum - 1)          # compose ``free`` into positive parts
    cuts = np.sort(rng.choice(np.arange(1, free), size=parts - 1, replace=False))
    pieces = np.diff(np.concatenate([[0], cuts, [free]]))
    return [int(p) + minimum - 1 for p in pieces]


def cu_from_rows(rows: Sequence[Sequence[int]], N: int, max_docs: Optional[int] = None) -> np.ndarray:
    """Rows of document lengths -> int32 ``[B, max_docs + 1]`` prefix sums padded with ``N``."""
    nd = max(len(r) for r in rows) if max_docs is None else max_docs
    cu = np.full((len(rows), nd + 1), N, dtype=np.int32)
    for b, r in enumerate(rows):
        if sum(r) != N:
            raise ValueError(f"row {b}: lengths sum to {sum(r)}, expected {N}")
        if len(r) > nd:
            raise ValueError(f"row {b}: {len(r)} documents exceed max_docs={nd}")
        cu[b, 0] = 0
        cu[b, 1:len(r) + 1] = np.cumsum(r)
    return cu


def rows_from_cu(cu: np.ndarray) -> List[List[int]]:
    return [[int(v) for v in np.diff(row) if v > 0] for row in np.asarray(cu)]


# --------------------------------------------------------------------------- workload
@dataclasses.dataclass
class Workload:
    name: str
    B: int
    N: int
    D: int
    L: int
    x_dtype: str                 # "f32" or "bf16"
    y_dtype: str
    cu_seqlens: np.ndarray       # int32 [B, max_docs+1]
    x: np.ndarray                # float32 [B, N, D] (exact device values)
    x_bits: Optional[np.ndarray]  # uint16 [B, N, D] for bf16, else None
    filters: np.ndarray          # float32 [D, L]
    seed: int

    @property
    def max_docs(self) -> int:
        return self.cu_seqlens.shape[1] - 1

    @property
    def n_docs(self) -> int:
        return int((np.diff(self.cu_seqlens, axis=1) > 0).sum())

    def cu_hash(self) -> str:
        return hashlib.sha256(np.ascontiguousarray(self.cu_seqlens).tobytes()).hexdigest()[:16]


def decaying_filters(rng: np.random.Generator, D: int, L: int) -> np.ndarray:
    """k_d[t] = g[d,t] * exp(-alpha_d * t / 1024), alpha_d ~ U[1,8], g ~ N(0,1) (fp32)."""
    alpha = rng.uniform(1.0, 8.0, size=D)
    g = rng.standard_normal((D, L), dtype=np.float32)
    t = np.arange(L, dtype=np.float64)
    out = np.empty((D, L), dtype=np.float32)
    for d in range(D):
        out[d] = (g[d].astype(np.float64) * np.exp(-alpha[d] * t / 1024.0)).astype(np.float32)
    return out


def draw_x(rng: np.random.Generator, B: int, N: int, D: int, x_dtype: str):
    x = rng.standard_normal((B, N, D), dtype=np.float32)
    if x_dtype == "bf16":
        bits = f32_to_bf16_bits(x)
        return bf16_bits_to_f32(bits).reshape(B, N, D), bits.reshape(B, N, D)
    if x_dtype != "f32":
        raise ValueError(x_dtype)
    return x, None


def make_workload(name: str, rows: Sequence[Sequence[int]], D: int, L: int, x_dtype: str,
                  rng: np.random.Generator, seed: int, y_dtype: Optional[str] = None,
                  filters: Optional[np.ndarray] = None) -> Workload:
    """Draw filters and x (in that order) for already-drawn rows of lengths."""
    B, N = len(rows), sum(rows[0])
    cu = cu_from_rows(rows, N)
    k = decaying_filters(rng, D, L) if filters is None else np.ascontiguousarray(filters, np.float32)
    x, bits = draw_x(rng, B, N, D, x_dtype)
    return Workload(name, B, N, D, L, x_dtype, y_dtype or x_dtype, cu, x, bits, k, seed)


# --------------------------------------------------------------------------- configs
CONFIG_NAMES = {
    0: "tiny-fp32 B1xN1024xD4 L1024 (5 docs, uniform composition)",
    1: "lm-packing-bf16 B8xN4096xD768 L4096 (lognormal 512, s1.0)",
    2: "mid-length-bf16 B4xN16384xD1024 L16384 (lognormal 2048, s1.2)",
    3: "boundary-stress-fp32 B4xN8192xD512 L8192",
    4: "long-context-bf16 B1xN262144xD256 L262144 (lognormal 16384, s1.5)",
}
CONFIG_SLUGS = {0: "tiny_fp32", 1: "lm_packing_bf16", 2: "mid_length_bf16",
                3: "boundary_stress_fp32", 4: "long_context_bf16"}


def config_rows(i: int, rng: np.random.Generator, n1: int = DEFAULT_N1) -> List[List[int]]:
    if i == 0:
        return [uniform_composition(rng, 1024, 5, 8)]
    if i == 1:
        return pack_rows(lognormal_draw(rng, 512, 1.0, 16, 4096), 8, 4096)
    if i == 2:
        return pack_rows(lognormal_draw(rng, 2048, 1.2, 32, 16384), 4, 16384)
    if i == 3:
        N = 8192
        row0 = [N]
        row1 = pack_rows(lambda: rng.integers(1, 65), 1, N)[0]
        row2, used = [], 0                      # 1, N1, 1, N1, ... (no draws)
        while used < N:
            n = min(1 if len(row2) % 2 == 0 else n1, N - used)
            row2.append(n)
            used += n
        row3 = pack_rows(lognormal_draw(rng, 300, 1.5, 1, 8192), 1, N)[0]
        return [row0, row1, row2, row3]
    if i == 4:
        return pack_rows(lognormal_draw(rng, 16384, 1.5, 64, 262144), 1, 262144)
    raise ValueError(f"no config {i}")


CONFIG_SHAPES = {  # D, L, x dtype
    0: (4, 1024, "f32"),
    1: (768, 4096, "bf16"),
    2: (1024, 16384, "bf16"),
    3: (512, 8192, "f32"),
    4: (256, 262144, "bf16"),
}


def make_config(i: int, seed: Optional[int] = None) -> Workload:
    """The five packed workloads; ``seed`` defaults to the config index."""
    s = i if seed is None else seed
    rng = np.random.default_rng(s)
    rows = config_rows(i, rng)
    D, L, dt = CONFIG_SHAPES[i]
    return make_workload(f"c{i}", rows, D, L, dt, rng, s)


def config_cu_seqlens(i: int, seed: Optional[int] = None) -> np.ndarray:
    """Only the document boundaries of config ``i`` (cheap: draws no tensors)."""
    s = i if seed is None else seed
    rows = config_rows(i, np.random.default_rng(s))
    return cu_from_rows(rows, sum(rows[0]))


def make_case(rows: Sequence[Sequence[int]], D: int, L: int, x_dtype: str = "f32",
              seed: int = 0, filters: Optional[np.ndarray] = None) -> Workload:
    """A small ad-hoc workload with given rows of document lengths."""
    rng = np.random.default_rng(seed)
    return make_workload("case", rows, D, L, x_dtype, rng, seed, filters=filters)


def random_rows(rng: np.random.Generator, B: int, N: int, max_len: int, p_short: float = 0.2):
    """Ragged rows mixing short (1..8) and longer documents, for edge-case tests."""
    def draw():
        if rng.random() < p_short:
            return int(rng.integers(1, 9))
        return int(rng.integers(1, max_len + 1))
    return pack_rows(draw, B, N)
