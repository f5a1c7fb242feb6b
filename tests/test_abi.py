"""The C-ABI library on the host (no GPU needed): symbols, plan tables, errors.

The document table must match the oracle's segment derivation exactly, and every
transform size must satisfy the causal padding rule of Algorithm 1
(P_i >= L_i + min(L_i, L) - 1, N1 divides P_i) with m_i the smallest listed (then
2^a 3^b 5^c) size that does, or with RUBICONV_EXACT_ROWS = 1 the smallest integer for
rows on the matrix cores (bf16 inputs, m_i <= 128).
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2605_08451_amd as rc
import workloads as wl
from tests.conftest import gpu_available

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")


def header_functions():
    names = set()
    for h in sorted(os.listdir(INCLUDE)):
        if not h.endswith(".h"):
            continue
        text = open(os.path.join(INCLUDE, h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(rubiconv_[a-z_]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function():
    lib = rc.load_library()
    declared = header_functions()
    assert declared, "no declarations parsed"
    for name in declared:
        assert hasattr(lib, name), f"{name} declared in include/ but not exported"
    assert sorted(rc.EXPORTED_SYMBOLS) == declared


def test_library_file_is_in_tree():
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    assert os.path.realpath(rc.library_path()).startswith(os.path.realpath(root))


ROW_SIZES = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                         "paper_2605_08451_amd", "csrc", "row_sizes.hpp")


def listed_row_sizes():
    """Row sizes with a register-resident kernel (the X(m, M1, M2) list)."""
    text = open(ROW_SIZES).read()
    sizes = [(int(m), int(a), int(b)) for m, a, b in
             re.findall(r"X\((\d+),\s*(\d+),\s*(\d+)\)", text)]
    assert sizes and all(m == a * b and a >= b for m, a, b in sizes)
    return sorted(m for m, _, _ in sizes)


#: rows of at most this many points take the matrix-core row kernels on complex fp16
#: grids (bf16 inputs), whose dense blocks apply a DFT of any size
DENSE_MAX_M = 128


def own_row_size(minimal_m, dtype, exact=False):
    """The row size the plan gives a document whose causal padding needs minimal_m grid
    columns, before class merging."""
    listed = listed_row_sizes()
    if exact and dtype == "bf16" and minimal_m <= DENSE_MAX_M:
        return minimal_m
    if minimal_m <= listed[-1]:
        return min(s for s in listed if s >= minimal_m)
    return next(c for c in range(minimal_m, 4 * minimal_m) if _smooth(c))


def _smooth(n):
    for p in (2, 3, 5):
        while n % p == 0:
            n //= p
    return n == 1


@pytest.mark.parametrize("exact", [False, True])
@pytest.mark.parametrize("i", range(5))
@pytest.mark.parametrize("n1", [0, 64])
def test_doc_table_matches_oracle_segments(i, n1, exact, monkeypatch):
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "0")
    monkeypatch.setenv("RUBICONV_EXACT_ROWS", "1" if exact else "0")
    cu = wl.config_cu_seqlens(i)
    D, L, dt = wl.CONFIG_SHAPES[i]
    N = int(cu[0, -1])
    k = 256 if n1 == 0 else n1
    ref = oracle.doc_table(cu, N, L, k)
    try:
        plan = rc.Plan(cu, N=N, D=D, L=L, x_dtype=dt, n1=n1)
    except rc.RubiconvError as e:   # N1 = 64 cannot reach the longest documents of config 4
        assert i == 4 and n1 == 64 and e.status == 3
        return
    t = plan.doc_table()
    np.testing.assert_array_equal(t[:, :4], ref[:, :4])   # row, index, start, length: exact
    m, P = t[:, 4].astype(np.int64), t[:, 5].astype(np.int64)
    np.testing.assert_array_equal(P, k * m)
    # documents of at most DIRECT_MAX tokens take the direct path (m = P = 0), all others
    # a transform
    direct = P == 0
    np.testing.assert_array_equal(direct, t[:, 3] <= plan.info()["direct_max"])
    assert plan.info()["n_direct"] == int(direct.sum())
    P, m, refP = P[~direct], m[~direct], ref[~direct, 4]
    assert np.all(P >= refP), "transform shorter than the causal padding rule allows"
    listed = listed_row_sizes()
    for mi, minimal in zip(m, refP // k):
        if exact and dt == "bf16" and minimal <= DENSE_MAX_M:   # matrix-core rows: the size itself
            assert mi == minimal, (mi, minimal)
            continue
        assert _smooth(int(mi))
        if minimal <= listed[-1]:   # the smallest listed size that is large enough
            assert mi == min(s for s in listed if s >= minimal), (mi, minimal)
        else:                       # the smallest 2^a 3^b 5^c size that is large enough
            assert all(not _smooth(c) for c in range(int(minimal), int(mi))), (mi, minimal)
    info = plan.info()
    assert info["n_docs"] == len(ref) and info["tokens"] == cu.shape[0] * N
    assert info["grid_points"] == int(P.sum())
    assert info["n_classes"] == len(set(m.tolist()))


def _own_sizes(plan_table, k, dtype, exact=False):
    """Each transform document's own row size (no class merging) for the minimal padded
    lengths of the oracle's table."""
    return [own_row_size(-(-int(minimal) // k), dtype, exact) for minimal in plan_table]


#: bytes per grid point and channel pair (in grid elements) of a document and of a
#: filter class, the cost the plan's class merging minimises
DOC_POINT, CLASS_POINT = 10, 3


def _cost(ms):
    return DOC_POINT * sum(ms) + CLASS_POINT * sum(set(ms))


def _brute_force_best_cost(own):
    """The least cost over every choice of classes (each a subset of the documents' own
    sizes that holds the largest one; a document takes the smallest class that fits)."""
    sizes = np.array(sorted(set(own)), dtype=np.int64)
    k = len(sizes)
    counts = np.array([own.count(int(v)) for v in sizes], dtype=np.int64)
    masks = np.arange(1 << (k - 1), dtype=np.int64)
    chosen = ((masks[:, None] >> np.arange(k - 1)) & 1).astype(bool)
    chosen = np.concatenate([chosen, np.ones((len(masks), 1), dtype=bool)], axis=1)
    # the class serving size i: the first chosen size at or after i
    idx = np.where(chosen, np.arange(k), k)
    serve = np.minimum.accumulate(idx[:, ::-1], axis=1)[:, ::-1]
    served = sizes[serve]
    cost = DOC_POINT * (served * counts).sum(axis=1) + CLASS_POINT * (chosen * sizes).sum(axis=1)
    return int(cost.min())


@pytest.mark.parametrize("exact", [False, True])
@pytest.mark.parametrize("i", range(5))
def test_class_merging(i, exact, monkeypatch):
    """With class merging (the default) every document keeps the segment of the oracle's
    table, a transform at least as long as the causal padding asks, and a row size that
    is some document's own size; the merged sizes cost no more than the unmerged ones, and
    no other choice of classes costs less (every subset of the sizes, brute force).  Both
    with listed sizes everywhere and with the matrix-core rows at their own sizes."""
    monkeypatch.setenv("RUBICONV_EXACT_ROWS", "1" if exact else "0")
    cu = wl.config_cu_seqlens(i)
    D, L, dt = wl.CONFIG_SHAPES[i]
    N = int(cu[0, -1])
    ref = oracle.doc_table(cu, N, L, 256)
    t = rc.Plan(cu, N=N, D=D, L=L, x_dtype=dt).doc_table()
    np.testing.assert_array_equal(t[:, :4], ref[:, :4])
    tr = t[:, 5] > 0
    m = [int(v) for v in t[tr, 4]]
    own = _own_sizes(ref[tr, 4], 256, dt, exact)
    assert all(mi >= oi and mi in own for mi, oi in zip(m, own)), (m, own)
    assert np.all(t[tr, 5] >= ref[tr, 4])
    assert _cost(m) <= _cost(own)
    if len(set(own)) <= 20:
        assert _cost(m) == _brute_force_best_cost(own)


def test_class_merging_switch(monkeypatch):
    """RUBICONV_CLASS_MERGE = 0 keeps each document at its own size; anything but 0 or 1
    is rejected when the plan is made."""
    cu = wl.config_cu_seqlens(2)
    D, L, dt = wl.CONFIG_SHAPES[2]
    N = int(cu[0, -1])
    ref = oracle.doc_table(cu, N, L, 256)
    merged = rc.Plan(cu, N=N, D=D, L=L, x_dtype=dt).info()["n_classes"]
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "0")
    t = rc.Plan(cu, N=N, D=D, L=L, x_dtype=dt).doc_table()
    assert [int(v) for v in t[:, 4]] == _own_sizes(ref[:, 4], 256, dt)
    assert merged < len(set(t[:, 4].tolist()))
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "2")
    with pytest.raises(rc.RubiconvError) as e:
        rc.Plan(cu, N=N, D=D, L=L, x_dtype=dt)
    assert e.value.status == 1


def test_empty_documents_are_skipped():
    cu = np.array([[0, 0, 3, 3, 3, 10], [0, 10, 10, 10, 10, 10]], dtype=np.int32)
    t = rc.Plan(cu, N=10, D=2, L=4, x_dtype="f32").doc_table()
    np.testing.assert_array_equal(t[:, :4], [[0, 1, 0, 3], [0, 4, 3, 7], [1, 0, 0, 10]])


@pytest.mark.parametrize("cu,N", [
    ([[1, 5, 10]], 10),          # does not start at 0
    ([[0, 5, 9]], 10),           # does not end at N
    ([[0, 6, 5, 10]], 10),       # decreasing
    ([[0, 11, 10]], 10),         # beyond N
    ([[0, -1, 10]], 10),         # negative
])
def test_bad_seqlens_status(cu, N):
    with pytest.raises(rc.RubiconvError) as e:
        rc.Plan(np.array(cu, dtype=np.int32), N=N, D=4, L=3)
    assert e.value.status == 2


@pytest.mark.parametrize("kw,status", [
    (dict(N=0), 1), (dict(D=0), 1), (dict(L=0), 1), (dict(n1=100), 3), (dict(n1=512), 3),
])
def test_bad_arguments_status(kw, status):
    args = dict(N=8, D=4, L=3, n1=0)
    args.update(kw)
    with pytest.raises(rc.RubiconvError) as e:
        rc.Plan(np.array([[0, max(args["N"], 0)]], dtype=np.int32), **args)
    assert e.value.status == status


def test_too_long_document_is_unsupported():
    N = 600000   # one document: P >= 2N - 1 needs m > 2048 at N1 = 256
    with pytest.raises(rc.RubiconvError) as e:
        rc.Plan(np.array([[0, N]], dtype=np.int32), N=N, D=2, L=N)
    assert e.value.status == 3


def test_32bit_offset_bound_is_unsupported():
    """Column passes address a document with 32-bit buffer offsets (below P D 4 bytes):
    a plan whose longest document would reach 2^30 bytes there is refused, the
    long-context shape (P D 4 = 5.4e8) is not."""
    N = 262144
    cu = np.array([[0, N]], dtype=np.int32)
    with pytest.raises(rc.RubiconvError) as e:
        rc.Plan(cu, N=N, D=2048, L=N, x_dtype="bf16")
    assert e.value.status == 3
    p = rc.Plan(cu, N=N, D=256, L=N, x_dtype="bf16")
    P = int(p.doc_table()[0, 5])
    assert P * 256 * 4 <= 1 << 30 < P * 2048 * 4


def test_null_arguments_rejected_before_any_device_work():
    lib = rc.load_library()
    plan = rc.Plan(np.array([[0, 8]], dtype=np.int32), N=8, D=2, L=3, x_dtype="f32")
    assert lib.rubiconv_packed_conv(None, None, None, None, None, None) == 1
    assert lib.rubiconv_packed_conv(plan.handle, None, None, None, None, None) == 1
    assert lib.rubiconv_filter_spectrum(plan.handle, None, None, None, None) == 1
    assert lib.rubiconv_filter_spectrum(plan.handle, 256, 512, 768 + 1, None) == 1  # misaligned
    assert lib.rubiconv_plan(None, 1, 8, 2, 3, 1, None, 0, 0, 0, None) == 1
    assert lib.rubiconv_spectrum_bytes(None) == 0 and lib.rubiconv_workspace_bytes(None) == 0
    assert lib.rubiconv_status_string(2) == b"invalid cu_seqlens"
    fake = 1 << 20   # never dereferenced: the calls return before launching
    assert lib.rubiconv_packed_conv_backward(None, fake, fake, fake, fake, fake, fake, None) == 1
    assert lib.rubiconv_packed_conv_backward(plan.handle, fake, fake, fake, None, fake, fake, None) == 1
    assert lib.rubiconv_packed_conv_backward(plan.handle, fake, fake, fake, fake, fake, fake + 4, None) == 1
    # the fused backward may run dx and dk in sequence in the dk workspace
    assert plan.dk_workspace_bytes >= plan.workspace_bytes
    lib.rubiconv_plan_destroy(None)


def test_noalloc_rejects_plans_beyond_its_scratch():
    """rubiconv_packed_conv_noalloc refuses, before any device work, a plan whose
    workspace exceeds the library's scratch array (the long-context workload needs
    more), and null arguments."""
    lib = rc.load_library()
    cu = wl.config_cu_seqlens(4)
    plan = rc.Plan(cu, N=int(cu[0, -1]), D=256, L=262144, x_dtype="bf16")
    assert plan.workspace_bytes > rc.NOALLOC_SCRATCH_BYTES
    fake = 1 << 20   # never dereferenced: the call returns before launching
    assert lib.rubiconv_packed_conv_noalloc(plan.handle, fake, fake, fake, None) == 3
    assert lib.rubiconv_packed_conv_noalloc(None, fake, fake, fake, None) == 1
    assert lib.rubiconv_packed_conv_noalloc(plan.handle, None, fake, fake, None) == 1
    small = rc.Plan(np.array([[0, 8]], dtype=np.int32), N=8, D=2, L=3, x_dtype="f32")
    assert small.workspace_bytes <= rc.NOALLOC_SCRATCH_BYTES


def test_noalloc_scratch_size_matches_header():
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    text = open(os.path.join(root, "include", "rubiconv.h")).read()
    m = re.search(r"#define RUBICONV_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == rc.NOALLOC_SCRATCH_BYTES


@pytest.mark.skipif(gpu_available(), reason="checks the host-only plan of a machine without a GPU")
def test_stream_calls_without_device_report_hip_error():
    lib = rc.load_library()
    plan = rc.Plan(np.array([[0, 8]], dtype=np.int32), N=8, D=2, L=3, x_dtype="f32")
    fake = 1 << 20   # never dereferenced: the call returns before launching
    assert lib.rubiconv_packed_conv(plan.handle, fake, fake, fake, fake, None) == 5
    assert lib.rubiconv_filter_spectrum(plan.handle, fake, fake, fake, None) == 5
    assert lib.rubiconv_packed_conv_backward(plan.handle, fake, fake, fake, fake, fake, fake, None) == 5


def test_buffer_sizes_cover_the_layouts():
    cu = wl.config_cu_seqlens(3)
    plan = rc.Plan(cu, N=8192, D=512, L=8192, x_dtype="f32")
    info = plan.info()
    npb = info["n_pair_blocks"]
    assert npb == 16
    # workspace holds at least the complex fp32 document grid of every pair block
    assert plan.workspace_bytes >= npb * 16 * 8 * info["grid_points"]
    assert plan.workspace_bytes % 256 == 0 and plan.spectrum_bytes % 256 == 0


def test_direct_path_defaults(monkeypatch):
    """The direct path runs on the matrix cores for bf16 plans with whole 32-channel
    blocks, for documents of up to 512 tokens, when together they hold at least 1/16 of
    the transform grid: the LM-packing workload's short documents take it, the mid-length
    workload's two short ones do not.  RUBICONV_DIRECT_MFMA = 0 returns to the VALU
    kernel's 64-token limit, and a limit above 512 is refused."""
    def info(i):
        cu = wl.config_cu_seqlens(i)
        D, L, dt = wl.CONFIG_SHAPES[i]
        return rc.Plan(cu, N=int(cu[0, -1]), D=D, L=L, x_dtype=dt).info()
    c1 = info(1)
    assert c1["direct_max"] == 512 and c1["n_direct"] > 20
    assert info(2)["n_direct"] == 0
    monkeypatch.setenv("RUBICONV_DIRECT_MFMA", "0")
    assert info(1)["direct_max"] in (0, 64)
    monkeypatch.setenv("RUBICONV_DIRECT_MFMA", "1")
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "513")
    with pytest.raises(rc.RubiconvError) as e:
        info(1)
    assert e.value.status == 1
