"""The HIP path against the oracle on the same seeded inputs (needs an MI355X).

Bars: relative L2 <= 1e-4 for fp32 workloads and <= 2e-2 for bf16 inputs with
fp32 accumulation, both over the whole output and over every document; zero
cross-document leakage.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as wl
from tests.common import (ORACLE_THREADS, TOL, assert_parity, parity_report, reference,
                          rel_l2, run_gpu, to_device)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


# ------------------------------------------------------------------ the five workloads
@pytest.mark.parametrize("i,method", [(0, "direct"), (1, "direct"), (3, "direct"), (2, "fft"),
                                      (4, "fft")])
def test_config_parity(device, i, method):
    _say(f"[parity] config {i} ({wl.CONFIG_NAMES[i]}), oracle {method}")
    W = wl.make_config(i)
    y, plan = run_gpu(W, device)
    ref = reference(W, method)
    g, d = assert_parity(y, ref, W.cu_seqlens, W.x_dtype, f"config {i}")
    _say(f"[parity] config {i}: global {g:.2e}, worst document {d:.2e}, docs {W.n_docs}")


@pytest.mark.parametrize("i", [2, 4])
def test_full_size_sampled_direct_sums(device, i):
    """The bench workloads at full size, sampled entries against the defining sum."""
    W = wl.make_config(i)
    y, _ = run_gpu(W, device)
    rng = np.random.default_rng(100 + i)
    n = 4000
    btd = np.stack([rng.integers(0, W.B, n), rng.integers(0, W.N, n), rng.integers(0, W.D, n)], 1)
    # include the first and last token of every document
    extra = []
    for b, row in enumerate(W.cu_seqlens):
        for s0, s1 in zip(row[:-1], row[1:]):
            if s1 > s0:
                extra += [(b, s0, rng.integers(W.D)), (b, s1 - 1, rng.integers(W.D))]
    btd = np.concatenate([btd, np.array(extra, dtype=np.int64)])
    ref = oracle.conv_at(W.x, W.filters, W.cu_seqlens, btd, threads=ORACLE_THREADS)
    got = y[btd[:, 0], btd[:, 1], btd[:, 2]]
    err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert err <= TOL[W.x_dtype], err


# ------------------------------------------------------------------ edge cases
N1_EDGE = [1, 255, 256, 257, 511, 512, 513]


@pytest.mark.parametrize("n1", [256, 64])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ragged_edges(device, n1, dtype):
    """Documents of length 1, N1 - 1, N1, N1 + 1, whole rows; L shorter and longer than them."""
    rng = np.random.default_rng(7)
    N = 2048
    rows = [[N],
            [1] * 5 + [n1 - 1, n1, n1 + 1] + [N - 5 - 3 * n1],
            wl.random_rows(rng, 1, N, 300, p_short=0.5)[0],
            [N - 1, 1]]
    for L in (1, 7, 300, N, 3 * N):
        W = wl.make_case(rows, D=6, L=L, x_dtype=dtype, seed=L)
        y, _ = run_gpu(W, device, n1=n1)
        assert_parity(y, reference(W), W.cu_seqlens, dtype, f"L={L}")


@pytest.mark.parametrize("D", [1, 2, 3, 8, 31, 33, 64, 96, 200])
def test_channel_counts(device, D):
    """Odd D (a lone last channel), D below and above one pair block of 32 channels, and
    D % 8 = 0 with partial 64-channel tiles of the filter transpose (96, 200)."""
    rng = np.random.default_rng(D)
    rows = wl.random_rows(rng, 2, 1000, 400)
    for dtype in ("f32", "bf16"):
        W = wl.make_case(rows, D=D, L=500, x_dtype=dtype, seed=D)
        y, _ = run_gpu(W, device)
        assert_parity(y, reference(W), W.cu_seqlens, dtype, f"D={D} {dtype}")


@pytest.mark.parametrize("N", [1, 2, 5, 100, 4096])
def test_short_rows(device, N):
    rng = np.random.default_rng(N)
    rows = wl.random_rows(rng, 3, N, max(1, N // 3))
    W = wl.make_case(rows, D=4, L=N + 3, seed=N)
    y, _ = run_gpu(W, device)
    assert_parity(y, reference(W), W.cu_seqlens, "f32", f"N={N}")


def test_mixed_dtypes(device):
    """bf16 input with fp32 output, and fp32 input with bf16 output."""
    rng = np.random.default_rng(3)
    rows = wl.random_rows(rng, 2, 3000, 1500)
    W = wl.make_case(rows, D=8, L=3000, x_dtype="bf16", seed=3)
    y, _ = run_gpu(W, device, y_dtype="f32")   # bf16 inputs: the bf16 bar applies
    assert_parity(y, reference(W), W.cu_seqlens, "bf16", "bf16 -> f32")
    W = wl.make_case(rows, D=8, L=3000, x_dtype="f32", seed=4)
    y, _ = run_gpu(W, device, y_dtype="bf16")
    assert_parity(y, reference(W), W.cu_seqlens, "bf16", "f32 -> bf16")


def test_leakage_impulses(device):
    """An impulse in document j, with an undecayed filter as long as the row, leaves every
    other document and row below 1e-6 of the impulse document's peak."""
    N, D = 4096, 4
    rng = np.random.default_rng(11)
    rows = [[1, 255, 256, 257, 1000, N - 1769], [N]]
    cu = wl.cu_from_rows(rows, N)
    k = rng.standard_normal((D, N)).astype(np.float32)   # no decay: long lags are live
    docs = [(b, int(s0), int(s1)) for b, r in enumerate(cu) for s0, s1 in zip(r[:-1], r[1:])
            if s1 > s0] + [(0, N - 1, N)]
    for (b, s0, s1) in docs:
        W = wl.make_case(rows, D=D, L=N, seed=0, filters=k)
        W.x[:] = 0.0
        t = s0 + int(rng.integers(0, s1 - s0))
        W.x[b, t, :] = rng.standard_normal(D)
        y, _ = run_gpu(W, device)
        inside = np.zeros(y.shape, dtype=bool)
        e = [(bb, a, z) for (bb, a, z) in docs[:-1] if bb == b and a <= t < z][0]
        inside[b, e[1]:e[2]] = True
        peak = np.abs(y[inside]).max()
        assert peak > 0
        assert np.abs(y[~inside]).max() <= 1e-6 * peak, (b, s0, s1)
        # causal: before the impulse only transform rounding remains (zero in exact arithmetic)
        assert np.abs(y[b, e[1]:t]).max(initial=0.0) <= 1e-6 * peak, (b, s0, s1)


def test_delta_filter_is_identity(device):
    rng = np.random.default_rng(5)
    rows = wl.random_rows(rng, 2, 3000, 1200)
    D = 16
    k = np.zeros((D, 50), dtype=np.float32)
    k[:, 0] = 1.0
    W = wl.make_case(rows, D=D, L=50, seed=5, filters=k)
    y, _ = run_gpu(W, device)
    assert np.abs(y - W.x).max() <= 1e-5 * np.abs(W.x).max()


def test_deterministic(device):
    W = wl.make_case(wl.random_rows(np.random.default_rng(2), 2, 5000, 3000), D=40, L=5000,
                     x_dtype="bf16", seed=2)
    ys, _ = run_gpu(W, device, repeats=3)
    for y in ys[1:]:
        np.testing.assert_array_equal(y, ys[0])


def test_plan_reused_with_two_filters(device):
    import torch
    import paper_2605_08451_amd as rc
    from tests.common import to_device
    rows = wl.random_rows(np.random.default_rng(9), 2, 2500, 900)
    W1 = wl.make_case(rows, D=10, L=2500, seed=1)
    W2 = wl.make_case(rows, D=10, L=2500, seed=2)
    plan = rc.Plan(W1.cu_seqlens, N=W1.N, D=W1.D, L=W1.L, x_dtype="f32")
    ws = plan.new_workspace(device)
    for W in (W1, W2, W1):
        x, k = to_device(W, device)
        spec = rc.filter_spectrum(plan, k, workspace=ws)
        y = rc.packed_conv(plan, x, spec, workspace=ws)
        torch.cuda.synchronize()
        assert_parity(y.cpu().numpy().astype(np.float64), reference(W), W.cu_seqlens, "f32")


@pytest.mark.parametrize("D", [32, 96])
@pytest.mark.parametrize("y_dtype", ["bf16", "f32"])
def test_matrix_core_column_path(device, D, y_dtype, monkeypatch):
    """bf16 inputs with whole 32-channel blocks take the matrix-core column passes:
    documents of length 1, N1 - 1, N1, N1 + 1, whole rows, short and long filters."""
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "0")   # every document on the transform path
    rng = np.random.default_rng(D)
    N = 3000
    rows = [[N], [1, 255, 256, 257, 1, 2230], wl.random_rows(rng, 1, N, 700, p_short=0.4)[0]]
    for L in (5, 600, N):
        W = wl.make_case(rows, D=D, L=L, x_dtype="bf16", seed=L + D)
        y, _ = run_gpu(W, device, y_dtype=y_dtype)
        assert_parity(y, reference(W), W.cu_seqlens, "bf16", f"D={D} L={L} y={y_dtype}")


@pytest.mark.parametrize("D", [32, 40])
def test_row_pass_every_block_count(device, D, monkeypatch):
    """bf16 inputs (complex fp16 grids): documents whose row DFT sizes cover every
    matrix-core block count (m <= 16, 17..32, ..., 113..128, at and next to the block
    edges) and the register-resident sizes above it (135, 160, 256).  A length of
    128 m needs exactly m grid columns at N1 = 256."""
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "0")   # every document on the transform path
    rows = [[32768],
            [20480, 12288],
            [17280, 12800, 2304, 384],
            [16384, 10368, 4608, 1408],
            [9216, 8192, 6400, 4096, 2048, 1920, 896]]
    W = wl.make_case(rows, D=D, L=32768, x_dtype="bf16", seed=D)
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "0")   # every document at its own size
    y, plan = run_gpu(W, device)
    ms = sorted(set(int(m) for m in plan.doc_table()[:, 4]))
    assert ms == [3, 8, 12, 15, 16, 18, 32, 36, 50, 64, 72, 81, 96, 100, 128, 135, 160, 256], ms
    assert_parity(y, reference(W, "fft"), W.cu_seqlens, "bf16", f"D={D}")


@pytest.mark.parametrize("n1", [64, 256])
def test_long_row_sizes_precision(device, n1, monkeypatch):
    """Row sizes 33..128 (the partner-row matrix-core kernel), including the rows that
    are their own partners (u = 0 and u = N1 / 2), at a bar tighter than the parity
    tolerance: a wrong value in one grid row of a document shows up as an error of a
    few percent on a few positions, which the 2e-2 bar alone could miss.  Healthy
    errors here are about 2e-3 (bf16 output rounding plus fp16 grids)."""
    ks = (34, 40, 45, 54, 64, 90, 126)
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "0")   # every document at its own size
    for short_filter in (True, False):
        # P >= len + min(len, L) - 1: about len for a 7-tap filter, 2 len for a full one
        lens = [n1 * (k - 1) + 3 if short_filter else n1 * k // 2 + 3 for k in ks]
        N = max(lens)
        L = 7 if short_filter else N
        rows = [[ln, N - ln] if ln < N else [ln] for ln in lens]
        W = wl.make_case(rows, D=6, L=L, x_dtype="bf16", seed=L)
        y, plan = run_gpu(W, device, n1=n1)
        ms = sorted(set(int(m) for m in plan.doc_table()[:, 4]))
        assert max(ms) > 100 and sum(33 <= m <= 128 for m in ms) >= 5, ms
        g, d = assert_parity(y, reference(W, "fft"), W.cu_seqlens, "bf16", f"n1={n1} L={L}")
        assert d <= 5e-3, (n1, L, d)


@pytest.mark.parametrize("family", ["lds", "batch", "partner"])
def test_row_kernel_sizes_precision(device, family, monkeypatch):
    """The same tight bar (5e-3 per document) for the other matrix-core row kernels on the
    matrix-core column path (D = 32): rows of 2..32 points (row_lds_kernel), rows of at
    most 8 points batched 16 / m documents to a block (row_batch_kernel) and rows of
    33..128 points (row_partner_kernel), every size as its own class: 2^a 3^b 5^c sizes
    and, with rows at their own sizes (RUBICONV_EXACT_ROWS = 1), the others (primes among
    them), which these kernels take as they are."""
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "0")   # every document on the transform path
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "0")
    monkeypatch.setenv("RUBICONV_EXACT_ROWS", "1")
    n1 = 256
    if family == "lds":
        ks = (2, 3, 4, 5, 6, 8, 9, 10, 12, 15, 16, 18, 20, 24, 25, 27, 30, 32,
              7, 11, 13, 14, 17, 19, 21, 22, 23, 26, 28, 29, 31)
        monkeypatch.setenv("RUBICONV_ROW_BATCH", "0")
    elif family == "batch":
        ks = (1, 2, 3, 4, 5, 6, 8, 1, 2, 4, 8, 7, 7, 3)
        monkeypatch.setenv("RUBICONV_ROW_BATCH", "8")
    else:
        ks = (36, 40, 45, 48, 50, 54, 60, 64, 72, 75, 80, 81, 90, 96, 100, 108, 120, 128,
              33, 37, 41, 44, 47, 53, 59, 61, 67, 71, 77, 83, 89, 97, 101, 109, 113, 127)
    # a 7-tap filter: P >= len + 6, so a document of n1 (k - 1) + 3 tokens takes m = k
    lens = [n1 * (k - 1) + 3 if k > 1 else 100 + 7 * i for i, k in enumerate(ks)]
    N = max(lens) + 1
    rows = [[ln, N - ln] for ln in lens]
    W = wl.make_case(rows, D=32, L=7, x_dtype="bf16", seed=len(ks))
    y, plan = run_gpu(W, device, n1=n1)
    ms = sorted(set(int(m) for m in plan.doc_table()[:, 4]))
    assert all(k in ms for k in ks), (ks, ms)
    g, d = assert_parity(y, reference(W, "fft"), W.cu_seqlens, "bf16", family)
    print(f"[row kernels] {family}: global {g:.2e}, worst document {d:.2e}", file=sys.stderr, flush=True)
    assert d <= 5e-3, (family, d)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_direct_path_limits(device, monkeypatch, dtype):
    """Short documents by their defining sums (the direct path) at several length limits,
    including rows made only of short documents and a limit above every document: the
    forward and both gradients meet the oracle bar at each limit."""
    import tests.test_gpu_grad as tg
    rng = np.random.default_rng(31)
    N = 1024
    rows = [[1] * 8 + [64, 65, 63, 128, 129] + [N - 8 - 449],
            [int(v) for v in rng.integers(1, 40, 40)],
            [N]]
    rows[1].append(N - sum(rows[1]))
    W = wl.make_case(rows, D=40, L=700, x_dtype=dtype, seed=31)
    ref = reference(W)
    for limit in (0, 16, 64, 128):
        monkeypatch.setenv("RUBICONV_DIRECT_MAX", str(limit))
        y, plan = run_gpu(W, device)
        info = plan.info()
        assert info["direct_max"] == limit
        assert info["n_direct"] == sum(1 for r in rows for n in r if 0 < n <= limit)
        assert_parity(y, ref, W.cu_seqlens, dtype, f"limit {limit}")
        dyv, dx, dk, _ = tg._run(W, device, seed=limit + 5)
        assert_parity(dx, oracle.grad_x(W.filters, dyv, W.cu_seqlens), W.cu_seqlens, dtype,
                      f"dx limit {limit}")
        tg._check_dk(dk, oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L), dtype, f"limit {limit}")


@pytest.mark.parametrize("limit", [64, 300, 512])
def test_direct_path_on_matrix_cores(device, monkeypatch, limit):
    """The direct path on the matrix cores (RUBICONV_DIRECT_MFMA=1): documents up to the
    limit by blocked Toeplitz products, whole 16-token blocks and ragged ones, one token,
    documents longer than the filter (L = 500) and transformed documents beside them; the
    forward, both gradients and the fused backward meet the oracle bar, and the direct
    documents reach it with room to spare (their sums run in fp32 with the taps in two
    bf16 parts)."""
    import torch
    import paper_2605_08451_amd as rc
    import tests.test_gpu_grad as tg
    monkeypatch.setenv("RUBICONV_DIRECT_MFMA", "1")
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", str(limit))
    N = 4096
    rows = [[1, 15, 16, 17, 31, 33, 100, 255, 256, 257, 700, 1024], [64, 300, 500, 501, 1000], [N]]
    for r in rows[:2]:
        r.append(N - sum(r))
    W = wl.make_case(rows, D=64, L=500, x_dtype="bf16", seed=limit)
    ref = reference(W)
    y, plan = run_gpu(W, device)
    info = plan.info()
    assert info["direct_max"] == limit
    assert info["n_direct"] == sum(1 for r in rows for n in r if 0 < n <= limit)
    g, d = assert_parity(y, ref, W.cu_seqlens, "bf16", f"limit {limit}")
    # the direct documents alone: fp32 sums of exact bf16 products (taps split in two)
    worst = 0.0
    for b, r in enumerate(rows):
        s0 = 0
        for n in r:
            if 0 < n <= limit:
                worst = max(worst, rel_l2(y[b, s0:s0 + n], ref[b, s0:s0 + n]))
            s0 += n
    assert worst <= 3e-3, worst  # the bf16 rounding of y alone is about 1.6e-3
    dyv, dx, dk, _ = tg._run(W, device, seed=limit + 7)
    refx = oracle.grad_x(W.filters, dyv, W.cu_seqlens)
    refk = oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L)
    assert_parity(dx, refx, W.cu_seqlens, "bf16", f"dx limit {limit}")
    tg._check_dk(dk, refk, "bf16", f"dk limit {limit}")
    x, k = to_device(W, device)
    dy = torch.from_numpy(wl.f32_to_bf16_bits(dyv.astype(np.float32)).view(np.int16)).view(
        torch.bfloat16).to(device)
    p2 = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype="bf16")
    dxf, dkf = rc.packed_conv_backward(p2, x, dy, rc.filter_spectrum(p2, k))
    assert_parity(dxf.float().cpu().numpy().astype(np.float64), refx, W.cu_seqlens, "bf16", "fused dx")
    tg._check_dk(dkf.cpu().numpy().astype(np.float64), refk, "bf16", "fused dk")
    print(f"[direct mfma] limit {limit}: y {g:.2e} / {d:.2e}, direct documents {worst:.2e}",
          file=sys.stderr, flush=True)


@pytest.mark.parametrize("L,D", [(20, 96), (512, 32)])
def test_direct_path_filter_lengths(device, monkeypatch, L, D):
    """The direct path on the matrix cores with a filter far shorter than its documents
    (20 taps: every document longer than the filter reads zero taps past it) and with one
    as long as the longest direct document, over six and two 16-channel groups: the
    forward and both gradients, alone and in one call, meet the oracle bar on every
    document, direct or not."""
    import tests.test_gpu_grad as tg
    monkeypatch.setenv("RUBICONV_DIRECT_MFMA", "1")
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "512")
    N = 2048
    rows = [[1, 19, 20, 21, 48, 511, 512, 513], [200, 17, 1000]]
    for r in rows:
        r.append(N - sum(r))
    W = wl.make_case(rows, D=D, L=L, x_dtype="bf16", seed=L + D)
    ref = reference(W)
    y, plan = run_gpu(W, device)
    assert plan.info()["n_direct"] == sum(1 for r in rows for n in r if 0 < n <= 512)
    assert_parity(y, ref, W.cu_seqlens, "bf16", f"L {L} D {D}")
    dyv, dx, dk, _ = tg._run(W, device, seed=L + D + 1)
    assert_parity(dx, oracle.grad_x(W.filters, dyv, W.cu_seqlens), W.cu_seqlens, "bf16", f"dx L {L} D {D}")
    refk = oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L)
    tg._check_dk(dk, refk, "bf16", f"dk L {L} D {D}")
    # both gradients in one call
    import torch
    import paper_2605_08451_amd as rc
    x, k = to_device(W, device)
    dy = torch.from_numpy(wl.f32_to_bf16_bits(dyv.astype(np.float32)).view(np.int16)).view(
        torch.bfloat16).to(device)
    p2 = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype="bf16")
    dxf, dkf = rc.packed_conv_backward(p2, x, dy, rc.filter_spectrum(p2, k))
    assert_parity(dxf.float().cpu().numpy().astype(np.float64), oracle.grad_x(W.filters, dyv, W.cu_seqlens),
                  W.cu_seqlens, "bf16", f"fused dx L {L} D {D}")
    tg._check_dk(dkf.cpu().numpy().astype(np.float64), refk, "bf16", f"fused dk L {L} D {D}")


def test_plan_and_calls_on_a_side_stream(device):
    """A plan made on a side stream and used there at once (its tables' upload is
    enqueued on that stream, not waited for), with the spectrum, workspace and outputs
    allocated by the binding for that stream: the outputs equal those of the calling
    stream bit for bit, for the forward and both gradients."""
    import torch
    import paper_2605_08451_amd as rc
    W = wl.make_case([[700, 300, 24], [1024]], D=64, L=1024, x_dtype="bf16", seed=91)
    x, k = to_device(W, device)
    rng = np.random.default_rng(92)
    dy = torch.from_numpy(wl.f32_to_bf16_bits(rng.standard_normal(x.shape, dtype=np.float32))
                          .view(np.int16)).view(torch.bfloat16).to(device)

    def run(stream):
        plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype="bf16", y_dtype="bf16", stream=stream)
        spec = rc.filter_spectrum(plan, k, stream=stream)
        y = rc.packed_conv(plan, x, spec, stream=stream)
        dx = rc.packed_conv_dx(plan, dy, spec, stream=stream)
        dk = rc.packed_conv_dk(plan, x, dy, stream=stream)
        return plan, y, dx, dk

    torch.cuda.synchronize(device)
    ref = run(None)
    torch.cuda.synchronize(device)
    side = torch.cuda.Stream(device)
    got = run(side)
    side.synchronize()
    for name, a, b in zip(("y", "dx", "dk"), ref[1:], got[1:]):
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b), name
    yv = got[1].float().cpu().numpy().astype(np.float64)
    assert_parity(yv, reference(W), W.cu_seqlens, "bf16", "side stream")
