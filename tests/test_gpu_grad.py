"""Gradients on the GPU (rubiconv_packed_conv_dx / _dk through the C ABI) against the
oracle's gradients on the same seeded inputs (needs an MI355X).

Bars as for the forward: relative L2 <= 1e-4 for fp32 workloads and <= 2e-2 for bf16
inputs with fp32 accumulation; dx also per document, dk also per channel.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as wl
from tests.common import ORACLE_THREADS, TOL, assert_parity, rel_l2, to_device

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _dy(W, seed):
    """Upstream gradient of y's dtype: values (float64) and the device tensor."""
    import torch
    vals, bits = wl.draw_x(np.random.default_rng(seed), W.B, W.N, W.D, W.y_dtype)
    if W.y_dtype == "bf16":
        t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(vals, dtype=np.float32))
    return vals.astype(np.float64), t


def _run(W, device, seed, n1=0, want_dk=True):
    import torch
    import paper_2605_08451_amd as rc
    x, k = to_device(W, device)
    dyv, dy = _dy(W, seed)
    dy = dy.to(device)
    plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=W.y_dtype, n1=n1)
    ws = plan.new_workspace(device)
    spec = rc.filter_spectrum(plan, k, workspace=ws)
    dx = rc.packed_conv_dx(plan, dy, spec, workspace=ws)
    dk = rc.packed_conv_dk(plan, x, dy) if want_dk else None
    torch.cuda.synchronize(device)
    dxv = dx.float().cpu().numpy().astype(np.float64)
    dkv = dk.cpu().numpy().astype(np.float64) if want_dk else None
    return dyv, dxv, dkv, plan


def _check_dk(dk, ref, dtype, label):
    """Relative L2 over all of dk, and per channel once a channel has 64 lags or more.
    With fewer lags the per-channel figure is the error of a few entries of a
    correlation computed through fp16 transforms, whose rounding scales with the
    whole correlation (every lag of every document), not with the lags kept."""
    tol = TOL[dtype]
    g = rel_l2(dk, ref)
    worst = 0.0
    if ref.shape[1] >= 64:
        worst = max(rel_l2(dk[d], ref[d]) for d in range(ref.shape[0]) if np.any(ref[d]))
    assert g <= tol and worst <= tol, f"{label}: dk global {g:.2e}, worst channel {worst:.2e}"
    return g, worst


@pytest.mark.parametrize("i", [0, 1, 3])
def test_gradients_config(device, i):
    _say(f"[grad] config {i} ({wl.CONFIG_NAMES[i]})")
    W = wl.make_config(i)
    dyv, dx, dk, _ = _run(W, device, seed=100 + i)
    g, d = assert_parity(dx, oracle.grad_x(W.filters, dyv, W.cu_seqlens, threads=ORACLE_THREADS),
                         W.cu_seqlens, W.x_dtype, f"dx config {i}")
    gk, wk = _check_dk(dk, oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L, threads=ORACLE_THREADS),
                       W.x_dtype, f"config {i}")
    _say(f"[grad] config {i}: dx {g:.2e} / {d:.2e}, dk {gk:.2e} / {wk:.2e}")


@pytest.mark.parametrize("i", [2, 4])
def test_gradients_full_size_sampled(device, i):
    """The bench workloads at full size: sampled dx and dk entries against the defining
    sums (first and last token of every document included)."""
    W = wl.make_config(i)
    dyv, dx, dk, _ = _run(W, device, seed=100 + i)
    rng = np.random.default_rng(200 + i)
    n = 3000
    bsd = np.stack([rng.integers(0, W.B, n), rng.integers(0, W.N, n), rng.integers(0, W.D, n)], 1)
    extra = [(b, s, rng.integers(W.D)) for b, row in enumerate(W.cu_seqlens)
             for s0, s1 in zip(row[:-1], row[1:]) if s1 > s0 for s in (s0, s1 - 1)]
    bsd = np.concatenate([bsd, np.array(extra, dtype=np.int64)])
    ref = oracle.grad_x_at(W.filters, dyv, W.cu_seqlens, bsd, threads=ORACLE_THREADS)
    got = dx[bsd[:, 0], bsd[:, 1], bsd[:, 2]]
    assert rel_l2(got, ref) <= TOL[W.x_dtype], rel_l2(got, ref)
    m = 400
    dt = np.stack([rng.integers(0, W.D, m), rng.integers(0, W.L, m)], 1)
    dt[: m // 4, 1] = rng.integers(0, 64, m // 4)   # the short lags every document has
    refk = oracle.grad_k_at(W.x, dyv, W.cu_seqlens, W.L, dt, threads=ORACLE_THREADS)
    gotk = dk[dt[:, 0], dt[:, 1]]
    assert rel_l2(gotk, refk) <= TOL[W.x_dtype], rel_l2(gotk, refk)


@pytest.mark.parametrize("n1", [256, 64])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gradient_edges(device, n1, dtype):
    """Documents of length 1, N1 - 1, N1, N1 + 1, whole rows; L shorter and longer than
    them; an odd channel count."""
    rng = np.random.default_rng(17)
    N = 2048
    rows = [[N],
            [1] * 5 + [n1 - 1, n1, n1 + 1] + [N - 5 - 3 * n1],
            wl.random_rows(rng, 1, N, 300, p_short=0.5)[0],
            [N - 1, 1]]
    for L in (1, 7, 300, N, 3 * N):
        W = wl.make_case(rows, D=5, L=L, x_dtype=dtype, seed=L)
        dyv, dx, dk, _ = _run(W, device, seed=L + 1, n1=n1)
        assert_parity(dx, oracle.grad_x(W.filters, dyv, W.cu_seqlens), W.cu_seqlens, dtype,
                      f"dx n1={n1} L={L}")
        _check_dk(dk, oracle.grad_k(W.x, dyv, W.cu_seqlens, L), dtype, f"n1={n1} L={L}")


@pytest.mark.parametrize("D", [32, 96])
def test_gradients_matrix_core_rows(device, D):
    """bf16 inputs with whole 32-channel blocks (matrix-core column passes) and row sizes
    across the short-row and partner-row kernels."""
    rows = [[20480, 12288], [17280, 12800, 2304, 384], [9216, 8192, 6400, 4096, 2048, 1920, 896]]
    W = wl.make_case(rows, D=D, L=32768, x_dtype="bf16", seed=D)
    dyv, dx, dk, plan = _run(W, device, seed=D + 1)
    ms = sorted(set(int(m) for m in plan.doc_table()[:, 4]))
    assert min(ms) <= 16 and max(ms) > 100, ms
    assert_parity(dx, oracle.grad_x(W.filters, dyv, W.cu_seqlens, threads=ORACLE_THREADS),
                  W.cu_seqlens, "bf16", f"dx D={D}")
    _check_dk(dk, oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L, threads=ORACLE_THREADS), "bf16",
              f"D={D}")


def test_gradients_unlisted_row_sizes(device, monkeypatch):
    """Row sizes outside the 2^a 3^b 5^c list (primes and others), which the matrix-core
    row kernels take as they are (RUBICONV_EXACT_ROWS = 1), for the forward, dx and dk:
    every size its own class, a 7-tap filter so that a document of 256 (k - 1) + 3
    tokens takes m = k."""
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "0")   # every document on the transform path
    import paper_2605_08451_amd as rc
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "0")
    monkeypatch.setenv("RUBICONV_EXACT_ROWS", "1")
    ks = (7, 11, 13, 23, 31, 37, 53, 67, 89, 101, 127)
    lens = [256 * (k - 1) + 3 for k in ks]
    N = max(lens) + 1
    rows = [[ln, N - ln] for ln in lens]
    W = wl.make_case(rows, D=32, L=7, x_dtype="bf16", seed=17)
    dyv, dx, dk, plan = _run(W, device, seed=18)
    ms = sorted(set(int(m) for m in plan.doc_table()[:, 4]))
    assert all(k in ms for k in ks), (ks, ms)
    x, k = to_device(W, device)
    y = rc.conv(x, k, W.cu_seqlens).float().cpu().numpy().astype(np.float64)
    assert_parity(y, oracle.conv_direct(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS),
                  W.cu_seqlens, "bf16", "forward")
    assert_parity(dx, oracle.grad_x(W.filters, dyv, W.cu_seqlens, threads=ORACLE_THREADS),
                  W.cu_seqlens, "bf16", "dx")
    _check_dk(dk, oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L, threads=ORACLE_THREADS), "bf16", "dk")


def test_dx_leakage(device):
    """An impulse of dy in one document leaves dx of every other document below 1e-6 of
    its peak; impulses at the first and last token of a row."""
    import torch
    import paper_2605_08451_amd as rc
    N, D, L = 4096, 4, 4096
    rows = [[1000, 1, 2000, 1095], [4096]]
    W = wl.make_case(rows, D=D, L=L, x_dtype="f32", seed=3)
    x, k = to_device(W, device)
    plan = rc.Plan(W.cu_seqlens, N=N, D=D, L=L, x_dtype="f32")
    spec = rc.filter_spectrum(plan, k)
    for b, s0, s1 in [(0, 1000, 1001), (0, 1001, 3001), (0, 3001, 4096), (0, 0, 1000)]:
        for t in (s0, s1 - 1):
            dy = torch.zeros((2, N, D), dtype=torch.float32, device=device)
            dy[b, t] = 1.0
            dx = rc.packed_conv_dx(plan, dy, spec).cpu().numpy()
            peak = np.abs(dx[b, s0:s1]).max()
            outside = np.abs(np.concatenate([dx[b, :s0].ravel(), dx[b, s1:].ravel(), dx[1].ravel()]))
            assert peak > 0 and outside.max() <= 1e-6 * peak, (b, s0, s1, t)


def test_gradients_deterministic(device):
    W = wl.make_case(wl.random_rows(np.random.default_rng(4), 2, 5000, 3000), D=40, L=5000,
                     x_dtype="bf16", seed=4)
    a = _run(W, device, seed=9)
    b = _run(W, device, seed=9)
    np.testing.assert_array_equal(a[1], b[1])
    np.testing.assert_array_equal(a[2], b[2])


def test_class_groups(device, monkeypatch):
    """Size classes holding one to ten documents: the matrix-core row kernels take a
    class's documents in groups of at most four sharing one filter-row transform (ten
    documents: groups of 4, 3 and 3), for short rows, 17-32-point rows and the partner
    kernel; the forward, dx and dk (whose tasks keep one document each) meet the bar."""
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "0")   # every document on the transform path
    import paper_2605_08451_amd as rc
    import torch
    N = 8192
    rows = [[500] * 10 + [N - 5000], [1500] * 5 + [N - 7500], [3000, 3000, N - 6000], [6000, N - 6000]]
    W = wl.make_case(rows, D=32, L=N, x_dtype="bf16", seed=77)
    x, k = to_device(W, device)
    dyv, dy = _dy(W, 78)
    dy = dy.to(device)
    plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype="bf16")
    ms = [int(v) for v in plan.doc_table()[:, 4]]
    assert max(ms.count(m) for m in set(ms)) >= 9 and max(ms) > 32, ms
    ws = plan.new_workspace(device)
    spec = rc.filter_spectrum(plan, k, workspace=ws)
    y = rc.packed_conv(plan, x, spec, workspace=ws)
    dx = rc.packed_conv_dx(plan, dy, spec, workspace=ws)
    dk = rc.packed_conv_dk(plan, x, dy)
    torch.cuda.synchronize(device)
    f64 = lambda t: t.float().cpu().numpy().astype(np.float64)
    assert_parity(f64(y), oracle.conv_direct(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS),
                  W.cu_seqlens, "bf16", "y")
    assert_parity(f64(dx), oracle.grad_x(W.filters, dyv, W.cu_seqlens, threads=ORACLE_THREADS),
                  W.cu_seqlens, "bf16", "dx")
    _check_dk(f64(dk), oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L, threads=ORACLE_THREADS), "bf16", "dk")


@pytest.mark.parametrize("D", [32, 64])
def test_filter_gradient_sum_groups(device, D, monkeypatch):
    """The filter gradient adds the correlation products of a size class's documents
    (up to eight, longest first) before one inverse transform: classes whose documents
    differ in length, with the longest neither first nor last in its row, classes of
    more than eight documents (several groups), a class of one document, short rows
    (8-16 points) and partner-kernel rows (33-128 points); every lag of dk against the
    oracle, per channel."""
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "0")   # every document on the transform path
    N = 12000
    rows = [[930, 1000, 960, 880, 990, 940, 905, 870, 1000, 975, N - 9450],
            [3000, 3100, 2950, 2900, N - 11950],
            [430, 500, 470, 450, 500, 420, 480, 460, 440, 490, N - 4640],
            [6000, N - 6000]]
    W = wl.make_case(rows, D=D, L=N, x_dtype="bf16", seed=D + 3)
    dyv, dx, dk, plan = _run(W, device, seed=D + 4)
    t = plan.doc_table()
    ms = [int(v) for v in t[:, 4]]
    assert max(ms.count(m) for m in set(ms)) > 8 and max(ms) > 32, ms
    g, worst = _check_dk(dk, oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L, threads=ORACLE_THREADS), "bf16",
                         f"D={D}")
    _say(f"[dk sum groups] D={D}: global {g:.2e}, worst channel {worst:.2e}")
    assert_parity(dx, oracle.grad_x(W.filters, dyv, W.cu_seqlens, threads=ORACLE_THREADS),
                  W.cu_seqlens, "bf16", f"dx D={D}")


@pytest.mark.parametrize("rows", [[[200] * 10 + [48]], [[200, 200, 1648]], [[200, 1848]],
                                  [[600] * 3 + [248]], [[100] * 20 + [48]]])
def test_batched_short_rows(device, rows, monkeypatch):
    """Rows of at most 8 points go 16 / m documents to a matrix-core block: full and
    partial blocks, a class of one document, rows of one point, and row 0 (one
    document per block); forward, dx and dk.  Slots past a block's documents must
    not read stale exchange values (a non-finite one would spread over its pair)."""
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "0")   # every document on the transform path
    import paper_2605_08451_amd as rc
    monkeypatch.setenv("RUBICONV_ROW_BATCH", "8")   # whatever share these rows hold
    W = wl.make_case(rows, D=32, L=2048, x_dtype="bf16", seed=sum(rows[0]))
    dyv, dx, dk, plan = _run(W, device, seed=5)
    assert min(int(v) for v in plan.doc_table()[:, 4]) <= 2
    x, k = to_device(W, device)
    p2 = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype="bf16")
    y = rc.packed_conv(p2, x, rc.filter_spectrum(p2, k)).float().cpu().numpy().astype(np.float64)
    assert np.isfinite(y).all() and np.isfinite(dx).all() and np.isfinite(dk).all()
    assert_parity(y, oracle.conv_direct(W.x, W.filters, W.cu_seqlens), W.cu_seqlens, "bf16", "y")
    assert_parity(dx, oracle.grad_x(W.filters, dyv, W.cu_seqlens), W.cu_seqlens, "bf16", "dx")
    _check_dk(dk, oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L), "bf16", "dk")


def test_long_rows(device, monkeypatch):
    """Rows longer than 256 points on fp16 grids go through a second four-step level
    (m = m1 m2 sub-rows of at most 64 points, run by the matrix-core row kernels with
    N1 m1 rows): first-level sizes 5, 15, 16 and sub-rows of 25 to 64 points, the
    forward against the full FFT oracle, dx and dk sampled against their sums.  (Sizes
    here: 270 = 5 x 54, 360 = 6 x 60, 375 = 15 x 25, 400 = 8 x 50, 675 = 15 x 45,
    1000 = 20 x 50, 1024 = 16 x 64.)"""
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "0")   # every document at its own size
    N = 130000
    rows = [[N], [47000, N - 47000], [51000, 33920, N - 84920], [2000, N - 2000]]
    W = wl.make_case(rows, D=32, L=N, x_dtype="bf16", seed=9)
    dyv, dx, dk, plan = _run(W, device, seed=10)
    ms = sorted(set(int(m) for m in plan.doc_table()[:, 4]))
    assert sum(m > 256 for m in ms) >= 4 and 375 in ms and 1024 in ms, ms
    import paper_2605_08451_amd as rc
    x, k = to_device(W, device)
    y = rc.packed_conv(plan, x, rc.filter_spectrum(plan, k)).float().cpu().numpy().astype(np.float64)
    g, d = assert_parity(y, oracle.conv_fft(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS),
                         W.cu_seqlens, "bf16", "y")
    print(f"[long rows] forward: global {g:.2e}, worst document {d:.2e}", file=sys.stderr, flush=True)
    # one more fp16 rounding of the grid than ordinary rows: a wrong root or partner in
    # one sub-row would show as a few percent on some positions, above this bar
    assert d <= 5e-3, d
    rng = np.random.default_rng(11)
    n = 3000
    bsd = np.stack([rng.integers(0, W.B, n), rng.integers(0, W.N, n), rng.integers(0, W.D, n)], 1)
    ref = oracle.grad_x_at(W.filters, dyv, W.cu_seqlens, bsd, threads=ORACLE_THREADS)
    assert rel_l2(dx[bsd[:, 0], bsd[:, 1], bsd[:, 2]], ref) <= TOL["bf16"]
    dt = np.stack([rng.integers(0, W.D, 300), rng.integers(0, W.L, 300)], 1)
    refk = oracle.grad_k_at(W.x, dyv, W.cu_seqlens, W.L, dt, threads=ORACLE_THREADS)
    assert rel_l2(dk[dt[:, 0], dt[:, 1]], refk) <= TOL["bf16"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_generic_long_rows(device, monkeypatch, dtype):
    """Rows longer than 256 points in the generic (Stockham in LDS) row kernel: every
    such row on fp32 grids, and on fp16 grids with the second four-step level off.
    Forward against the full FFT oracle, dx sampled against its defining sums."""
    monkeypatch.setenv("RUBICONV_CLASS_MERGE", "0")
    if dtype == "bf16":
        monkeypatch.setenv("RUBICONV_LONG_ROWS", "0")
    N = 130000
    rows = [[N], [51000, 33920, N - 84920]]
    W = wl.make_case(rows, D=32, L=N, x_dtype=dtype, seed=19)
    dyv, dx, _, plan = _run(W, device, seed=20, want_dk=False)
    ms = sorted(set(int(m) for m in plan.doc_table()[:, 4]))
    assert sum(m > 256 for m in ms) >= 2, ms
    import paper_2605_08451_amd as rc
    x, k = to_device(W, device)
    y = rc.packed_conv(plan, x, rc.filter_spectrum(plan, k)).float().cpu().numpy().astype(np.float64)
    g, d = assert_parity(y, oracle.conv_fft(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS),
                         W.cu_seqlens, dtype, "y")
    _say(f"[generic long rows] {dtype}: global {g:.2e}, worst document {d:.2e}, sizes {ms}")
    rng = np.random.default_rng(21)
    n = 2000
    bsd = np.stack([rng.integers(0, W.B, n), rng.integers(0, W.N, n), rng.integers(0, W.D, n)], 1)
    ref = oracle.grad_x_at(W.filters, dyv, W.cu_seqlens, bsd, threads=ORACLE_THREADS)
    assert rel_l2(dx[bsd[:, 0], bsd[:, 1], bsd[:, 2]], ref) <= TOL[dtype]


def _fused_and_separate(W, device, seed):
    """dx and dk from rubiconv_packed_conv_backward and from the two separate calls on one
    plan and the same inputs (float64 arrays), and the plan."""
    import torch
    import paper_2605_08451_amd as rc
    x, k = to_device(W, device)
    dyv, dy = _dy(W, seed)
    dy = dy.to(device)
    plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=W.y_dtype)
    ws = plan.new_dk_workspace(device)
    spec = rc.filter_spectrum(plan, k, workspace=ws)
    dx_s = rc.packed_conv_dx(plan, dy, spec, workspace=ws)
    dk_s = rc.packed_conv_dk(plan, x, dy, workspace=ws)
    dx_f, dk_f = rc.packed_conv_backward(plan, x, dy, spec, workspace=ws)
    torch.cuda.synchronize(device)
    same_dx = bool(torch.equal(dx_s, dx_f))
    out = [t.float().cpu().numpy().astype(np.float64) for t in (dx_s, dk_s, dx_f, dk_f)]
    return dyv, same_dx, out, plan


FUSED_CASES = {
    # every document on the matrix-core row kernels: the fused path
    "mid-length": dict(config=2),
    "sum-groups": dict(rows=[[930, 1000, 960, 880, 990, 940, 905, 870, 1000, 975, 12000 - 9450],
                             [3000, 3100, 2950, 2900, 12000 - 11950], [6000, 6000]], N=12000, D=32),
    "direct": dict(rows=[[40] * 30 + [2800], [17, 63, 5, 1, 64] * 8 + [4000 - 1200]], N=4000, D=32,
                   direct=64),
    # the two calls in sequence: fp32 grids, and rows of 129-256 points on the VALU kernels
    "fp32": dict(config=0),
    "valu-rows": dict(rows=[[20000, 4000]], N=24000, D=32),
}


@pytest.mark.parametrize("case", list(FUSED_CASES))
def test_fused_backward(device, monkeypatch, case):
    """rubiconv_packed_conv_backward against the separate dx and dk calls: dx bit for bit,
    dk within the bar of the oracle (every lag where the oracle is cheap, sampled at full
    size) and close to the separate call's; on the fallback both bit for bit."""
    spec = FUSED_CASES[case]
    if "direct" in spec:
        monkeypatch.setenv("RUBICONV_DIRECT_MAX", str(spec["direct"]))
    if "config" in spec:
        W = wl.make_config(spec["config"])
    else:
        W = wl.make_case(spec["rows"], D=spec["D"], L=spec["N"], x_dtype="bf16", seed=len(case))
    _say(f"[fused backward] {case}")
    dyv, same_dx, (dx_s, dk_s, dx_f, dk_f), plan = _fused_and_separate(W, device, seed=3 + len(case))
    assert same_dx, f"{case}: dx differs from rubiconv_packed_conv_dx"
    fused = W.x_dtype == "bf16" and max(int(m) for m in plan.doc_table()[:, 4]) <= 128
    if not fused:
        assert np.array_equal(dk_f, dk_s), f"{case}: the fallback's dk differs"
        return
    if "direct" in spec:
        assert plan.info()["n_direct"] > 0
    close = rel_l2(dk_f, dk_s)
    if W.B * W.N * W.D <= 2_000_000:
        g, worst = _check_dk(dk_f, oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L, threads=ORACLE_THREADS),
                             "bf16", case)
    else:
        rng = np.random.default_rng(31)
        dt = np.stack([rng.integers(0, W.D, 400), rng.integers(0, W.L, 400)], 1)
        refk = oracle.grad_k_at(W.x, dyv, W.cu_seqlens, W.L, dt, threads=ORACLE_THREADS)
        g = worst = rel_l2(dk_f[dt[:, 0], dt[:, 1]], refk)
        assert g <= TOL["bf16"], f"{case}: sampled dk {g:.2e}"
    _say(f"[fused backward] {case}: dk {g:.2e} / {worst:.2e}, against the separate call {close:.2e}")
    assert close <= 5e-3, close
