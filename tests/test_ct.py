"""The masked Cooley-Tukey variant (Algorithm 2): plan tables on the host, then the
HIP path against the oracle on the same seeded inputs (GPU tests).

The variant computes the same convolution as the four-step path, so its outputs are
held to the same bars against the same direct oracle: relative L2 <= 1e-4 (fp32) and
<= 2e-2 (bf16 inputs), over the whole output and over every document, and zero
cross-document leakage.  Its document table must give exactly the oracle's segments
and the power-of-two sizes of ``oracle.masked_fft.ct_padded_size``.
"""
import sys

import numpy as np
import pytest

import oracle
import paper_2605_08451_amd as rc
import workloads as wl
from oracle.masked_fft import ct_padded_size
from tests.common import ORACLE_THREADS, TOL, assert_parity, reference


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


# ------------------------------------------------------------------ host: plan tables
@pytest.mark.parametrize("i", [0, 1, 2, 3, 4])
def test_doc_table_matches_oracle(i):
    cu = wl.config_cu_seqlens(i)
    D, L, dt = wl.CONFIG_SHAPES[i]
    N = int(cu[0, -1])
    plan = rc.CTPlan(cu, N=N, D=D, L=L, x_dtype=dt)
    t = plan.doc_table()
    ref = oracle.doc_table(cu, N, L, 256)
    np.testing.assert_array_equal(t[:, :4], ref[:, :4])      # row, index, start, length
    P = t[:, 4].astype(np.int64)
    np.testing.assert_array_equal(P, [ct_padded_size(int(n), L) for n in t[:, 3]])
    off = t[:, 5].astype(np.int64)
    assert np.all(off % P == 0)                              # every document aligned to its size
    order = np.argsort(off)
    assert np.all(off[order][1:] == (off + P)[order][:-1])   # packed back to back from 0
    assert off[order][0] == 0
    assert np.all(np.diff(P[order]) <= 0)                    # longest first
    plan.close()


def test_plan_errors():
    cu = np.array([[0, 3, 8]], dtype=np.int32)
    with pytest.raises(rc.RubiconvError) as e:
        rc.CTPlan(cu, N=8, D=3, L=4, x_dtype="f32")          # channels go in pairs
    assert e.value.status == 3
    with pytest.raises(rc.RubiconvError) as e:
        rc.CTPlan(np.array([[0, 5, 4]], dtype=np.int32), N=4, D=2, L=4, x_dtype="f32")
    assert e.value.status == 2
    with pytest.raises(rc.RubiconvError) as e:
        rc.CTPlan(np.array([[0, 262145]], dtype=np.int32), N=262145, D=2, L=262145, x_dtype="f32")
    assert e.value.status == 3                               # needs 2^20 points
    p = rc.CTPlan(np.array([[0, 262144]], dtype=np.int32), N=262144, D=2, L=262144, x_dtype="f32")
    assert p.doc_table()[0, 4] == 524288
    p = rc.CTPlan(np.array([[0, 16385]], dtype=np.int32), N=16385, D=2, L=16385, x_dtype="f32")
    assert p.doc_table()[0, 4] == 65536
    p = rc.CTPlan(np.array([[0, 20000]], dtype=np.int32), N=20000, D=2, L=12000, x_dtype="f32")
    assert p.doc_table()[0, 4] == 32768                      # 20000 + 12000 - 1 <= 2^15
    p = rc.CTPlan(wl.config_cu_seqlens(4), N=262144, D=256, L=262144, x_dtype="bf16")
    assert p.doc_table()[:, 4].max() == 524288


# ------------------------------------------------------------------ GPU parity
def run_ct(W, device, y_dtype=None, repeats=1):
    import torch
    from tests.common import to_device
    x, k = to_device(W, device)
    yd = W.y_dtype if y_dtype is None else y_dtype
    plan = rc.CTPlan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=yd)
    ws = plan.new_workspace(device)
    spec = rc.ct_filter_spectrum(plan, k, workspace=ws)
    outs = []
    for _ in range(repeats):
        y = rc.ct_packed_conv(plan, x, spec, workspace=ws)
        torch.cuda.synchronize(device)
        outs.append(y.float().cpu().numpy().astype(np.float64))
    plan.close()
    return outs if repeats > 1 else outs[0]


@pytest.mark.gpu
@pytest.mark.parametrize("i", [0, 1, 3])
def test_ct_config_parity(device, i):
    _say(f"[ct] config {i} ({wl.CONFIG_NAMES[i]})")
    W = wl.make_config(i)
    y = run_ct(W, device)
    g, d = assert_parity(y, reference(W), W.cu_seqlens, W.x_dtype, f"ct config {i}")
    _say(f"[ct] config {i}: global {g:.2e}, worst document {d:.2e}")


@pytest.mark.gpu
def test_ct_full_size_sampled(device):
    """The mid-length bf16 workload at full size, sampled entries against the defining sum."""
    W = wl.make_config(2)
    _say("[ct] config 2 sampled")
    y = run_ct(W, device)
    rng = np.random.default_rng(102)
    n = 4000
    btd = np.stack([rng.integers(0, W.B, n), rng.integers(0, W.N, n), rng.integers(0, W.D, n)], 1)
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


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ct_long_documents(device, dtype):
    """Documents of 2^16 to 2^19 transform points (the middle pass between the tile
    and the column pass), with filters as long as the row and short ones."""
    N = 262144
    rows = [[N], [70000, 30000, 16385, N - 116385]]
    for L in (N, 5000):
        W = wl.make_case(rows, D=4 if dtype == "f32" else 32, L=L, x_dtype=dtype, seed=L)
        P = sorted(set(int(v) for v in rc.CTPlan(W.cu_seqlens, N=N, D=W.D, L=L,
                                                  x_dtype=dtype).doc_table()[:, 4]))
        _say(f"[ct] long documents {dtype} L={L}: sizes {P}")
        assert max(P) >= 65536
        y = run_ct(W, device)
        assert_parity(y, reference(W, "fft"), W.cu_seqlens, dtype, f"long {dtype} L={L}")


@pytest.mark.gpu
def test_ct_long_context_sampled(device):
    """The long-context workload (documents up to 2^19 transform points) at full size,
    sampled entries against the defining sum."""
    W = wl.make_config(4)
    _say("[ct] config 4 sampled")
    y = run_ct(W, device)
    rng = np.random.default_rng(104)
    n = 3000
    btd = np.stack([np.zeros(n, dtype=np.int64), rng.integers(0, W.N, n), rng.integers(0, W.D, n)], 1)
    extra = [(0, s, rng.integers(W.D)) for s0, s1 in zip(W.cu_seqlens[0][:-1], W.cu_seqlens[0][1:])
             if s1 > s0 for s in (s0, s1 - 1)]
    btd = np.concatenate([btd, np.array(extra, dtype=np.int64)])
    ref = oracle.conv_at(W.x, W.filters, W.cu_seqlens, btd, threads=ORACLE_THREADS)
    got = y[btd[:, 0], btd[:, 1], btd[:, 2]]
    err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    _say(f"[ct] config 4 sampled error {err:.2e}")
    assert err <= TOL[W.x_dtype], err


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ct_ragged_edges(device, dtype):
    """Lengths around the tile size (P = 512 / 1024 boundaries), length 1, whole rows,
    the largest document (P = 2^15), and L shorter and longer than the documents."""
    rng = np.random.default_rng(17)
    N = 16384
    edge = [255, 256, 257, 511, 512, 513, 1024, 1025]
    rows = [[N],
            [1] * 5 + edge + [N - 5 - sum(edge)],
            wl.random_rows(rng, 1, N, 3000, p_short=0.5)[0],
            [N - 1, 1]]
    for L in (1, 7, 300, N):
        W = wl.make_case(rows, D=6, L=L, x_dtype=dtype, seed=L)
        y = run_ct(W, device)
        assert_parity(y, reference(W), W.cu_seqlens, dtype, f"L={L}")


@pytest.mark.gpu
@pytest.mark.parametrize("D", [2, 30, 32, 34, 64])
def test_ct_channel_counts(device, D):
    """Channel counts below, at and above one block of 16 pairs."""
    rng = np.random.default_rng(D)
    rows = wl.random_rows(rng, 2, 3000, 1500)
    for dtype in ("f32", "bf16"):
        W = wl.make_case(rows, D=D, L=2000, x_dtype=dtype, seed=D)
        y = run_ct(W, device)
        assert_parity(y, reference(W), W.cu_seqlens, dtype, f"D={D} {dtype}")


@pytest.mark.gpu
@pytest.mark.parametrize("N", [1, 2, 5, 100])
def test_ct_short_rows(device, N):
    rng = np.random.default_rng(N)
    rows = wl.random_rows(rng, 3, N, max(1, N // 3))
    W = wl.make_case(rows, D=4, L=N + 3, seed=N)
    y = run_ct(W, device)
    assert_parity(y, reference(W), W.cu_seqlens, "f32", f"N={N}")


@pytest.mark.gpu
def test_ct_mixed_dtypes(device):
    rng = np.random.default_rng(3)
    rows = wl.random_rows(rng, 2, 3000, 1500)
    W = wl.make_case(rows, D=8, L=3000, x_dtype="bf16", seed=3)
    assert_parity(run_ct(W, device, y_dtype="f32"), reference(W), W.cu_seqlens, "bf16", "bf16 -> f32")
    W = wl.make_case(rows, D=8, L=3000, x_dtype="f32", seed=4)
    assert_parity(run_ct(W, device, y_dtype="bf16"), reference(W), W.cu_seqlens, "bf16", "f32 -> bf16")


@pytest.mark.gpu
def test_ct_leakage_impulses(device):
    """An impulse in document j, with an undecayed filter as long as the row, leaves every
    other document and row below 1e-6 of the impulse document's peak."""
    N, D = 4096, 4
    rng = np.random.default_rng(11)
    rows = [[1, 255, 256, 257, 1000, N - 1769], [N]]
    cu = wl.cu_from_rows(rows, N)
    k = rng.standard_normal((D, N)).astype(np.float32)
    docs = [(b, int(s0), int(s1)) for b, r in enumerate(cu) for s0, s1 in zip(r[:-1], r[1:])
            if s1 > s0]
    for (b, s0, s1) in docs:
        W = wl.make_case(rows, D=D, L=N, seed=0, filters=k)
        W.x[:] = 0.0
        t = s0 + int(rng.integers(0, s1 - s0))
        W.x[b, t, :] = rng.standard_normal(D)
        y = run_ct(W, device)
        inside = np.zeros(y.shape, dtype=bool)
        inside[b, s0:s1] = True
        peak = np.abs(y[inside]).max()
        assert peak > 0
        assert np.abs(y[~inside]).max() <= 1e-6 * peak, (b, s0, s1)
        assert np.abs(y[b, s0:t]).max(initial=0.0) <= 1e-6 * peak, (b, s0, s1)


@pytest.mark.gpu
def test_ct_deterministic_and_matches_four_step(device):
    """Repeated calls give identical bits; the two methods agree within the bar."""
    from tests.common import run_gpu
    W = wl.make_config(1)
    a, b = run_ct(W, device, repeats=2)
    assert np.array_equal(a, b)
    y4, _ = run_gpu(W, device)
    assert_parity(a, y4, W.cu_seqlens, "bf16", "ct vs four-step")
