"""Value range of the bf16 path (needs an MI355X).

bf16 inputs run on complex fp16 grids.  These cases leave the N(0, 1) inputs of the
parity tests: a DC offset under an all-ones filter (the per-document prefix sum, whose
outputs reach 8e4), wide activations, and the small upstream gradients of training.
Each must meet the bf16 bar (2e-2 relative L2, globally and per document) against the
oracle on the mid-length workload's document boundaries.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as wl
from tests.common import ORACLE_THREADS, assert_parity, to_device

pytestmark = pytest.mark.gpu

D = 32


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _workload(x, filters):
    cu = wl.config_cu_seqlens(2)
    B, N = cu.shape[0], int(cu[0, -1])
    bits = wl.f32_to_bf16_bits(x).reshape(B, N, D)
    xv = wl.bf16_bits_to_f32(bits).reshape(B, N, D)
    return wl.Workload("range", B, N, D, filters.shape[1], "bf16", "bf16", cu, xv, bits,
                       np.ascontiguousarray(filters, np.float32), 0)


def _shape():
    cu = wl.config_cu_seqlens(2)
    return cu.shape[0], int(cu[0, -1])


def _forward(W, device):
    import torch
    import paper_2605_08451_amd as rc
    x, k = to_device(W, device)
    plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype="bf16", y_dtype="bf16")
    ws = plan.new_workspace(device)
    spec = rc.filter_spectrum(plan, k, workspace=ws)
    y = rc.packed_conv(plan, x, spec, workspace=ws)
    torch.cuda.synchronize()
    return y.float().cpu().numpy().astype(np.float64), plan, spec, ws


def _case_inputs(case, B, N):
    rng = np.random.default_rng(77)
    if case == "dc5_all_ones":
        x = 5.0 + rng.standard_normal((B, N, D), dtype=np.float32)
        k = np.ones((D, N), dtype=np.float32)
    elif case == "dc5_tiny_filter":      # the all-ones case with every tap 1e-6
        x = 5.0 + rng.standard_normal((B, N, D), dtype=np.float32)
        k = np.full((D, N), 1e-6, dtype=np.float32)
    elif case == "mixed_1e-4":          # documents alternately at 1 and 1e-4 (one scale per call)
        x = rng.standard_normal((B, N, D), dtype=np.float32)
        cu = wl.config_cu_seqlens(2)
        for b in range(B):
            for i in range(cu.shape[1] - 1):
                if i % 2:
                    x[b, cu[b, i]:cu[b, i + 1]] *= 1e-4
        k = wl.decaying_filters(rng, D, N)
    else:
        scale = {"wide_300": 300.0, "small_1e-4": 1e-4, "tiny_1e-6": 1e-6, "huge_1e4": 1e4}[case]
        x = scale * rng.standard_normal((B, N, D), dtype=np.float32)
        k = wl.decaying_filters(rng, D, N)
    return x, k


@pytest.mark.parametrize("case", ["dc5_all_ones", "dc5_tiny_filter", "wide_300", "small_1e-4",
                                  "tiny_1e-6", "huge_1e4", "mixed_1e-4"])
def test_forward_range(device, case):
    B, N = _shape()
    W = _workload(*_case_inputs(case, B, N))
    y, _, _, _ = _forward(W, device)
    ref = oracle.conv_fft(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS)
    assert np.isfinite(y).all(), case
    g, d = assert_parity(y, ref, W.cu_seqlens, "bf16", case)
    _say(f"[range] {case}: max |y| {np.abs(ref).max():.3g}, global {g:.2e}, worst document {d:.2e}")


@pytest.mark.parametrize("case", ["dc5_all_ones", "wide_300", "small_1e-4"])
def test_forward_range_without_prescale(device, monkeypatch, case):
    """RUBICONV_PRESCALE=0 (x taken as it is): the range the forward then keeps (a
    constant 5 plus unit noise under an all-ones filter, rms(x) from 1e-4 to 300) still
    meets the bar."""
    monkeypatch.setenv("RUBICONV_PRESCALE", "0")
    B, N = _shape()
    W = _workload(*_case_inputs(case, B, N))
    y, _, _, _ = _forward(W, device)
    ref = oracle.conv_fft(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS)
    assert np.isfinite(y).all(), case
    g, d = assert_parity(y, ref, W.cu_seqlens, "bf16", case)
    _say(f"[range, no prescale] {case}: global {g:.2e}, worst document {d:.2e}")


@pytest.mark.parametrize("scale", [1e-6, 1e3])
def test_gradient_range(device, scale):
    """Upstream gradients far from 1: dx and dk meet the bar."""
    import torch
    import paper_2605_08451_amd as rc
    from tests.test_gpu_grad import _check_dk
    B, N = _shape()
    rng = np.random.default_rng(78)
    x = rng.standard_normal((B, N, D), dtype=np.float32)
    k = wl.decaying_filters(rng, D, N)
    W = _workload(x, k)
    dyv = wl.round_to_bf16(scale * rng.standard_normal((B, N, D), dtype=np.float32)).astype(np.float64)
    dy = torch.from_numpy(wl.f32_to_bf16_bits(dyv.astype(np.float32)).view(np.int16)).view(
        torch.bfloat16).to(device)
    xd, kd = to_device(W, device)
    plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype="bf16", y_dtype="bf16")
    ws = plan.new_workspace(device)
    spec = rc.filter_spectrum(plan, kd, workspace=ws)
    dx = rc.packed_conv_dx(plan, dy, spec, workspace=ws).float().cpu().numpy().astype(np.float64)
    dk = rc.packed_conv_dk(plan, xd, dy).cpu().numpy().astype(np.float64)
    # the fused backward: dy's grid at dx's scale, dk's split applied in the row stage
    dxf, dkf = rc.packed_conv_backward(plan, xd, dy, spec)
    dxf, dkf = dxf.float().cpu().numpy().astype(np.float64), dkf.cpu().numpy().astype(np.float64)
    assert np.isfinite(dx).all() and np.isfinite(dk).all(), scale
    assert np.isfinite(dxf).all() and np.isfinite(dkf).all(), scale
    refx = oracle.grad_x(W.filters, dyv, W.cu_seqlens, threads=ORACLE_THREADS)
    refk = oracle.grad_k(W.x, dyv, W.cu_seqlens, W.L, threads=ORACLE_THREADS)
    g, d = assert_parity(dx, refx, W.cu_seqlens, "bf16", f"dx scale {scale}")
    gk, wk = _check_dk(dk, refk, "bf16", f"dk scale {scale}")
    _say(f"[range] dy scale {scale}: dx {g:.2e} / {d:.2e}, dk {gk:.2e} / {wk:.2e}")
    g, d = assert_parity(dxf, refx, W.cu_seqlens, "bf16", f"fused dx scale {scale}")
    gk, wk = _check_dk(dkf, refk, "bf16", f"fused dk scale {scale}")
    _say(f"[range] fused, dy scale {scale}: dx {g:.2e} / {d:.2e}, dk {gk:.2e} / {wk:.2e}")


@pytest.mark.parametrize("loud", ["direct", "transform"])
def test_forward_range_direct_documents(device, monkeypatch, loud):
    """Short documents on the direct path beside transformed ones, one group 1e3 times
    louder than the other.  The x scale of the transforms comes from the documents the
    column pass loads, so the direct path's values do not set it; both groups must meet
    the bar per document."""
    monkeypatch.setenv("RUBICONV_DIRECT_MAX", "64")
    rng = np.random.default_rng(79)
    N = 4096
    short = [int(v) for v in rng.integers(1, 65, 40)]
    rows = [short + [N - sum(short)], [1500, 30, 2566], [N]]
    W0 = wl.make_case(rows, D=D, L=N, x_dtype="bf16", seed=79)
    x = W0.x.astype(np.float32).copy()
    for b, r in enumerate(W0.cu_seqlens):
        for s0, s1 in zip(r[:-1], r[1:]):
            is_direct = 0 < s1 - s0 <= 64
            if is_direct == (loud == "direct"):
                x[b, s0:s1] *= 1e3
    bits = wl.f32_to_bf16_bits(x)
    W = wl.Workload("range-direct", W0.B, W0.N, D, W0.L, "bf16", "bf16", W0.cu_seqlens,
                    wl.bf16_bits_to_f32(bits).reshape(x.shape), bits, W0.filters, 0)
    y, plan, _, _ = _forward(W, device)
    assert plan.info()["n_direct"] > 0
    ref = oracle.conv_direct(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS)
    g, d = assert_parity(y, ref, W.cu_seqlens, "bf16", f"loud {loud}")
    _say(f"[range] loud {loud} documents: global {g:.2e}, worst document {d:.2e}")


def test_scale_guess_sequence(device):
    """The matrix-core column pass starts at the range scale its plan's last call on the same
    input buffer found and redoes the pass when the call's own scale differs.  A sequence of calls whose x scale
    changes (1, 100, 100, 1e-3, 1) must give, for each input, the same bits whether the
    guess was right or wrong, and the forward must meet the bar at every step; dx likewise
    for dy scales 1e-6, 1e-6, 1."""
    import torch
    import paper_2605_08451_amd as rc
    B, N = _shape()
    rng = np.random.default_rng(80)
    x = rng.standard_normal((B, N, D), dtype=np.float32)
    k = wl.decaying_filters(rng, D, N)
    W = _workload(x, k)
    xd, kd = to_device(W, device)
    plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype="bf16", y_dtype="bf16")
    ws = plan.new_workspace(device)
    spec = rc.filter_spectrum(plan, kd, workspace=ws)
    outs = {}
    xs = torch.empty_like(xd)   # one buffer: the guess is kept per input buffer
    for sc in (1.0, 100.0, 100.0, 1e-3, 1.0, 1e-3):
        xs.copy_((xd.float() * sc).to(torch.bfloat16))
        y = rc.packed_conv(plan, xs, spec, workspace=ws)
        torch.cuda.synchronize()
        bits = y.view(torch.int16).cpu().numpy().copy()
        if sc in outs:
            assert np.array_equal(outs[sc], bits), f"x scale {sc}: output depends on the guess"
        else:
            outs[sc] = bits
            yv = y.float().cpu().numpy().astype(np.float64)
            ref = oracle.conv_fft(xs.float().cpu().numpy().astype(np.float64), W.filters, W.cu_seqlens,
                                  threads=ORACLE_THREADS)
            assert_parity(yv, ref, W.cu_seqlens, "bf16", f"x scale {sc}")
    douts = {}
    dy = torch.empty_like(xd)
    for sc in (1e-6, 1e-6, 1.0, 1e-6):
        dyv = wl.round_to_bf16(sc * rng.standard_normal((B, N, D), dtype=np.float32)) if sc not in douts else douts[sc][0]
        dy.copy_(torch.from_numpy(wl.f32_to_bf16_bits(dyv.astype(np.float32)).view(np.int16)).view(torch.bfloat16))
        dx = rc.packed_conv_dx(plan, dy, spec, workspace=ws)
        torch.cuda.synchronize()
        bits = dx.view(torch.int16).cpu().numpy().copy()
        if sc in douts:
            assert np.array_equal(douts[sc][1], bits), f"dy scale {sc}: dx depends on the guess"
        else:
            douts[sc] = (dyv, bits)
            ref = oracle.grad_x(W.filters, dyv.astype(np.float64), W.cu_seqlens, threads=ORACLE_THREADS)
            assert_parity(dx.float().cpu().numpy().astype(np.float64), ref, W.cu_seqlens, "bf16", f"dx {sc}")
    # dk: both column passes guess (x's and dy's scales); a repeated call must match
    from tests.test_gpu_grad import _check_dk
    dkb = {}
    for sc in (1e-6, 1e-6, 1.0, 1e-6):
        dyv = douts[sc][0]
        dy.copy_(torch.from_numpy(wl.f32_to_bf16_bits(dyv.astype(np.float32)).view(np.int16)).view(torch.bfloat16))
        dk = rc.packed_conv_dk(plan, xd, dy)
        torch.cuda.synchronize()
        v = dk.cpu().numpy().copy()
        if sc in dkb:
            assert np.array_equal(dkb[sc], v), f"dy scale {sc}: dk depends on the guess"
        else:
            dkb[sc] = v
            _check_dk(v.astype(np.float64), oracle.grad_k(W.x, dyv.astype(np.float64), W.cu_seqlens, W.L,
                                                          threads=ORACLE_THREADS), "bf16", f"dk {sc}")
    _say("[range] scale guesses: outputs independent of the guess")
