"""Helpers shared by the tests: run the HIP path on a workload, compare with the oracle.

Nothing here computes the convolution: the GPU side calls the library through the
binding, the reference side calls ``oracle``.
"""
import os

import numpy as np

import oracle
import workloads as wl

#: oracle threads: one GPU's share of a host's cores (16)
ORACLE_THREADS = min(16, os.cpu_count() or 1)

#: parity bars: relative L2 error, globally and per document
TOL = {"f32": 1e-4, "bf16": 2e-2}


def to_device(W, device):
    import torch
    if W.x_dtype == "bf16":
        x = torch.from_numpy(W.x_bits.view(np.int16)).view(torch.bfloat16)
    else:
        x = torch.from_numpy(np.ascontiguousarray(W.x, dtype=np.float32))
    return x.to(device), torch.from_numpy(W.filters).to(device)


def run_gpu(W, device, n1=0, y_dtype=None, repeats=1):
    """The library on workload W; returns y as float64 numpy (and the plan)."""
    import torch
    import paper_2605_08451_amd as rc
    x, k = to_device(W, device)
    yd = W.y_dtype if y_dtype is None else y_dtype
    plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=yd, n1=n1)
    ws = plan.new_workspace(device)
    spec = rc.filter_spectrum(plan, k, workspace=ws)
    outs = []
    for _ in range(repeats):
        y = rc.packed_conv(plan, x, spec, workspace=ws)
        torch.cuda.synchronize(device)
        outs.append(y.float().cpu().numpy().astype(np.float64))
    return (outs if repeats > 1 else outs[0]), plan


def reference(W, method="direct"):
    if method == "direct":
        return oracle.conv_direct(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS)
    return oracle.conv_fft(W.x, W.filters, W.cu_seqlens, threads=ORACLE_THREADS)


def rel_l2(a, b):
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a))


def parity_report(y, ref, cu):
    """Global and worst per-document relative L2 errors."""
    worst = 0.0
    worst_doc = None
    for b, row in enumerate(np.asarray(cu)):
        for s0, s1 in zip(row[:-1], row[1:]):
            if s1 <= s0:
                continue
            e = rel_l2(y[b, s0:s1], ref[b, s0:s1])
            if e > worst:
                worst, worst_doc = e, (b, int(s0), int(s1))
    return rel_l2(y, ref), worst, worst_doc


def assert_parity(y, ref, cu, dtype, label=""):
    tol = TOL[dtype]
    g, d, where = parity_report(y, ref, cu)
    assert g <= tol, f"{label}: global relative L2 {g:.3e} > {tol}"
    assert d <= tol, f"{label}: document {where} relative L2 {d:.3e} > {tol}"
    return g, d
