"""rubiconv_packed_conv_noalloc (the convolution with the library's per-device scratch
array as its workspace) against rubiconv_packed_conv on the same inputs (needs an
MI355X): two calls in a row, the second on a smaller plan, each identical to the
workspace call and within the oracle bar."""
import sys

import numpy as np
import pytest

import workloads as wl
from tests.common import assert_parity, reference, to_device

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_call(device, dtype):
    import torch
    import paper_2605_08451_amd as rc
    rng = np.random.default_rng(41)
    cases = [(wl.random_rows(rng, 3, 6000, 2500), 64, 4000),   # first call
             (wl.random_rows(rng, 2, 1500, 700), 32, 900)]     # second call: smaller
    for rows, D, L in cases:
        W = wl.make_case(rows, D=D, L=L, x_dtype=dtype, seed=D + L)
        _say(f"[noalloc] {dtype} B={W.B} N={W.N} D={D} L={L}")
        x, k = to_device(W, device)
        plan = rc.Plan(W.cu_seqlens, N=W.N, D=D, L=L, x_dtype=dtype, y_dtype=dtype)
        assert plan.workspace_bytes <= rc.NOALLOC_SCRATCH_BYTES
        ws = plan.new_workspace(device)
        spec = rc.filter_spectrum(plan, k, workspace=ws)
        y_ws = rc.packed_conv(plan, x, spec, workspace=ws)
        y_na = torch.full_like(y_ws, float("nan"))
        rc.packed_conv_noalloc(plan, x, spec, y_na)
        torch.cuda.synchronize()
        a = y_na.float().cpu().numpy().astype(np.float64)
        b = y_ws.float().cpu().numpy().astype(np.float64)
        np.testing.assert_array_equal(a, b)
        assert_parity(a, reference(W), W.cu_seqlens, dtype, f"noalloc {dtype} N={W.N}")
