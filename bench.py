"""Throughput of the packed causal long convolution on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2]

A step is one pass of the whole hot path over one batch: the filter spectra of
the batch's size classes (rubiconv_filter_spectrum) and the packed convolution
(rubiconv_packed_conv), on inputs already resident in HBM.  The plan (document
table, size classes, twiddles) is built once per batch and shared by every layer,
so it is built before the timed region and timed separately.  The step is captured
once as a HIP graph and replayed: about 50 ms of untimed replays let the GPU's clocks
settle, then W warm-up replays, then K timed replays between two events.

Prints one JSON line: value = B*N*D / seconds per step / 1e6 (Mtokens*channels/s) on
the mid-length workload (B=4, N=16384, D=1024), then
  - roofline: the step's algorithmic bytes (x + y + one complex fp32 half-spectrum
    per channel, D*L*8) over the average duration of the dominant stage (the row
    stage, timed from its fork to its join with HIP events on the calling stream),
    against the 8 TB/s HBM peak; the stage's own compulsory bytes per launch are a
    separate field;
  - configs: every workload timed by the benchmarking protocol of Section 4.1 (warm-up
    replays, then 20 trials; mean and 95% confidence interval), with the fractions of
    the HBM roofline (peak and measured copy bandwidth) and of the FP32 VALU peak;
  - cpu_baseline: the CPU oracle on bounded samples of every workload (1 warm-up and
    3 timed runs each), with the host's CPU model and core count.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, published
FP32_VALU_TFLOPS = 157.3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2, help="workload index (2 = N=16384, D=1024)")
    ap.add_argument("--n1", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true",
                    help="launch every step from Python instead of replaying a captured HIP graph")
    ap.add_argument("--layers", type=int, default=4,
                    help="layers of the stacked measurement (one plan, one filter bank per layer)")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the benchmark line: the forward step over channel counts D and "
                         "filter lengths L on the same document structure, one JSON line each")
    ap.add_argument("--no-ct", action="store_true",
                    help="skip the masked Cooley-Tukey variant's measurement")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the gradient measurement (dx and dk steps after the forward)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the protocol timing (and CPU oracle sample) of every workload")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the run, copy a buffer of this many MiB three times (a plain copy "
                         "kernel of known size, the scale for the hardware byte counters)")
    return ap.parse_args()


def progress(msg):
    """One line per phase on stderr, so that a run that stops names where it was."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# calls timed stage by stage with the library's HIP events (up to 16 per call)
PROFILE_CALLS = 20


def time_step(launch, stream, steps, warmup, eager):
    """Milliseconds per call of launch(stream): a captured HIP graph replayed steps times
    (or eager launches), bracketed by events on the timing stream."""
    import torch
    dev = stream.device
    graph = None
    if not eager:
        launch(stream)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            launch(torch.cuda.current_stream(dev))
        torch.cuda.synchronize()

    def step():
        if graph is not None:
            graph.replay()
        else:
            launch(stream)
    settle_until = time.perf_counter() + 0.05   # clocks settle under load (untimed)
    while time.perf_counter() < settle_until:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def backward_measurement(rc, plan, W, x, k, spec, ws, stream, args):
    """The two gradient calls on the same batch: dx (rubiconv_packed_conv_dx) and dk
    (rubiconv_packed_conv_dk) for a seeded upstream gradient of y's shape and dtype, each
    timed as its own step, with per-kernel event times of the same calls; then both in
    one call (rubiconv_packed_conv_backward) as a step of its own (graph replay only)."""
    import torch
    import workloads as wl
    dev = x.device
    vals, bits = wl.draw_x(np.random.default_rng(1000 + args.config), W.B, W.N, W.D, W.y_dtype)
    if W.y_dtype == "bf16":
        dy = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)
    else:
        dy = torch.from_numpy(np.ascontiguousarray(vals, dtype=np.float32)).to(dev)
    dx = torch.empty(x.shape, dtype=x.dtype, device=dev)
    dk = torch.empty((W.D, W.L), dtype=torch.float32, device=dev)
    dk_ws = plan.new_dk_workspace(dev)

    def launch_dx(s):
        rc.packed_conv_dx(plan, dy, spec, dx=dx, workspace=ws, stream=s)

    def launch_dk(s):
        rc.packed_conv_dk(plan, x, dy, dk=dk, workspace=dk_ws, stream=s)
    progress("dx step")
    dx_ms = time_step(launch_dx, stream, args.steps, args.warmup, args.eager)
    progress("dk step")
    dk_ms = time_step(launch_dk, stream, args.steps, args.warmup, args.eager)
    def launch_bwd(s):
        rc.packed_conv_backward(plan, x, dy, spec, dx=dx, dk=dk, workspace=dk_ws, stream=s)
    progress("fused backward step")
    bwd_ms = time_step(launch_bwd, stream, args.steps, args.warmup, args.eager)
    progress("gradient stages")
    calls = min(args.steps, PROFILE_CALLS)
    plan.profile_start(2 * calls)
    for _ in range(calls):
        launch_dx(stream)
        launch_dk(stream)
    kt = plan.profile_read()
    plan.profile_start(0)
    tok_ch = W.B * W.N * W.D
    sx = 2 if W.x_dtype == "bf16" else 4
    sy = 2 if W.y_dtype == "bf16" else 4
    # compulsory bytes: dx reads dy and the filter spectrum (D L 8, as for the forward)
    # and writes dx; dk reads x and dy and writes dk (D L 4)
    dx_min = tok_ch * (sx + sy) + W.D * W.L * 8
    dk_min = tok_ch * (sx + sy) + W.D * W.L * 4
    out = {"dx_ms": round(dx_ms, 4), "dk_ms": round(dk_ms, 4), "backward_ms": round(bwd_ms, 4),
           "dx_value": round(tok_ch / (dx_ms * 1e-3) / 1e6, 1),
           "dk_value": round(tok_ch / (dk_ms * 1e-3) / 1e6, 1),
           "backward_value": round(tok_ch / (bwd_ms * 1e-3) / 1e6, 1),
           "unit": "Mtokens*channels/s",
           "dx_hbm_roofline_frac_step": round(dx_min / (dx_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "dk_hbm_roofline_frac_step": round(dk_min / (dk_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "stages_us": {n: round(1e3 * tot / calls, 1) for n, (c, tot) in kt.items()}}
    del dk_ws, dx, dk, dy
    return out


def ct_measurement(rc, W, x, k, y, stream, four_step_ms, args):
    """The masked Cooley-Tukey variant (Algorithm 2) on the same batch: its own plan,
    then a step of the same scope (filter spectra + convolution), and the convolution
    alone, with the padded transform size the power-of-two rule gives."""
    import torch
    dev = x.device
    t0 = time.perf_counter()
    try:
        plan = rc.CTPlan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=W.y_dtype)
    except rc.RubiconvError as e:
        return {"skipped": str(e)}
    plan_ms = (time.perf_counter() - t0) * 1e3
    ws = plan.new_workspace(dev)
    spec = plan.new_spectrum(dev)
    yc = torch.empty_like(y)

    def launch(s):
        rc.ct_filter_spectrum(plan, k, spectrum=spec, workspace=ws, stream=s)
        rc.ct_packed_conv(plan, x, spec, y=yc, workspace=ws, stream=s)

    def launch_conv(s):
        rc.ct_packed_conv(plan, x, spec, y=yc, workspace=ws, stream=s)
    ms = time_step(launch, stream, args.steps, args.warmup, args.eager)
    conv_ms = time_step(launch_conv, stream, args.steps, args.warmup, args.eager)
    t = plan.doc_table()
    padded = int(t[:, 4].astype(np.int64).sum())
    tok_ch = W.B * W.N * W.D
    out = {"ms_per_step": round(ms, 4), "conv_ms": round(conv_ms, 4),
           "value": round(tok_ch / (ms * 1e-3) / 1e6, 1), "unit": "Mtokens*channels/s",
           "four_step_speedup": round(ms / four_step_ms, 3),
           "padded_points_per_token": round(padded / (W.B * W.N), 3),
           "spectrum_MB": round(plan.spectrum_bytes / 1e6, 1),
           "workspace_MB": round(plan.workspace_bytes / 1e6, 1), "plan_ms": round(plan_ms, 3)}
    plan.close()
    del ws, spec, yc
    return out


def stacked_measurement(rc, plan, W, x, stream, plan_ms, args):
    """One plan shared by a stack of layers (the plan depends only on the document
    boundaries): each layer transforms its own filter bank and convolves the previous
    layer's output.  Reports the per-layer cost and the per-layer cost with the plan
    amortised over the stack."""
    import torch
    import workloads as wl
    dev = x.device
    rng = np.random.default_rng(2000 + args.config)
    banks = [torch.from_numpy(wl.decaying_filters(rng, W.D, W.L)).to(dev) for _ in range(args.layers)]
    chain = W.x_dtype == W.y_dtype
    ydt = x.dtype if chain else (torch.float32 if W.y_dtype == "f32" else torch.bfloat16)
    outs = [torch.empty(x.shape, dtype=ydt, device=dev) for _ in range(args.layers)]
    ws = plan.new_workspace(dev)
    specs = [plan.new_spectrum(dev) for _ in range(args.layers)]

    def launch(s):
        inp = x
        for i in range(args.layers):
            rc.filter_spectrum(plan, banks[i], spectrum=specs[i], workspace=ws, stream=s)
            rc.packed_conv(plan, inp, specs[i], y=outs[i], workspace=ws, stream=s)
            if chain:
                inp = outs[i]
    ms = time_step(launch, stream, args.steps, args.warmup, args.eager)
    per_layer = ms / args.layers
    del banks, outs, specs, ws
    # a new batch's plan once the process has built one (operand tables cached)
    t0 = time.perf_counter()
    plan2 = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=W.y_dtype,
                    n1=args.n1)
    warm_ms = (time.perf_counter() - t0) * 1e3
    plan2.close()
    return {"layers": args.layers, "ms_per_stack": round(ms, 4),
            "ms_per_layer": round(per_layer, 4),
            "ms_per_layer_with_plan": round((ms + warm_ms) / args.layers, 4),
            "plan_ms_first": round(plan_ms, 3), "plan_ms": round(warm_ms, 3), "chained": chain}


def sweep(args):
    """Forward step (filter spectra + convolution, graph replay) over D and L on the
    document structure of the chosen workload."""
    import torch
    import paper_2605_08451_amd as rc
    import workloads as wl
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    base = wl.make_config(args.config)
    rows = wl.rows_from_cu(base.cu_seqlens)
    for D in (256, 512, 1024, 2048):
        for L in (1024, 4096, 16384):
            W = wl.make_case(rows, D=D, L=min(L, 4 * base.N), x_dtype=base.x_dtype, seed=D + L)
            if W.x_dtype == "bf16":
                x = torch.from_numpy(W.x_bits.view(np.int16)).view(torch.bfloat16).to(dev)
            else:
                x = torch.from_numpy(W.x).to(dev)
            k = torch.from_numpy(W.filters).to(dev)
            plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=W.y_dtype)
            ws, spec = plan.new_workspace(dev), plan.new_spectrum(dev)
            y = torch.empty(x.shape, dtype=x.dtype if W.y_dtype == W.x_dtype else torch.float32,
                            device=dev)

            def launch(s):
                rc.filter_spectrum(plan, k, spectrum=spec, workspace=ws, stream=s)
                rc.packed_conv(plan, x, spec, y=y, workspace=ws, stream=s)
            ms = time_step(launch, stream, args.steps, args.warmup, args.eager)
            tok_ch = W.B * W.N * W.D
            print(json.dumps({"sweep": wl.CONFIG_NAMES[args.config], "D": D, "L": W.L,
                              "ms_per_step": round(ms, 4),
                              "value": round(tok_ch / (ms * 1e-3) / 1e6, 1),
                              "unit": "Mtokens*channels/s"}), flush=True)
            del x, k, plan, ws, spec, y
            torch.cuda.empty_cache()


def kernel_bytes(info, W, plan):
    """Compulsory HBM bytes of each launch: its inputs read once and its outputs written
    once.  Grid elements hold two channels (complex fp32 for fp32 inputs, complex fp16
    for bf16 inputs: esz / 2 bytes per grid point and channel)."""
    D, G, Gc, n1 = W.D, info["grid_points"], info["class_points"], info["n1"]
    sx = 2 if W.x_dtype == "bf16" else 4
    sy = 2 if W.y_dtype == "bf16" else 4
    esz = 4 if W.x_dtype == "bf16" else 8
    tok = W.B * W.N * D
    ms = [int(m) for m in plan.doc_table()[:, 4]]
    classes = sorted(set(ms))
    taps = {m: min(W.L, (n1 * m + 1) // 2) for m in classes}
    row = 0
    for m in classes:   # document grids read + written, the class's filter grid read per document
        row += ms.count(m) * (n1 * m * D * esz + n1 * m * D * esz // 2)
    # the matrix-core column passes (bf16 x, N1 = 256, whole 32-channel blocks) take the
    # filter taps as fp16 channel pairs, the others as fp32
    st = 2 if (W.x_dtype == "bf16" and n1 == 256 and D % 32 == 0) else 4
    out = {
        "row_conv": row,
        "col_fwd": tok * sx + G * D * esz // 2,
        "col_inv": G * D * esz // 2 + tok * sy,
        "filter_transpose": (4 + st) * D * max(taps.values()),
        "filter_col_fwd": st * D * sum(taps.values()) + Gc * D * esz // 2,
        "prescale": tok * sx,
    }
    return out


def sources_digest():
    """SHA-256 over the library's kernel and runtime sources (name + bytes, sorted)."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2605_08451_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".cpp", ".hpp")):
            h.update(name.encode())
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def recorded_traffic(stage, workload):
    """HBM bytes per launch of `stage` from the committed counter summary of this workload
    (rocprofv3 FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known size), or None
    when there is none or the library sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    for line in open(path):
        if line.strip().startswith("traffic {"):
            rec = json.loads(line.strip()[len("traffic "):])
            if rec.get("sources_sha256") != sources_digest():
                return None
            return rec["stages"].get(stage)
    return None


def recorded_mfma(workload):
    """Matrix-core counters of this workload's step from the committed summary
    (profiles/mfma_<workload>.md), or None when there is none or the library sources
    changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"mfma_{workload}.md")
    if not os.path.exists(path):
        return None
    for line in open(path):
        if line.strip().startswith("mfma {"):
            rec = json.loads(line.strip()[len("mfma "):])
            if rec.get("sources_sha256") != sources_digest():
                return None
            rec.pop("sources_sha256", None)
            return rec
    return None


def cpu_info():
    """The host's CPU model and logical CPU count (as the OS reports them)."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, os.cpu_count() or 1


ORACLE_THREADS = 16   # one GPU's share of the host's cores


def cpu_baseline(W, target_s=1.0, variants=("fft",)):
    """The CPU oracle on a bounded sample of workload W: all rows and tokens, the first
    nch channels, nch chosen so that one run takes about target_s seconds; 1 warm-up and
    3 timed runs per variant (per-document radix-2 FFT, and the defining sum where it is
    the parity reference)."""
    import oracle
    threads = min(ORACLE_THREADS, os.cpu_count() or 1)
    fns = {"fft": oracle.conv_fft, "direct": oracle.conv_direct}
    out = {}
    for var in variants:
        fn = fns[var]

        def run(nch):
            x = np.ascontiguousarray(W.x[:, :, :nch])
            k = np.ascontiguousarray(W.filters[:nch])
            t0 = time.perf_counter()
            fn(x, k, W.cu_seqlens, threads=threads)
            return time.perf_counter() - t0
        probe = min(W.D, 4)
        t_probe = run(probe)
        nch = int(max(1, min(W.D, round(probe * target_s / max(t_probe, 1e-4)))))
        if nch > probe:   # one more sizing step from the larger sample (the probe's overheads weigh less)
            nch = int(max(1, min(W.D, round(nch * target_s / max(run(nch), 1e-4)))))
        run(nch)                                     # warm-up
        ts = [run(nch) for _ in range(3)]
        t = float(np.mean(ts))
        out[var] = {"value": round(W.B * W.N * nch / t / 1e6, 3), "unit": "Mtokens*channels/s",
                    "channels": nch, "of_channels": W.D, "run_s": [round(v, 4) for v in ts]}
    return out, threads


def t_quantile_975(dof):
    from scipy import stats
    return float(stats.t.ppf(0.975, dof))


def protocol_time(launch, stream, warmup=5, trials=20, target_ms=3.0):
    """Section 4.1's protocol on one captured step: warm-up replays, then `trials` timed
    trials of `reps` replays each (HIP events on the timing stream); mean and the 95%
    confidence half-width of the per-step time over the trials, in ms."""
    import torch
    dev = stream.device
    launch(stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        launch(torch.cuda.current_stream(dev))
    torch.cuda.synchronize()
    settle_until = time.perf_counter() + 0.05   # clocks settle under load (untimed)
    while time.perf_counter() < settle_until:
        for _ in range(10):
            graph.replay()
        torch.cuda.synchronize()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    reps = int(max(1, min(200, target_ms / max(e0.elapsed_time(e1), 1e-3))))
    per = []
    for _ in range(trials):
        e0.record(stream)
        for _ in range(reps):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        per.append(e0.elapsed_time(e1) / reps)
    per = np.array(per)
    mean = float(per.mean())
    ci = float(t_quantile_975(trials - 1) * per.std(ddof=1) / np.sqrt(trials))
    del graph
    return mean, ci, reps


def step_min_bytes(W):
    """Algorithmic bytes of one step: x and y once each and one complex fp32
    half-spectrum per channel (D * L * 8 bytes), whatever the implementation stores."""
    sx = 2 if W.x_dtype == "bf16" else 4
    sy = 2 if W.y_dtype == "bf16" else 4
    return W.B * W.N * W.D * (sx + sy) + W.D * W.L * 8


def alg_flops(W, n1=256):
    """Algorithmic flops of one step: per document and channel one forward and one
    inverse real transform at Algorithm 1's padded size P = n1 ceil((L_i + min(L_i, L)
    - 1) / n1) (5 P log2 P per complex transform, half of it for a real one) and 3 P for
    the product."""
    tot = 0.0
    for row in np.asarray(W.cu_seqlens):
        for s0, s1 in zip(row[:-1], row[1:]):
            n = int(s1 - s0)
            if n <= 0:
                continue
            P = n1 * -(-(n + min(n, W.L) - 1) // n1)
            tot += 5.0 * P * np.log2(P) + 3.0 * P
    return tot * W.D


def copy_bandwidth(dev, mib=1024):
    """Read + write bytes per second of a plain device copy of `mib` MiB (GB/s)."""
    import torch
    src = torch.ones((mib << 20) // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbps = 2 * (mib << 20) / (e0.elapsed_time(e1) / 10 * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbps


def configs_measurement(args, copy_gbps, cpu):
    """Every workload: the step (filter spectra + convolution) by the protocol, its
    throughput and roofline fractions, and (cpu) the oracle baseline on a sample."""
    import torch
    import paper_2605_08451_amd as rc
    import workloads as wl
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    out, cpu_out, threads = {}, {}, None
    for i in range(5):
        progress(f"workload {wl.CONFIG_NAMES[i]}")
        W = wl.make_config(i)
        if W.x_dtype == "bf16":
            x = torch.from_numpy(W.x_bits.view(np.int16)).view(torch.bfloat16).to(dev)
        else:
            x = torch.from_numpy(W.x).to(dev)
        k = torch.from_numpy(W.filters).to(dev)
        plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=W.y_dtype)
        ws, spec = plan.new_workspace(dev), plan.new_spectrum(dev)
        y = torch.empty_like(x)

        def launch(s):
            rc.filter_spectrum(plan, k, spectrum=spec, workspace=ws, stream=s)
            rc.packed_conv(plan, x, spec, y=y, workspace=ws, stream=s)
        mean, ci, reps = protocol_time(launch, stream, warmup=args.warmup, trials=20)
        tok_ch = W.B * W.N * W.D
        mb = step_min_bytes(W)
        fl = alg_flops(W)
        out[f"c{i}"] = {
            "workload": wl.CONFIG_NAMES[i], "ms_mean": round(mean, 5), "ms_ci95": round(ci, 5),
            "trials": 20, "replays_per_trial": reps,
            "value": round(tok_ch / (mean * 1e-3) / 1e6, 1), "unit": "Mtokens*channels/s",
            "min_bytes": mb, "hbm_frac_of_peak": round(mb / (mean * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "hbm_frac_of_copy": round(mb / (mean * 1e-3) / 1e9 / copy_gbps, 4),
            "alg_flops": round(fl), "valu_frac_of_peak": round(fl / (mean * 1e-3) / 1e12 / FP32_VALU_TFLOPS, 4),
            "docs": plan.info()["n_docs"], "cu_seqlens_sha256_16": W.cu_hash()}
        print(f"[bench] c{i}: {mean:.4f} +- {ci:.4f} ms", file=sys.stderr, flush=True)
        if i == 4 and not args.no_ct:   # the masked Cooley-Tukey variant on the long documents
            ctp = rc.CTPlan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=W.y_dtype)
            cws, cspec = ctp.new_workspace(dev), ctp.new_spectrum(dev)

            def launch_ct(s):
                rc.ct_filter_spectrum(ctp, k, spectrum=cspec, workspace=cws, stream=s)
                rc.ct_packed_conv(ctp, x, cspec, y=y, workspace=cws, stream=s)
            cm, cc, _ = protocol_time(launch_ct, stream, warmup=args.warmup, trials=20)
            out[f"c{i}"]["cooley_tukey_ms_mean"] = round(cm, 5)
            out[f"c{i}"]["cooley_tukey_ms_ci95"] = round(cc, 5)
            del ctp, cws, cspec
        del x, k, plan, ws, spec, y
        torch.cuda.empty_cache()
        if cpu:
            variants = ("fft", "direct") if i in (0, 1, 3) else ("fft",)
            cpu_out[f"c{i}"], threads = cpu_baseline(W, target_s=1.0 if i == args.config else 0.5,
                                                     variants=variants)
            print(f"[bench] c{i} cpu oracle done", file=sys.stderr, flush=True)
    return out, cpu_out, threads


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the convolution shards over channels with no exchange; see the design notes)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2605_08451_amd as rc
    import workloads as wl

    if args.sweep:
        sweep(args)
        return
    dev = torch.device("cuda:0")
    progress(f"step of {wl.CONFIG_NAMES[args.config]}")
    W = wl.make_config(args.config)
    if W.x_dtype == "bf16":
        x = torch.from_numpy(W.x_bits.view(np.int16)).view(torch.bfloat16).to(dev)
    else:
        x = torch.from_numpy(W.x).to(dev)
    k = torch.from_numpy(W.filters).to(dev)

    t0 = time.perf_counter()
    plan = rc.Plan(W.cu_seqlens, N=W.N, D=W.D, L=W.L, x_dtype=W.x_dtype, y_dtype=W.y_dtype,
                   n1=args.n1)
    plan_ms = (time.perf_counter() - t0) * 1e3
    info = plan.info()
    ws = plan.new_workspace(dev)
    spec = plan.new_spectrum(dev)
    y = torch.empty_like(x) if W.y_dtype == W.x_dtype else torch.empty(
        x.shape, dtype=torch.float32 if W.y_dtype == "f32" else torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream(dev)

    def launch(s):
        rc.filter_spectrum(plan, k, spectrum=spec, workspace=ws, stream=s)
        rc.packed_conv(plan, x, spec, y=y, workspace=ws, stream=s)

    graph = None
    if not args.eager:
        # one step captured as a HIP graph (the library only enqueues kernels and event
        # fork/joins on the capturing stream), replayed on the timing stream
        launch(stream)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            launch(torch.cuda.current_stream(dev))
        torch.cuda.synchronize()

    def step():
        if graph is not None:
            graph.replay()
        else:
            launch(stream)

    # the GPU's clocks ramp up under load: replay untimed for about 50 ms before the
    # warm-up steps (measured: 5 warm-ups alone leave the timed steps 7% slow)
    settle_until = time.perf_counter() + 0.05
    while time.perf_counter() < settle_until:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = e0.elapsed_time(e1) / args.steps

    # stage durations: HIP events the library records on the stream each stage runs on
    # (a stage that forks to side streams is timed from before its fork to after its join)
    progress("stages")
    calls = min(args.steps, PROFILE_CALLS)
    plan.profile_start(2 * calls)
    for _ in range(calls):
        launch(stream)
    kt = plan.profile_read()
    plan.profile_start(0)
    kb = kernel_bytes(info, W, plan)
    stages = {n: {"launches_per_step": c / calls, "avg_us": 1e3 * tot / c,
                  "us_per_step": 1e3 * tot / calls,
                  "compulsory_bytes_per_launch": round(kb[n] * calls / c) if n in kb else None,
                  "compulsory_GBps": (kb[n] * calls / c) / (tot / c * 1e-3) / 1e9 if n in kb else None}
              for n, (c, tot) in kt.items()}
    # the dominant stage: the longest one of a step
    dom = max(stages, key=lambda n: stages[n]["us_per_step"])
    dom_us = stages[dom]["avg_us"]
    min_bytes = step_min_bytes(W)
    achieved = min_bytes / (dom_us * 1e-6) / 1e9
    copy_gbps = copy_bandwidth(dev)

    tok_ch = W.B * W.N * W.D
    value = tok_ch / (ms * 1e-3) / 1e6
    flops = alg_flops(W)
    out = {
        "metric": "packed-conv Mtokens*channels/s at N=16384,D=1024; % HBM roofline",
        "value": round(value, 1),
        "unit": "Mtokens*channels/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        # arithmetic type of the path: complex fp16 grids and matrix-core products with
        # fp32 accumulation for bf16 inputs, fp32 throughout for fp32 inputs
        "dtype": "f16" if W.x_dtype == "bf16" else "f32", "accumulate": "f32", "data": "synthetic",
        "config": {"workload": wl.CONFIG_NAMES[args.config], "B": W.B, "N": W.N, "D": W.D,
                   "L": W.L, "x_dtype": W.x_dtype, "y_dtype": W.y_dtype, "n1": info["n1"],
                   "docs": info["n_docs"], "size_classes": info["n_classes"],
                   "cu_seqlens_sha256_16": W.cu_hash(), "parallelism": "none (1 GPU)"},
        "step_min_bytes": min_bytes,
        "hbm_roofline_frac_step": round(min_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "hbm_frac_of_copy_step": round(min_bytes / (ms * 1e-3) / 1e9 / copy_gbps, 4),
        "valu_frac_step": round(flops / (ms * 1e-3) / 1e12 / FP32_VALU_TFLOPS, 4),
        "copy_GBps": round(copy_gbps, 1),
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic(dom, wl.CONFIG_SLUGS[args.config]),
                     "bytes": min_bytes, "avg_us": round(dom_us, 2),
                     "compulsory_bytes_per_launch": stages[dom]["compulsory_bytes_per_launch"]},
        "stages": {n: {kk: (round(vv, 2) if isinstance(vv, float) else vv) for kk, vv in d.items()}
                   for n, d in stages.items()},
        "mfma": recorded_mfma(wl.CONFIG_SLUGS[args.config]),
        "plan_ms": round(plan_ms, 3),
        "execution": "eager launches" if graph is None else "HIP graph replay of one captured step",
        "wall_s_timed": round(wall, 4),
    }
    del graph
    cpu_cfg, threads = {}, None
    if not args.no_configs:
        progress("every workload")
        out["configs"], cpu_cfg, threads = configs_measurement(args, copy_gbps, not args.no_cpu_baseline)
    if not args.no_backward:
        out["backward"] = backward_measurement(rc, plan, W, x, k, spec, ws, stream, args)
    if not args.no_ct:
        progress("Cooley-Tukey variant")
        out["cooley_tukey"] = ct_measurement(rc, W, x, k, y, stream, ms, args)
    if args.layers > 0:
        progress("stacked layers")
        out["stacked"] = stacked_measurement(rc, plan, W, x, stream, plan_ms, args)
    if not args.no_cpu_baseline:
        progress("cpu baseline")
        model, ncpu = cpu_info()
        key = f"c{args.config}"
        if key not in cpu_cfg:
            cpu_cfg[key], threads = cpu_baseline(W, target_s=1.0)
        c = cpu_cfg[key]["fft"]
        out["cpu_baseline"] = {
            "value": c["value"], "unit": "Mtokens*channels/s", "cores": threads, "kind": "oracle",
            "sample": f"per-document radix-2 FFT variant (fp64) on {W.B} rows x {W.N} tokens x "
                      f"{c['channels']} of {W.D} channels of {wl.CONFIG_NAMES[args.config]}; "
                      f"1 warm-up and 3 timed runs ({', '.join(str(v) for v in c['run_s'])} s)",
            "cpu_model": model, "host_logical_cpus": ncpu, "configs": cpu_cfg}
    print(json.dumps(out), flush=True)
    if args.copy_probe_mib > 0:
        # an elementwise kernel that reads and writes copy_probe_mib MiB once each
        src = torch.zeros((args.copy_probe_mib << 20) // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()


if __name__ == "__main__":
    main()
