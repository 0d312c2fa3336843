"""Throughput of one LR-QAT linear layer (forward + STE backward) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 2] [--no-cpu-baseline]

A step is lrqat_forward followed by lrqat_backward (dX, dA, dB) for every linear
of the workload, each on its own batch of seeded synthetic inputs already
resident in device memory.  The value is the rate of eager launches on one
stream; the same step is also captured once in a HIP graph and replayed (each
replay checked bit for bit against an eager step), its rate reported beside
it, and the per-kernel times come from eager steps.
Before the W warm-up steps the step runs, untimed, for --settle-ms of wall time
(reported as clock_settle): the GPU's clocks rise over the first few hundred
steps, and a short warm-up would time a clock that is still rising.  The default workload is the
LLaMA-7B q_proj-shaped layer 4096 -> 4096 with 8 x 1024 tokens, rank 32,
alpha 32, W4 per-channel and Phi0 in fixed point Q4.4.  Prints one JSON line.

value = algorithmic flops per step (sum over the layers of 6 T m k + 8 m k r)
/ step time, in TFLOP/s.
roofline: the kernel with the largest share of the step, timed with HIP events
on the library's stream, against the bf16 dense MFMA peak of 2.5 PFLOP/s.
cpu_baseline: the CPU oracle on a bounded token sample of the same layer.
Also reported: per-step p10/p50/p90, the merge (lrqat_merge_to_int4) as
algorithmic GB/s beside a measured device-copy rate, and the device memory the
layer holds (analytic, with checkpointing) beside torch's measured peak.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "LR-QAT linear fwd+bwd TFLOP/s at LLaMA-7B shapes; % of bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=500)
    ap.add_argument("--settle-ms", type=float, default=400.0,
                    help="untimed repetitions of the step for this long before the warm-up steps (0: none)")
    ap.add_argument("--workload", type=int, default=2)
    ap.add_argument("--rank", type=int, default=0, help="override the workload's rank r (and alpha = r)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true", help="time eager launches only (no HIP graph)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    ap.add_argument("--vendor-gemm", action="store_true",
                    help="only time the vendor library's plain bf16 GEMMs of the layer's three shapes and exit")
    ap.add_argument("--rows", action="store_true",
                    help="only time the rows after the hot path (scale gradient with a zero offset, inference "
                         "on merged weights, the AdamW step, the L^p and LoftQ initialisations) and exit")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (calibrates rocprofv3 byte counters) and exit")
    return ap.parse_args()


def copy_probe(mib):
    """A plain device-to-device copy of known size, for scaling FETCH_SIZE / WRITE_SIZE."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4}), flush=True)


def _time_us(fn, reps=20, warm=5):
    import torch
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return 1e3 * e0.elapsed_time(e1) / reps


def rows_bench():
    """The rows after the hot path, each on its paper-scale shape with seeded synthetic inputs:
    the backward with the scale gradient and an asymmetric zero offset (vs without), inference on
    the merged int4 weights (vs the training forward), the AdamW step over every adapter and scale
    of a LLaMA-7B model, and the two setup-side initialisations."""
    import torch
    from paper_2406_06385_amd import inputs as I
    from paper_2406_06385_amd import lrqat
    lrqat.load_library()
    dev = torch.device("cuda:0")
    bf = lambda a: torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(dev)
    out = {}
    wl = I.WORKLOADS[2]
    L0 = wl.layers[0]
    T, m, k, r = wl.tokens, L0.m, L0.k, wl.rank
    inp = I.make_layer_inputs(wl, 0)
    W0 = torch.from_numpy(inp.W0).to(dev)
    A, B = torch.from_numpy(inp.A).to(dev), torch.from_numpy(inp.B).to(dev)
    X, dY = bf(inp.X), bf(inp.dY)
    gemm_flop = 2.0 * T * m * k

    # f1: backward with ds and z (asymmetric Q4.4), against the symmetric backward without ds
    spec = lrqat.LayerSpec(m, k, r, wl.alpha, 4, "q8", 0, 0, "bf16")
    s_sym, phi_sym = lrqat.lrqat_init_from_weights(spec, W0)
    s_as, z_as, phi_as = lrqat.lrqat_init_from_weights(spec, W0, asymmetric=True)
    dX = torch.empty_like(X)
    dA, dB = torch.empty((m, r), device=dev), torch.empty((r, k), device=dev)
    ds = torch.empty(s_as.shape, device=dev)
    wb = lrqat.workspace(lrqat.lrqat_backward_workspace_size(spec, T), dev)
    t_plain = _time_us(lambda: lrqat.lrqat_backward(spec, X, phi_sym, s_sym, A, B, dY, dX=dX, dA=dA, dB=dB, ws=wb))
    t_ds = _time_us(lambda: lrqat.lrqat_backward(spec, X, phi_as, s_as, A, B, dY, dX=dX, dA=dA, dB=dB, ws=wb,
                                                 z=z_as, ds=ds))
    out["f1_backward_ds_z"] = {"layer": [m, k], "tokens": T, "us": t_ds, "us_without_ds_z": t_plain,
                               "overhead": t_ds / t_plain - 1.0, "TFLOP/s": 2 * gemm_flop / (t_ds * 1e-6) / 1e12}

    # f2: inference on the merged weights (packed INT4 Phi0 as for W_Z), against the training forward
    spec4 = lrqat.LayerSpec(m, k, r, wl.alpha, 4, "int_packed2", 0, 0, "bf16")
    s4, phi4 = lrqat.lrqat_init_from_weights(spec4, W0)
    Wz = lrqat.lrqat_merge_to_int4(spec4, phi4, A, B)
    Y = torch.empty((T, m), dtype=torch.bfloat16, device=dev)
    wi = lrqat.workspace(lrqat.lrqat_infer_workspace_size(spec4, T), dev)
    wf = lrqat.workspace(lrqat.lrqat_forward_workspace_size(spec4, T), dev)
    t_inf = _time_us(lambda: lrqat.lrqat_infer_forward(spec4, X, Wz, s4, Y=Y, ws=wi))
    t_fwd = _time_us(lambda: lrqat.lrqat_forward(spec4, X, phi4, s4, A, B, Y=Y, ws=wf))
    out["f2_inference_merged_int4"] = {"layer": [m, k], "tokens": T, "us": t_inf, "TFLOP/s": gemm_flop / (t_inf * 1e-6) / 1e12,
                                       "training_forward_us": t_fwd, "saved_by_merge_us": t_fwd - t_inf}
    del Wz, wi, wf

    # f3: AdamW over all adapters (A, B) and scales of a LLaMA-7B model at r = 32 (32 blocks of
    # q, k, v, o 4096x4096 and gate, up 11008x4096, down 4096x11008), three parameter groups
    shapes = [(4096, 4096)] * 4 + [(11008, 4096)] * 2 + [(4096, 11008)]
    nA = 32 * sum(mm * r for mm, kk in shapes)
    nB = 32 * sum(r * kk for mm, kk in shapes)
    ns = 32 * sum(mm for mm, kk in shapes)
    gen = torch.Generator(device=dev).manual_seed(7)
    groups = []
    for n, lr_max, wd in ((nA, 1e-3, 0.0), (nB, 1e-3, 0.0), (ns, 1e-5, 0.0)):
        P = torch.randn(n, device=dev, generator=gen) * 0.01
        groups.append(dict(param=P, grad=torch.randn(n, device=dev, generator=gen) * 1e-4,
                           exp_avg=torch.zeros_like(P), exp_avg_sq=torch.zeros_like(P), lr_max=lr_max, weight_decay=wd))
    step = [0]

    def adam():
        step[0] += 1
        lrqat.lrqat_adamw_step(groups, step[0], 10000, 100)
    t_adam = _time_us(adam)
    nparam = nA + nB + ns
    bytes_adam = nparam * (4 * 5 + 4 * 3)  # reads: g (norm pass and update), p, m, v; writes: p, m, v
    out["f3_adamw_llama7b_adapters"] = {"params": nparam, "us": t_adam, "algorithmic_bytes": bytes_adam,
                                        "GB/s": bytes_adam / (t_adam * 1e-6) / 1e9,
                                        "frac_of_hbm_peak": bytes_adam / (t_adam * 1e-6) / 1e9 / PEAK_HBM_GBS}
    del groups

    # f4: L^p range search (p = 2.4, 100 candidates) on the q_proj layer; LoftQ (T = 1) on the MLP's
    # gate projection, packed INT4, r = 32, 32 subspace iterations
    specq = lrqat.LayerSpec(m, k, r, wl.alpha, 4, "q8", 0, 0, "bf16")
    t_lp = _time_us(lambda: lrqat.lrqat_init_lp(specq, W0, 2.4, 100), reps=5, warm=1)
    wl3 = I.WORKLOADS[3]
    L3 = wl3.layers[0]
    W3 = torch.from_numpy(I.gen_w0(L3.m, L3.k, 11, 12, 0.02, 0.0)).to(dev)
    spec3 = lrqat.LayerSpec(L3.m, L3.k, 32, 32.0, 4, "int_packed2", 0, 0, "bf16")
    s3, _ = lrqat.lrqat_init_from_weights(spec3, W3)
    t_lq = _time_us(lambda: lrqat.lrqat_init_loftq(spec3, W3, s3, 32), reps=3, warm=1)
    out["f4_init"] = {"lp_search": {"layer": [m, k], "p": 2.4, "candidates": 100, "us": t_lp,
                                    "GB/s_of_W0": m * k * 4 / (t_lp * 1e-6) / 1e9},
                      "loftq": {"layer": [L3.m, L3.k], "rank": 32, "iterations": 32, "us": t_lq}}
    print(json.dumps({"rows": out}), flush=True)


def vendor_gemm(wl):
    """Context, not part of the path: torch.matmul (hipBLASLt) on plain bf16 GEMMs of the same three
    shapes as the layer's forward (X W^T), dX (dY W) and dW (dY^T X), with no quantisation work."""
    import torch
    spec = wl.layers[0]
    T, m, k = wl.tokens, spec.m, spec.k
    X = torch.randn(T, k, dtype=torch.bfloat16, device="cuda")
    W = torch.randn(m, k, dtype=torch.bfloat16, device="cuda")
    dY = torch.randn(T, m, dtype=torch.bfloat16, device="cuda")
    out = {}
    for name, fn in (("fwd_X_Wt", lambda: X @ W.t()), ("dx_dY_W", lambda: dY @ W), ("dw_dYt_X", lambda: dY.t() @ X)):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(20):
            fn()
        e1.record()
        torch.cuda.synchronize()
        us = 1e3 * e0.elapsed_time(e1) / 20
        out[name] = {"us": us, "TFLOP/s": 2.0 * T * m * k / (us * 1e-6) / 1e12}
    print(json.dumps({"vendor_gemm": out, "workload": wl.name}), flush=True)


def kernel_flops(name, wl):
    """Algorithmic flops of one step's launches of a library kernel (the useful
    work they do), summed over the workload's layers."""
    T, r = wl.tokens, wl.rank
    per = {"gemm_fwd": lambda m, k: 2.0 * T * m * k,
           "gemm_dx": lambda m, k: 2.0 * T * m * k,
           "gemm_dw": lambda m, k: 2.0 * T * m * k + 4.0 * m * k * r,
           "grid": lambda m, k: 2.0 * m * k * r}.get(name)
    return None if per is None else sum(per(L.m, L.k) for L in wl.layers)


# Sources each library kernel is compiled from: a traffic record stays valid
# while these files are unchanged.
KERNEL_SOURCES = {
    "gemm_fwd": ["gemm_impl.h", "gemm_fwd.hip", "kernels.h", "common.h"],
    "gemm_dx": ["gemm_impl.h", "gemm_dx.hip", "kernels.h", "common.h"],
    "gemm_dw": ["gemm_impl.h", "gemm_dw.hip", "kernels.h", "common.h"],
    "grid": ["grid.hip", "grid_swar.h", "kernels.h", "common.h"],
    "reduce": ["gemm.hip", "kernels.h", "common.h"],
}


def traffic_record(kernel):
    """HBM bytes per launch measured with rocprofv3 counters, if the kernel's
    sources are unchanged since the measurement (else None)."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}.json")
    if not os.path.exists(path) or kernel not in KERNEL_SOURCES:
        return None
    rec = json.load(open(path))
    if rec.get("sources_sha256") != sources_sha(kernel):
        return None
    return rec.get("hbm_bytes_per_launch")


def sources_sha(kernel):
    """sha256 over the kernel's source files (names and contents)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2406_06385_amd", "csrc")
    for f in sorted(KERNEL_SOURCES[kernel]):
        h.update(f.encode())
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()


def cpu_baseline(wl, inp, target_s):
    """Oracle forward + backward of the workload's first layer on its first Ts tokens."""
    from oracle import lrqat_oracle as O
    from paper_2406_06385_amd import inputs as I
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    spec = wl.layers[0]
    L = O.Layer(spec.m, spec.k, wl.rank, wl.alpha, wl.bits, wl.phi_format, wl.group_size, wl.act_bits)
    s0 = O.minmax_scale(inp.W0, wl.bits, wl.group_size)
    phi0 = O.encode_phi0(inp.W0, s0, wl.bits, wl.phi_format, wl.group_size)
    X = I.bf16_bits_to_fp32(inp.X) if wl.act_dtype == "bf16" else inp.X
    dY = (I.bf16_bits_to_fp32(inp.dY) if wl.act_dtype == "bf16" else inp.dY).astype(np.float64)

    def run(ts):
        t0 = time.perf_counter()
        O.forward(L, X[:ts], phi0, s0, inp.A, inp.B)
        O.backward(L, X[:ts], phi0, s0, inp.A, inp.B, dY[:ts])
        return time.perf_counter() - t0

    ts = 64
    dt = run(ts)
    while dt < target_s / 4 and ts < wl.tokens:
        ts = min(wl.tokens, ts * 4)
        dt = run(ts)
    # the whole layer can take well under the target: repeat it to about target_s of CPU work
    reps, total = 1, dt
    while total < target_s * 0.6 and reps < 64:
        total += run(ts)
        reps += 1
    flops = (6.0 * ts * spec.m * spec.k + 8.0 * spec.m * spec.k * wl.rank) * reps
    return {"value": flops / total / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"float64 numpy oracle forward+backward of layer {spec.name} ({spec.m}x{spec.k}) on its first "
                      f"{ts} of {wl.tokens} tokens, {reps} run(s), {total:.1f} s"}


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.rows:
        rows_bench()
        return
    if args.vendor_gemm:
        from paper_2406_06385_amd import inputs as I
        vendor_gemm(I.WORKLOADS[args.workload])
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); runs on several GPUs are not "
              f"implemented (the layer would shard along tokens with an all-reduce of dA, dB and ds)",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2406_06385_amd import inputs as I
    from paper_2406_06385_amd import lrqat

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    lrqat.load_library()
    wl = I.WORKLOADS[args.workload]
    if args.rank:
        wl = dataclasses.replace(wl, rank=args.rank, alpha=float(args.rank))
    T, r = wl.tokens, wl.rank
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def act(a):
        if wl.act_dtype == "bf16":
            return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    layers = []
    inp0 = None
    for li, lspec in enumerate(wl.layers):
        print(f"[bench] workload {wl.name}: generating inputs of layer {lspec.name} ({lspec.m}x{lspec.k})",
              file=sys.stderr, flush=True)
        inp = I.make_layer_inputs(wl, li)
        if li == 0:
            inp0 = inp
        m, k = lspec.m, lspec.k
        spec = lrqat.LayerSpec(m, k, r, wl.alpha, wl.bits, wl.phi_format, wl.group_size, wl.act_bits, wl.act_dtype)
        W0 = torch.from_numpy(inp.W0).to(dev)
        s0, phi0 = lrqat.lrqat_init_from_weights(spec, W0)
        torch.cuda.synchronize()
        del W0
        layers.append(dict(
            spec=spec, s0=s0, phi0=phi0, A=torch.from_numpy(inp.A).to(dev), B=torch.from_numpy(inp.B).to(dev),
            X=act(inp.X), dY=act(inp.dY),
            Y=torch.empty((T, m), dtype=spec.torch_dtype, device=dev),
            dX=torch.empty((T, k), dtype=spec.torch_dtype, device=dev),
            dA=torch.empty((m, r), dtype=torch.float32, device=dev),
            dB=torch.empty((r, k), dtype=torch.float32, device=dev)))
        if li:
            inp.X = inp.dY = None
    # one forward and one backward workspace, sized for the largest layer, shared by all layers
    # (the calls run one after another on one stream)
    ws_f = lrqat.workspace(max(lrqat.lrqat_forward_workspace_size(l["spec"], T) for l in layers), dev)
    ws_b = lrqat.workspace(max(lrqat.lrqat_backward_workspace_size(l["spec"], T) for l in layers), dev)
    stream = torch.cuda.current_stream()

    def step():
        # on the current stream: the default one, or the capture stream of a HIP graph
        for l in layers:
            lrqat.lrqat_forward(l["spec"], l["X"], l["phi0"], l["s0"], l["A"], l["B"], Y=l["Y"], ws=ws_f)
            lrqat.lrqat_backward(l["spec"], l["X"], l["phi0"], l["s0"], l["A"], l["B"], l["dY"], dX=l["dX"],
                                 dA=l["dA"], dB=l["dB"], ws=ws_b)

    def outputs():
        return [t.clone() for l in layers for t in (l["Y"], l["dX"], l["dA"], l["dB"])]

    def same(a, b):
        return all(torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                               y.view(torch.int16) if y.dtype == torch.bfloat16 else y) for x, y in zip(a, b))

    # clock settle: the step repeated, untimed, for a fixed wall time before the warm-up steps, so
    # that the timed steps do not run while the GPU's clocks are still rising from idle
    torch.cuda.synchronize()
    settle_steps, t_settle = 0, time.perf_counter()
    while (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
        for _ in range(10):
            step()
        settle_steps += 10
        torch.cuda.synchronize()
    settle = {"steps": settle_steps, "ms": (time.perf_counter() - t_settle) * 1e3,
              "note": "untimed repetitions of the step before the warm-up steps (clocks rise over the first "
                      "few hundred steps)"}
    print(f"[bench] clock settle: {settle_steps} steps in {settle['ms']:.0f} ms", file=sys.stderr, flush=True)
    torch.cuda.reset_peak_memory_stats(dev)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    def time_steps(run):
        """(ms per step over K steps bracketed by one pair of events, per-step ms from a second
        pass of K steps with an event after each; events between graph launches can delay
        them, so the mean comes from the pass without)."""
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            run()
        e1.record()
        torch.cuda.synchronize()
        ms_mean = e0.elapsed_time(e1) / args.steps
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        torch.cuda.synchronize()
        evs[0].record()
        for i in range(args.steps):
            run()
            evs[i + 1].record()
        torch.cuda.synchronize()
        return ms_mean, np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])

    ms_eager, per_step_eager = time_steps(step)
    # device memory of the training steps themselves (before the graph-check copies below)
    peak_mem_steps = torch.cuda.max_memory_allocated(dev)
    print(f"[bench] timed {args.steps} eager steps: {ms_eager:.4f} ms/step", file=sys.stderr, flush=True)
    # the same step captured once in a HIP graph and replayed; every replay must give the eager step's bits
    ref = outputs()
    graph_ok, graph_note = False, "not tried"
    if not args.eager:
        try:
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                step()
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step()
            graph_ok = True
            for _ in range(3):
                for l in layers:
                    for key in ("Y", "dX", "dA", "dB"):
                        l[key].fill_(float("nan"))
                g.replay()
                torch.cuda.synchronize()
                graph_ok = graph_ok and same(outputs(), ref)
                step()  # eager work between replays
                torch.cuda.synchronize()
            graph_note = "replays bit-identical to the eager step" if graph_ok else "replay differs: eager timing used"
        except Exception as e:  # pragma: no cover - capture unsupported
            graph_ok, graph_note = False, f"capture failed: {type(e).__name__}: {e}"
    # the value is the eager rate (the library's ordinary use); the graph replays run the same
    # kernels and are reported beside it
    ms, per_step = ms_eager, per_step_eager
    ms_graph, per_step_graph = None, None
    if graph_ok:
        ms_graph, per_step_graph = time_steps(g.replay)
        print(f"[bench] timed {args.steps} graph replays: {ms_graph:.4f} ms/step", file=sys.stderr, flush=True)
    peak_mem = torch.cuda.max_memory_allocated(dev)
    flops = wl.flops_fwd_bwd()
    value = flops / (ms * 1e-3) / 1e12

    # per-kernel durations (HIP events around each launch on the library's stream)
    lrqat.lrqat_timing_reset()
    lrqat.lrqat_timing_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    per = lrqat.lrqat_timing_read()
    lrqat.lrqat_timing_enable(False)
    lrqat.lrqat_timing_reset()
    nl = len(layers)
    kernels = {n: {"launches": c, "avg_us": 1e3 * t / c, "us_per_step": 1e3 * t / args.steps}
               for n, (c, t) in per.items()}
    dom = max(per, key=lambda n: per[n][1])
    dom_step_s = per[dom][1] / args.steps * 1e-3        # the dominant kernel's time per step
    dom_flops = kernel_flops(dom, wl)                    # its algorithmic flops per step
    traffic = traffic_record(dom) if nl == 1 else None
    achieved = dom_flops / dom_step_s / 1e12 if dom_flops else None
    roofline = {"kernel": dom, "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_BF16_TFLOPS if achieved else None, "traffic": traffic,
                "avg_launch_us": 1e3 * per[dom][1] / per[dom][0], "launches_per_step": per[dom][0] // args.steps}

    # the integer-grid pass against HBM: algorithmic bytes of one launch (codes in, q out, A and B,
    # plus the clip mask in the backward's launches), averaged over the step's forward and backward launches
    grid_pass = None
    if "grid" in per:
        def grid_bytes(l, mask):
            L = l["spec"]
            b = l["phi0"].numel() * l["phi0"].element_size() + 4 * (L.out_features + L.in_features) * r
            b += L.out_features * L.in_features // (2 if wl.bits <= 4 else 1)
            return b + (L.out_features * L.in_features // 8 if mask else 0)
        gb = sum(grid_bytes(l, False) + grid_bytes(l, True) for l in layers) / (2 * nl)
        g_us = 1e3 * per["grid"][1] / per["grid"][0]
        grid_pass = {"bound": "hbm", "achieved": gb / (g_us * 1e-6) / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": gb / (g_us * 1e-6) / 1e9 / PEAK_HBM_GBS, "bytes_per_launch": gb, "avg_launch_us": g_us,
                     "traffic": traffic_record("grid") if nl == 1 else None}

    # merge of every layer (W_Z for inference) and a plain device copy, as bandwidth
    merge_bytes = sum(l["phi0"].numel() * l["phi0"].element_size() + 4 * (l["spec"].out_features +
                      l["spec"].in_features) * r + l["spec"].out_features * l["spec"].in_features // 2
                      for l in layers)
    W_int4 = [torch.empty((l["spec"].out_features, l["spec"].in_features // 2), dtype=torch.uint8, device=dev)
              for l in layers]

    def time_merge(Bs):
        """Average time of merging every layer with adapters Bs (HIP-graph replays when the
        step's graph check passed: eager launches of these short kernels measure the host)."""
        def merge_all():
            # on the current stream (the capture stream inside a HIP graph)
            for l, w, b in zip(layers, W_int4, Bs):
                lrqat.lrqat_merge_to_int4(l["spec"], l["phi0"], l["A"], b, out=w)
        for _ in range(3):
            merge_all()
        torch.cuda.synchronize()
        ref_w = [w.clone() for w in W_int4]
        # ten merges per graph, so that the replays' own launch gaps are amortised
        run, how, per_run = merge_all, "eager", 1
        if graph_ok:
            gm = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gm):
                for _ in range(10):
                    merge_all()
            for w in W_int4:
                w.fill_(0)
            gm.replay()
            torch.cuda.synchronize()
            if all(torch.equal(w, r) for w, r in zip(W_int4, ref_w)):
                run, how, per_run = gm.replay, "hip_graph", 10
        for _ in range(2):
            run()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        nrun = 40 // per_run
        e0.record()
        for _ in range(nrun):
            run()
        e1.record()
        torch.cuda.synchronize()
        us = 1e3 * e0.elapsed_time(e1) / (nrun * per_run)
        return {"us": us, "layers": nl, "launch": how, "algorithmic_bytes": merge_bytes,
                "GB/s": merge_bytes / (us * 1e-6) / 1e9, "frac_of_hbm_peak": merge_bytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}

    merge = None
    if wl.bits <= 4:
        merge = time_merge([l["B"] for l in layers])
        # the same merge with adapters as after training: B scaled so that delta has a standard
        # deviation of about a quarter code (about 1% of the codes move), the exact paths engaged
        b_scale = 5000.0
        Bt = [l["B"] * b_scale for l in layers]
        merge["trained_state"] = {"b_scale": b_scale, **time_merge(Bt)}
        del Bt
    del W_int4
    src = torch.empty(256 << 18, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(10):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * src.numel() * 4 * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    if merge:
        merge["device_copy_GB/s"] = copy_gbs
    # device memory the layers hold across forward + backward (checkpointing: nothing saved but the inputs)
    act_b = 2 if wl.act_dtype == "bf16" else 4
    analytic = {"phi0": sum(l["phi0"].numel() * l["phi0"].element_size() for l in layers),
                "s": sum(l["s0"].numel() * 4 for l in layers),
                "A+B": sum(4 * (L.m + L.k) * r for L in wl.layers),
                "X+dY": sum(act_b * T * (L.k + L.m) for L in wl.layers),
                "Y+dX": sum(act_b * T * (L.m + L.k) for L in wl.layers),
                "dA+dB": sum(4 * (L.m + L.k) * r for L in wl.layers),
                "workspace_fwd": ws_f.numel(), "workspace_bwd": ws_b.numel()}
    inp = inp0

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, inp, args.cpu_seconds)

    out = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "clock_settle": settle,
        "vs_baseline": None, "dtype": "bf16" if wl.act_dtype == "bf16" else "fp32", "data": "synthetic",
        "config": {"workload": wl.name, "tokens": T,
                   "layers": [[L.name, L.m, L.k] for L in wl.layers], "rank": r,
                   "alpha": wl.alpha, "bits": wl.bits, "phi_format": wl.phi_format, "group_size": wl.group_size,
                   "act_bits": wl.act_bits, "parallelism": "none"},
        "step_ms_p10_p50_p90": [float(np.percentile(per_step, q)) for q in (10, 50, 90)],
        "launch": "eager",
        "hip_graph": {"note": graph_note, "ms_per_step": ms_graph,
                      "step_ms_p10_p50_p90": [float(np.percentile(per_step_graph, q)) for q in (10, 50, 90)]
                      if per_step_graph is not None else None},
        "pct_of_bf16_peak": 100.0 * value / PEAK_BF16_TFLOPS,
        "tokens_per_s": T / (ms * 1e-3),
        "peak_device_mem_bytes": int(peak_mem_steps),
        "peak_device_mem_bytes_process": int(peak_mem),
        "analytic_mem_bytes": {**analytic, "total": int(sum(analytic.values()))},
        "merge": merge,
        "kernels": kernels,
        "roofline": roofline,
        "grid_pass": grid_pass,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
