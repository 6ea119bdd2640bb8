#!/usr/bin/env python3
"""Throughput of randomized per-sample norm estimation (DP-SGD-RC) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload stack|q_proj|tiny|mlp|decoder]
                    [--probe rademacher|gaussian]

One step is one pass of the workload's hot path over one batch already
resident in HBM: the norm estimates of every layer (Hutchinson, or Hutch++ for
``decoder``) summed per sample, the clip factors, and -- where the workload
has them -- the clipped accumulation of every layer and the Gaussian noise.
The default workload is the whole Llama-3.2-1B linear stack: 16 decoder layers
x 7 projections plus a 2048 -> 128256 lm_head, B=8, T=4096, bf16, k=32
Rademacher probes, clip C=1, clipped accumulation and noise sigma=0.8 (54.7 GB
of inputs).  Inputs are synthetic (seeded); workloads smaller than the 256 MB
Infinity Cache rotate several input copies.

Prints one JSON line.  ``value`` is the norm stage's tokens/s, B*T / t_norm,
with t_norm the wall time of the norm call (every pass, the finishing kernels
and the clip factors) between HIP events on the launch stream, averaged over
the K timed steps; ``ms_per_step`` is the whole step.  ``roofline`` covers the
norm stage's dominant streaming kernel: algorithmic bytes per launch over its
average launch duration, each launch bracketed by HIP events that the dispatch
itself stamps, during the same timed steps.  ``extra.accumulate`` gives the
clipped-accumulation GEMM's matrix-core throughput on the same workload and
steps; ``cpu_baseline`` is the CPU oracle timed on a bounded sample of the
same workload (its norm leg, plus its accumulation-and-noise leg).
"""

import argparse
import ctypes
import json
import math
import os
import sys
import time

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0       # MI355X dense bf16 matrix cores


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="stack")
    ap.add_argument("--probe", default="rademacher", choices=["rademacher", "gaussian"],
                    help="Hutchinson probe family (Gaussian: dense columns, k <= 32)")
    ap.add_argument("--rotate-bytes", type=float, default=1.2e9,
                    help="total bytes of rotated input copies (defeats the 256 MB Infinity Cache)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the context measurements (vendor GEMM and read references)")
    ap.add_argument("--graph", action="store_true",
                    help="replay a captured HIP graph per step instead of launching from the host")
    ap.add_argument("--copy-calibration", type=float, default=0.0, metavar="BYTES",
                    help="only run 5 device copies of BYTES bytes (calibrates FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


class Hip:
    """HIP events through the runtime the process already uses."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def events(self, n):
        arr = (ctypes.c_void_p * n)()
        for j in range(n):
            e = ctypes.c_void_p()
            if self.lib.hipEventCreate(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")
            arr[j] = e
        return arr

    def elapsed_ms(self, a, b):
        self.lib.hipEventSynchronize(b)
        t = ctypes.c_float()
        if self.lib.hipEventElapsedTime(ctypes.byref(t), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(t.value)

    def destroy(self, arr):
        for e in arr:
            self.lib.hipEventDestroy(e)


def make_inputs(cfg, torch, workloads, copies):
    sets = []
    for c in range(copies):
        layers = []
        for li in range(len(cfg["layers"])):
            A, E = workloads.layer_inputs(cfg, li, device="cuda", seed=c)
            layers.append((A, E, li))
        sets.append(layers)
    return sets


def probe_id(D, cfg):
    return D.PROBE_GAUSSIAN if cfg.get("probe") == "gaussian" else D.PROBE_RADEMACHER


def step_fn(cfg, D, torch, ws_norm, grads, ws_acc):
    """One step: the norm stage (with the clip factors), then the clipped accumulation and the
    noise of every layer where the workload has them.  `marks` (two events, may be None) are
    recorded on the launch stream around the norm stage."""
    C = cfg["C"]
    probe = probe_id(D, cfg)

    def step(layers, n2, c, marks=None):
        if marks is not None:
            marks[0].record()
        if cfg["estimator"] == "hutch":       # norms and clip factors in the same launches
            D.dprc_norm_hutch_clip(layers, cfg["k"], 0, C, n2=n2, c=c, ws=ws_norm, probe=probe)
        else:
            D.dprc_norm_hutchpp(layers, cfg["s"], cfg["r"], 0, n2=n2, ws=ws_norm)
            D.dprc_clip_scale(n2, C, c=c)
        if marks is not None:
            marks[1].record()
        if cfg["accumulate"]:
            accumulate_layers(cfg, D, layers, c, grads, ws_acc)
    return step


def accumulate_layers(cfg, D, layers, c, grads, ws_acc):
    """The clipped accumulation of every layer (bf16: one call for all of them, so the small
    layers share launches instead of splitting over tokens), then the noise of each."""
    if cfg["dtype"] == "bf16":
        D.dprc_clip_accumulate_layers(layers, c, grads=grads)
    else:
        for (A, E, li), g in zip(layers, grads):
            D.dprc_clip_accumulate(A, E, c, grad=g, ws=ws_acc)
    if cfg["noise_sigma"] is not None:
        for (A, E, li), g in zip(layers, grads):
            D.dprc_add_noise(g, cfg["noise_sigma"], cfg["C"], 0, li)


class LaunchTrace:
    """While active, every library launch from this thread is bracketed by HIP events that the
    dispatch stamps itself (dprc_trace_launches); records() gives (kind, ms) per launch."""

    def __init__(self, hip, D, capacity):
        self.hip, self.D, self.capacity = hip, D, capacity
        self.events = hip.events(2 * capacity)
        self.kinds = (ctypes.c_int32 * capacity)()
        self.count = ctypes.c_int32(0)

    def __enter__(self):
        self.D.dprc_trace_launches(ctypes.cast(self.events, ctypes.c_void_p), ctypes.cast(self.kinds, ctypes.c_void_p),
                                   self.capacity, ctypes.cast(ctypes.pointer(self.count), ctypes.c_void_p))
        return self

    def __exit__(self, *exc):
        self.D.dprc_trace_launches(None, None, 0, None)
        return False

    def records(self):
        if self.count.value >= self.capacity:
            raise RuntimeError(f"launch trace full ({self.capacity} launches): per-kernel figures would be wrong")
        out = [(self.D.KERNEL_NAMES.get(self.kinds[j], str(self.kinds[j])),
                self.hip.elapsed_ms(self.events[2 * j], self.events[2 * j + 1])) for j in range(self.count.value)]
        self.hip.destroy(self.events)
        return out


def trace_kernels(hip, D, fn, reps, capacity=4096):
    """Run fn() reps times with every library launch bracketed by events; per-kind launch durations."""
    import torch
    events = hip.events(2 * capacity)
    kinds = (ctypes.c_int32 * capacity)()
    count = ctypes.c_int32(0)
    D.dprc_trace_launches(ctypes.cast(events, ctypes.c_void_p), ctypes.cast(kinds, ctypes.c_void_p), capacity,
                          ctypes.cast(ctypes.pointer(count), ctypes.c_void_p))
    try:
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
    finally:
        D.dprc_trace_launches(None, None, 0, None)
    if count.value >= capacity:
        hip.destroy(events)
        raise RuntimeError(f"launch trace full ({capacity} launches): per-kernel figures would be wrong")
    out = []
    for j in range(count.value):
        out.append((D.KERNEL_NAMES.get(kinds[j], str(kinds[j])), hip.elapsed_ms(events[2 * j], events[2 * j + 1])))
    hip.destroy(events)
    return out


def kernel_bytes_per_step(cfg):
    """Algorithmic HBM bytes per step for the streaming kernels (inputs read once per launch)."""
    elem = 4 if cfg["dtype"] == "f32" else 2
    proj = tok = 0
    for (_, d, p) in cfg["layers"]:
        B, T = cfg["B"], cfg["T"]
        m, n = p, d          # sketched side "out"
        if cfg["estimator"] == "hutch":
            proj += B * T * m * elem
            tok += B * T * n * elem
        else:                # three passes; pass 2 swaps the roles
            proj += B * T * (2 * m + n) * elem
            tok += B * T * (2 * n + m) * elem
    return {"project": proj, "token_reduce": tok}


# launch kind -> the kernel families it dispatches (single-layer and batched) and their source
TRAFFIC_KERNELS = {"project": (("project_kernel", "project_batch_kernel"), "paper_2605_24879_amd/csrc/k_project.hip"),
                   "token_reduce": (("tokred_kernel", "tokred_batch_kernel"), "paper_2605_24879_amd/csrc/k_tokred.hip"),
                   "accumulate": (("gemm_kernel", "gemm_batch_kernel"), "paper_2605_24879_amd/csrc/k_gemm.hip")}
# sources every launch's traffic depends on besides its kernel's own file
TRAFFIC_SHARED_SOURCES = ("paper_2605_24879_amd/csrc/device.hpp", "paper_2605_24879_amd/csrc/kernels.hpp",
                          "paper_2605_24879_amd/csrc/api.hip")


def measured_traffic(workload, kernel):
    """HBM bytes per launch (read + write) from the committed rocprofv3 counter summary, or None
    when there is none for this workload or when the kernel's source, the shared device header,
    the launch-side headers or the host code that groups layers into launches changed since the
    counters were taken."""
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(root, "profiles", f"{workload}_hbm_traffic.json")
    if kernel not in TRAFFIC_KERNELS or not os.path.exists(path):
        return None
    keys, src = TRAFFIC_KERNELS[kernel]
    kernels = json.load(open(path)).get("kernels", {})
    recs = [kernels[k] for k in keys if k in kernels]
    if not recs:
        return None
    sha = lambda p: hashlib.sha256(open(os.path.join(root, p), "rb").read()).hexdigest()[:16]
    want = {p: sha(p) for p in (src,) + TRAFFIC_SHARED_SOURCES}
    for rec in recs:
        if rec.get("sources_sha256_16") != want:
            return None
    # per launch, averaged over the dispatches of the kind's kernel families
    n = sum(rec.get("dispatches", 1) for rec in recs)
    return int(sum((rec["read_bytes"] + rec["write_bytes"]) * rec.get("dispatches", 1) for rec in recs) / n)


CPU_MAX_COLS = 1 << 15      # widest operand slice the CPU oracle sample takes (cost is linear in width)


def cpu_baseline(cfg, layers, budget_s):
    """The oracle (fp64 numpy, explicit per-sample gradients G_i = A_i^T E_i) timed on one sample
    of each distinct layer shape of the workload, and scaled to the whole workload by the number
    of (layer, sample) pairs of that shape.  Legs: the norm stage (G_i, then the estimator) and
    the clipped accumulation plus noise (G_i scaled into the layer sum, noise on every element).
    Operands wider than CPU_MAX_COLS columns are cut to that many and the time scaled by the
    width.  Shapes are cycled until the budget is spent (every shape at least once)."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import estimators as est
    B = cfg["B"]
    first = {}
    for (A, E, li) in layers:
        first.setdefault((A.shape[2], E.shape[2]), (A, E, li))
    count = {}
    for (_, d, p) in cfg["layers"]:
        count[(d, p)] = count.get((d, p), 0) + 1
    t_norm = {s: [] for s in first}
    t_acc = {s: [] for s in first}
    t_noise = []
    kind = cfg.get("probe", "rademacher")
    t0 = time.perf_counter()
    while True:
        for (d, p), (A, E, li) in first.items():
            pc = min(p, CPU_MAX_COLS)
            scale = p / pc
            t1 = time.perf_counter()
            Ai = A[0:1].float().cpu().numpy().astype(np.float64)
            Ei = E[0:1, :, :pc].float().cpu().numpy().astype(np.float64)
            if cfg["estimator"] == "hutch":
                est.hutch_layer(Ai, Ei, cfg["k"], 0, li, probe=kind)
            else:
                est.hutchpp_layer(Ai, Ei, cfg["s"], cfg["r"], 0, li)
            t2 = time.perf_counter()
            if cfg["accumulate"]:
                est.clip_accumulate(Ai, Ei, np.array([0.5]))
            t3 = time.perf_counter()
            t_norm[(d, p)].append((t2 - t1) * scale)
            t_acc[(d, p)].append((t3 - t2) * scale)
        if cfg["noise_sigma"] is not None:
            n = 1 << 22
            t1 = time.perf_counter()
            est.add_noise(np.zeros(n), cfg["noise_sigma"], cfg["C"], 0, 0)
            t_noise.append((time.perf_counter() - t1) / n)
        if time.perf_counter() - t0 > budget_s:
            break
    wall = time.perf_counter() - t0
    mean = lambda v: sum(v) / len(v)
    norm_s = sum(count[s] * B * mean(t_norm[s]) for s in first)
    noise_s = sum(count[(d, p)] * d * p for (d, p) in first) * mean(t_noise) if t_noise else 0.0
    acc_s = sum(count[s] * B * mean(t_acc[s]) for s in first) + noise_s if cfg["accumulate"] else None
    info = threadpool_info()
    threads = max([x.get("num_threads", 1) for x in info] or [1])
    blas = ",".join(sorted(set(f"{x.get('internal_api', '?')}" for x in info))) or "unknown"
    shapes = ", ".join(f"{d}x{p}" + (f" (first {CPU_MAX_COLS} cols, x{p / CPU_MAX_COLS:.2f})" if p > CPU_MAX_COLS else "")
                       + f" x{len(t_norm[(d, p)])}" for (d, p) in first)
    out = {"value": B * cfg["T"] / norm_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "sample": f"fp64 oracle on one sample of each distinct layer shape ({shapes} passes), scaled by the "
                     f"workload's {sum(count.values())} layers x B={B} samples; {wall:.1f} s of CPU work; "
                     f"blas={blas}, os.cpu_count={os.cpu_count()}, affinity={len(os.sched_getaffinity(0))}",
           "norm_s_per_step": round(norm_s, 3)}
    if acc_s is not None:
        out["accumulate_noise_s_per_step"] = round(acc_s, 3)
        out["accumulate_noise_note"] = ("explicit G_i scaled into the layer sum for every (layer, sample) pair, "
                                        "plus Box-Muller noise per element (timed on 4M elements)"
                                        if noise_s else "explicit G_i scaled into the layer sum")
    return out


def accumulate_roofline(cfg, per_kind, steps):
    """The clipped-accumulation GEMM of the timed steps against the bf16 matrix-core peak."""
    tot_ms, cnt = per_kind.get("accumulate", (0.0, 0))
    if not cnt:
        return None
    flops = workloads_accumulate_flops(cfg)
    tf = flops * steps / (tot_ms * 1e-3) / 1e12
    red_ms = per_kind.get("splitk_reduce", (0.0, 0))[0]
    return {"kernel": "accumulate", "bound": "mfma", "achieved": round(tf, 1), "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(tf / BF16_PEAK_TFLOPS, 4), "launches_per_step": cnt / steps,
            "avg_launch_us": round(tot_ms / cnt * 1e3, 2), "flops_per_step": flops,
            "gemm_ms_per_step": round(tot_ms / steps, 3), "splitk_reduce_ms_per_step": round(red_ms / steps, 3),
            "with_splitk_reduce_frac": round(flops * steps / ((tot_ms + red_ms) * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)}


def workloads_accumulate_flops(cfg):
    return sum(2 * cfg["B"] * cfg["T"] * d * p for (_, d, p) in cfg["layers"])


def vendor_gemm(torch, A, E, steps):
    """Context only: the vendor bf16 GEMM (hipBLASLt through torch) on one layer's operands in the
    accumulation's layout (both token-major, A^T E over B*T tokens), without per-sample factors."""
    A2 = A.reshape(-1, A.shape[2])
    E2 = E.reshape(-1, E.shape[2])
    for _ in range(2):
        A2.t() @ E2
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        A2.t() @ E2
    ev1.record()
    torch.cuda.synchronize()
    flops = 2.0 * A2.shape[0] * A2.shape[1] * E2.shape[1]
    return round(flops / (ev0.elapsed_time(ev1) / steps * 1e-3) / 1e12, 1)


def read_reference(torch, sets, copies, steps):
    """Context only: torch's own reduction reading the first layer's E (the operand the
    projection streams) of each rotated input copy in turn, one launch per copy, back to back."""
    Es = [layers[0][1] for layers in sets]
    for e in Es[:3]:
        torch.sum(e, dtype=torch.float32)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for k in range(steps):
        torch.sum(Es[k % copies], dtype=torch.float32)
    ev1.record()
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) / steps * 1e3
    nbytes = Es[0].numel() * Es[0].element_size()
    return {"op": "torch.sum (fp32 accumulation) of E, rotated input copies", "bytes": nbytes,
            "avg_us": round(us, 2), "GB/s": round(nbytes / (us * 1e-6) / 1e9, 1)}


NORM_KINDS = ("project", "token_reduce", "token_splits", "sample_sum", "qr", "qr_combine", "qr_expand",
              "hutchpp_final", "hutchpp_sum", "project_f32", "token_reduce_f32", "sample_sq", "probe_bits",
              "probe_gauss", "clip_scale")


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (this library has no "
              f"multi-GPU path).", file=sys.stderr)
        sys.exit(2)
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import torch
    import workloads
    from paper_2605_24879_amd import dprc as D
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration > 0:
        n = int(args.copy_calibration) // 16 * 16
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "copies": 5}))
        return
    D.lib()
    if args.workload == "llama_step":
        return run_llama_step(args, torch, D)
    if args.workload == "accountant":
        return run_accountant(args, torch, D)
    cfg = dict(workloads.BY_NAME[args.workload])
    if args.probe != "rademacher":
        if cfg["estimator"] != "hutch":
            sys.exit(f"--probe {args.probe} applies to Hutchinson workloads only")
        cfg["probe"] = args.probe
    B, T = cfg["B"], cfg["T"]
    elem = 4 if cfg["dtype"] == "f32" else 2
    in_bytes = sum(B * T * (d + p) * elem for (_, d, p) in cfg["layers"])
    copies = max(1, min(32, math.ceil(args.rotate_bytes / in_bytes))) if in_bytes < 256e6 else 1
    print(f"[bench] workload={cfg['name']} layers={len(cfg['layers'])} input={in_bytes/1e9:.3f} GB "
          f"copies={copies}: drawing inputs", file=sys.stderr, flush=True)
    sets = make_inputs(cfg, torch, workloads, copies)
    pairs0 = sets[0]
    if cfg["estimator"] == "hutch":
        ws_n = torch.empty(max(1, D.dprc_norm_hutch_workspace(pairs0, cfg["k"], probe=probe_id(D, cfg))),
                           dtype=torch.uint8, device="cuda")
    else:
        ws_n = torch.empty(max(1, D.dprc_norm_hutchpp_workspace(pairs0, cfg["s"], cfg["r"])), dtype=torch.uint8,
                           device="cuda")
    grads = [torch.empty(d, p, device="cuda") for (_, d, p) in cfg["layers"]] if cfg["accumulate"] else []
    n2 = torch.zeros(B, device="cuda")
    c = torch.zeros(B, device="cuda")
    ws_acc = None
    if cfg["accumulate"]:
        need = max(D.dprc_clip_accumulate_workspace(A, E) for (A, E, _) in pairs0)
        ws_acc = torch.empty(max(1, need), dtype=torch.uint8, device="cuda")
    step = step_fn(cfg, D, torch, ws_n, grads, ws_acc)
    torch.cuda.synchronize()
    print("[bench] inputs resident; warming up", file=sys.stderr, flush=True)

    for w in range(max(args.warmup, 1)):
        step(sets[w % copies], n2, c)
    torch.cuda.synchronize()
    Ev = lambda: torch.cuda.Event(enable_timing=True)
    graphs = None
    if args.graph:
        # per input copy: one captured graph for the norm stage and one for the rest of the step,
        # so that events between the replays bracket the norm stage
        graphs = []
        for ci in range(copies):
            gn, gr = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
            with torch.cuda.graph(gn):
                step_norm_only(cfg, D, sets[ci], n2, c, ws_n)
            with torch.cuda.graph(gr):
                step_rest_only(cfg, D, sets[ci], c, grads, ws_acc)
            graphs.append((gn, gr))
        for w in range(args.warmup):
            graphs[w % copies][0].replay()
            graphs[w % copies][1].replay()
        torch.cuda.synchronize()

    # launches per step, to size the per-launch trace of the timed steps
    hip = Hip()
    probe_trace = LaunchTrace(hip, D, 1 << 15)
    with probe_trace:
        step(sets[0], n2, c)
    torch.cuda.synchronize()
    per_step = len(probe_trace.records())

    # the timed steps: a whole-step bracket, the norm stage bracketed per step, and every
    # library launch bracketed by the events its dispatch stamps (graph replays are not traced)
    marks = [(Ev(), Ev()) for _ in range(args.steps)]
    t_start, t_end = Ev(), Ev()
    trace = LaunchTrace(hip, D, per_step * args.steps + 16)
    with trace:
        t_start.record()
        for s_ in range(args.steps):
            if graphs is None:
                step(sets[s_ % copies], n2, c, marks[s_])
            else:
                marks[s_][0].record()
                graphs[s_ % copies][0].replay()
                marks[s_][1].record()
                graphs[s_ % copies][1].replay()
        t_end.record()
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_end) / args.steps
    norm_ms = sum(a.elapsed_time(b) for (a, b) in marks) / args.steps
    print(f"[bench] timed {args.steps} steps ({'graph replay' if args.graph else 'eager'}): "
          f"{ms_per_step:.3f} ms/step, norm stage {norm_ms:.3f} ms", file=sys.stderr, flush=True)
    recs = trace.records()

    # context only: the same steps on one input copy, which the 256 MB Infinity Cache may hold
    hot_norm_ms = None
    if copies > 1:
        for _ in range(3):
            step(sets[0], n2, c)
        hm = [(Ev(), Ev()) for _ in range(args.steps)]
        for s_ in range(args.steps):
            step(sets[0], n2, c, hm[s_])
        torch.cuda.synchronize()
        hot_norm_ms = sum(a.elapsed_time(b) for (a, b) in hm) / args.steps

    per_kind = {}
    for k, ms in recs:
        tot, cnt = per_kind.get(k, (0.0, 0))
        per_kind[k] = (tot + ms, cnt + 1)
    kb = kernel_bytes_per_step(cfg)
    streaming = [k for k in kb if k in per_kind]
    dom = max(streaming, key=lambda k: per_kind[k][0]) if streaming else None

    def stream_roof(kind):
        tot_ms, cnt = per_kind[kind]
        achieved = kb[kind] * args.steps / (tot_ms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic(cfg["name"] + ("_gaussian" if cfg.get("probe") == "gaussian" else ""), kind),
                "kernel": kind, "bytes_per_launch": int(kb[kind] / (cnt / args.steps)),
                "avg_launch_us": round(tot_ms / cnt * 1e3, 2), "launches_per_step": cnt / args.steps}

    roof = stream_roof(dom) if dom else {"bound": "hbm", "achieved": None, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                         "frac": None, "traffic": None, "kernel": None}
    norm_bytes = workloads.algorithmic_norm_bytes(cfg)
    kernels = {k: {"launches_per_step": v[1] / args.steps, "avg_launch_us": round(v[0] / v[1] * 1e3, 2),
                   "us_per_step": round(v[0] / args.steps * 1e3, 2)} for k, v in sorted(per_kind.items())}
    norm_kernel_ms = sum(per_kind.get(k, (0.0, 0))[0] for k in NORM_KINDS) / args.steps
    extra = {"norm_stage": {"ms": round(norm_ms, 4), "algorithmic_bytes": norm_bytes,
                            "GB/s": round(norm_bytes / (norm_ms * 1e-3) / 1e9, 1),
                            "frac_of_hbm_peak": round(norm_bytes / (norm_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                            "kernel_ms_summed": round(norm_kernel_ms, 4)},
             "whole_step": {"ms": round(ms_per_step, 4), "tokens_per_s": round(B * T / (ms_per_step * 1e-3), 1),
                            "parts": step_parts(cfg)},
             "streaming_kernels": {k: stream_roof(k) for k in streaming},
             "kernels": kernels, "input_copies_rotated": copies,
             "hot_cache_norm_tokens_per_s": round(B * T / (hot_norm_ms * 1e-3), 1) if hot_norm_ms else None}
    acc = accumulate_roofline(cfg, per_kind, args.steps)
    if acc is not None:
        acc["traffic"] = measured_traffic(cfg["name"], "accumulate")
        extra["accumulate"] = acc
    if not args.no_extra:
        if cfg["accumulate"] and cfg["dtype"] == "bf16":
            A, E, _ = max(pairs0, key=lambda t: t[0].shape[2] * t[1].shape[2] if t[1].shape[2] <= 8192 else 0)
            extra["accumulate"]["vendor_gemm_tflops_context"] = {
                "layer": f"{A.shape[2]}x{E.shape[2]}", "tflops": vendor_gemm(torch, A, E, 5)}
        if len(cfg["layers"]) == 1 and copies > 1:
            extra["vendor_read_same_operand"] = read_reference(torch, sets, copies, args.steps)
    rec = {"metric": "per-sample norm-estimation tokens/s + HBM GB/s (% peak), Llama-3.2-1B shapes",
           "value": round(B * T / (norm_ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg["dtype"],
           "data": "synthetic (seeded; Llama-3.2-1B layer shapes)",
           "config": workloads.describe(cfg) | {"C": cfg["C"], "steps_include": step_parts(cfg),
                                                "value_is": "B*T / norm-stage wall time",
                                                "launch": "hip_graph_replay" if args.graph else "eager"},
           "roofline": roof, "extra": extra}
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(cfg, pairs0, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


def step_norm_only(cfg, D, layers, n2, c, ws_n):
    if cfg["estimator"] == "hutch":
        probe = D.PROBE_GAUSSIAN if cfg.get("probe") == "gaussian" else D.PROBE_RADEMACHER
        D.dprc_norm_hutch_clip(layers, cfg["k"], 0, cfg["C"], n2=n2, c=c, ws=ws_n, probe=probe)
    else:
        D.dprc_norm_hutchpp(layers, cfg["s"], cfg["r"], 0, n2=n2, ws=ws_n)
        D.dprc_clip_scale(n2, cfg["C"], c=c)


def step_rest_only(cfg, D, layers, c, grads, ws_acc):
    if cfg["accumulate"]:
        accumulate_layers(cfg, D, layers, c, grads, ws_acc)


LLAMA_STEP = dict(B=2, T=2048, k=16, C=1.0, sigma=0.8, lr=1e-4)


def run_llama_step(args, torch, D):
    """The whole DP-SGD-RC training step on the Llama-3.2-1B-shaped stack (16 blocks, untied
    lm_head, random weights, synthetic tokens): forward, capture of every linear layer's (A, E),
    norms, clip factors, clipped gradients, noise and AdamW.  Context lines: a plain non-private
    step (loss.backward-style weight gradients + AdamW) and the same private step with the
    algorithm's second backward pass instead of the direct clipped GEMM."""
    from paper_2605_24879_amd import dpsgd
    from workloads import llama
    cfg = LLAMA_STEP
    B, T, k, C, sigma = cfg["B"], cfg["T"], cfg["k"], cfg["C"], cfg["sigma"]
    steps, warmup = min(args.steps, 10), max(1, min(args.warmup, 3))
    print(f"[bench] workload=llama_step B={B} T={T}: building the model", file=sys.stderr, flush=True)
    model = llama.build(seed=0, device="cuda")
    tok = llama.tokens(B, T, llama.LLAMA_3_2_1B["vocab"], device="cuda")
    drv = dpsgd.DPSGDRC(model.linears(), C=C, sigma=sigma, k=k, lr=cfg["lr"])
    loss_fn = lambda: llama.per_sample_loss(model(tok[:, :-1]), tok[:, 1:])
    layer_shapes = [(lin.in_features, lin.out_features) for lin in drv.linears]
    Ev = lambda: torch.cuda.Event(enable_timing=True)

    def private_step(ev=None):
        mark = (lambda j: ev[j].record()) if ev else (lambda j: None)
        mark(0)
        losses, pairs = drv.capture(loss_fn)
        mark(1)
        key = dpsgd.step_seed(0, drv.steps)
        n2, c = D.dprc_norm_hutch_clip(pairs, k, key, C)
        mark(2)
        grads = drv.clipped_sums(pairs, c)
        mark(3)
        del pairs
        drv.update(grads, B, key)            # noise + 1/B + AdamW + bf16 weights, one pass per layer
        mark(4)

    need = max(D.dprc_clip_accumulate_workspace(torch.empty(B, T, d, dtype=torch.bfloat16, device="cuda"),
                                                torch.empty(B, T, p, dtype=torch.bfloat16, device="cuda"))
               for (d, p) in set(layer_shapes))
    drv._ws_acc = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
    for _ in range(warmup):
        private_step()
    torch.cuda.synchronize()
    print(f"[bench] llama_step: warm, timing {steps} steps", file=sys.stderr, flush=True)
    stage = [0.0] * 4
    t0, t1 = Ev(), Ev()
    t0.record()
    evs = []
    for _ in range(steps):
        ev = [Ev() for _ in range(5)]
        private_step(ev)
        evs.append(ev)
    t1.record()
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / steps
    for ev in evs:
        for j in range(4):
            stage[j] += ev[j].elapsed_time(ev[j + 1]) / steps
    print(f"[bench] llama_step: {ms_per_step:.2f} ms/step", file=sys.stderr, flush=True)

    # library kernels of one step, each launch timed with HIP events on its stream
    hip = Hip()
    recs = trace_kernels(hip, D, lambda: private_step(), 1, capacity=2048)
    per_kind = {}
    for name, ms in recs:
        t, n = per_kind.get(name, (0.0, 0))
        per_kind[name] = (t + ms, n + 1)
    acc_ms, acc_n = per_kind.get("accumulate", (0.0, 0))
    flops = sum(2 * B * T * d * p for (d, p) in layer_shapes)
    acc_tf = flops / (acc_ms * 1e-3) / 1e12 if acc_ms else None
    roof = {"bound": "mfma", "achieved": round(acc_tf, 1) if acc_tf else None, "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(acc_tf / BF16_PEAK_TFLOPS, 4) if acc_tf else None, "traffic": None,
            "kernel": "accumulate", "flops_per_step": int(flops), "launches_per_step": acc_n,
            "avg_launch_us": round(acc_ms / max(acc_n, 1) * 1e3, 2)}
    kernels = {kk: {"launches_per_step": v[1], "us_per_step": round(v[0] * 1e3, 1)} for kk, v in sorted(per_kind.items())}

    extra = {"stages_ms": {"forward_and_capture": round(stage[0], 3), "norms_and_clip": round(stage[1], 3),
                           "clipped_gemm": round(stage[2], 3), "noise_and_adamw_fused": round(stage[3], 3)},
             "library_kernels": kernels}
    if not args.no_extra:
        extra.update(llama_context_steps(torch, D, dpsgd, drv, loss_fn, model, B, T, k, C, sigma, steps))
    rec = {"metric": "DP-SGD-RC training-step tokens/s, Llama-3.2-1B-shaped stack",
           "value": round(B * T / (ms_per_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": steps, "warmup": warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded tokens; random-init Llama-3.2-1B-shaped weights)",
           "config": {"workload": "llama_step", "B": B, "T": T, "blocks": 16, "hidden": 2048, "mlp": 8192,
                      "heads": "32q/8kv", "vocab": 128256, "trained": "all 113 linear layers",
                      "estimator": "hutch", "probes": k, "C": C, "sigma": sigma, "optimizer": "AdamW",
                      "steps_include": ["forward", "capture E (autograd to layer outputs)", "norm-hutch",
                                        "clip_scale", "clip_accumulate", "private_adamw (noise + AdamW)"]},
           "roofline": roof, "extra": extra}
    print(json.dumps(rec), flush=True)


def run_accountant(args, torch, D):
    """Privacy accounting for Hutchinson with k = 32 probes: MiddleRegionCDF (all two-level forms
    of a d-dimensional envelope, 51 lambda values, on the GPU) at growing d, the x_+ search at
    d = 128, and eps / sigma solves with the envelope; the oracle's brute force timed beside it."""
    from paper_2605_24879_amd import accountant as A
    k, nl = 32, 51
    ev = lambda: torch.cuda.Event(enable_timing=True)
    rows = {}
    for d in (64, 256, 1024):
        x = torch.tensor([1.0 + 1.0 / (d * k)], dtype=torch.float64, device="cuda")
        D.dprc_envelope_middle(x, k, d, nl)
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record()
        D.dprc_envelope_middle(x, k, d, nl)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b)
        ncand = d * (d - 1) // 2 * nl
        rows[f"d={d}"] = {"candidates": ncand, "ms": round(ms, 3), "candidates_per_s": round(ncand / (ms * 1e-3), 1),
                          "quadrature_nodes_per_s": round(ncand * 256 / (ms * 1e-3), 1)}
        print(f"[bench] accountant: MiddleRegionCDF d={d}: {ms:.2f} ms", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    xp = A.x_plus(k, 128, tol=1e-7, n_lambda=nl)
    xp_s = time.perf_counter() - t0
    t0 = time.perf_counter()
    env = A.envelope_law(k, 128, n_bins=4000, n_lambda=nl)
    env_s = time.perf_counter() - t0
    t0 = time.perf_counter()
    eps_rc = A.epsilon(1.0, 10000, 256, 3, 1e-5, envelope=env)
    eps_s = time.perf_counter() - t0
    eps_dp = A.epsilon(1.0, 10000, 256, 3, 1e-5)
    t0 = time.perf_counter()
    sig_rc = A.noise_multiplier(2.0, 10000, 256, 3, 1e-5, envelope=env, tol=1e-3)
    sig_s = time.perf_counter() - t0
    sig_dp = A.noise_multiplier(2.0, 10000, 256, 3, 1e-5, tol=1e-3)
    # the oracle's brute force (scipy quadrature per form) on a bounded sample
    from oracle import accountant as ac
    t0 = time.perf_counter()
    n = 0
    while time.perf_counter() - t0 < args.cpu_seconds / 4:
        ac.middle_region(1.0 + 1.0 / (8 * k), k, 8, 11)
        n += 8 * 7 // 2 * 11
    cpu_rate = n / (time.perf_counter() - t0)
    big = rows["d=1024"]
    rec = {"metric": "MiddleRegionCDF two-level forms evaluated per second (envelope CDF, k=32)",
           "value": big["candidates_per_s"], "unit": "forms/s", "n_gpus": 1, "steps": 1, "warmup": 1,
           "ms_per_step": big["ms"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "f64", "data": "none (closed-form distributions)",
           "config": {"workload": "accountant", "k": k, "n_lambda": nl, "quadrature": "16 panels x 16 nodes"},
           "roofline": {"bound": "alu", "achieved": None, "peak": 78.6, "unit": "TFLOP/s", "frac": None,
                        "traffic": None, "kernel": "envelope",
                        "note": "fp64 series / continued fractions of the incomplete gamma per node"},
           "extra": {"middle_region": rows, "x_plus_d128_s": round(xp_s, 2), "x_plus_d128": xp,
                     "x_plus_asymptotic": 1 + 2 / (128 * k), "envelope_law_d128_s": round(env_s, 2),
                     "epsilon_s": round(eps_s, 3),
                     "eps_sigma1_N10000_B256_E3_delta1e-5": {"randomized_clipping": eps_rc, "dp_sgd": eps_dp},
                     "sigma_for_eps2": {"randomized_clipping": sig_rc, "dp_sgd": sig_dp, "solve_s": round(sig_s, 2)}},
           "cpu_baseline": {"value": round(cpu_rate, 1), "unit": "forms/s", "cores": 1, "kind": "oracle",
                            "sample": f"{n} two-level forms (d=8, k=32, 11 lambdas) by scipy quadrature"}}
    print(json.dumps(rec), flush=True)


def llama_context_steps(torch, D, dpsgd, drv, loss_fn, model, B, T, k, C, sigma, steps):
    """Times of a plain non-private step and of the private step with the second backward pass."""
    weights = [lin.weight for lin in drv.linears]
    masters = [w.detach().t().float().contiguous() for w in weights]
    opt = torch.optim.AdamW(masters, lr=1e-4)

    def plain():
        gw = torch.autograd.grad(loss_fn().mean(), weights)
        for m, g in zip(masters, gw):
            m.grad = g.t().float().contiguous()
        opt.step()
        opt.zero_grad(set_to_none=True)

    def second_backward():
        drv.remove_hooks()
        hooks = [lin.register_forward_hook(drv._tap(j)) for j, lin in enumerate(drv.linears)]
        losses = loss_fn()
        E = torch.autograd.grad(losses.sum(), drv._S, retain_graph=True)
        pairs = [(dpsgd._rows(drv._A[j].detach()), dpsgd._rows(E[j]), j) for j in range(len(weights))]
        drv._A = [None] * len(weights)
        drv._S = [None] * len(weights)
        for h in hooks:
            h.remove()
        key = dpsgd.step_seed(0, drv.steps)
        n2 = D.dprc_norm_hutch(pairs, k, key)
        c = D.dprc_clip_scale(n2, C)
        del pairs, E
        gw = torch.autograd.grad((losses * c).sum(), weights)
        for j, (m, g) in enumerate(zip(masters, gw)):
            gt = g.t().float().contiguous()
            D.dprc_add_noise(gt, sigma, C, key, j)
            m.grad = gt.div_(B)
        opt.step()
        opt.zero_grad(set_to_none=True)

    def unfused():
        losses, pairs = drv.capture(loss_fn)
        key = dpsgd.step_seed(0, drv.steps)
        n2 = D.dprc_norm_hutch(pairs, k, key)
        c = D.dprc_clip_scale(n2, C)
        for (A, E, j), m, g in zip(pairs, masters, drv.clipped_sums(pairs, c)):
            D.dprc_add_noise(g, sigma, C, key, j)
            m.grad = g.div_(B)
        del pairs
        opt.step()
        opt.zero_grad(set_to_none=True)
        with torch.no_grad():
            for lin, m in zip(drv.linears, masters):
                lin.weight.copy_(m.t())

    out = {}
    for name, fn in (("plain_nonprivate_step_ms", plain), ("private_step_torch_adamw_ms", unfused),
                     ("second_backward_private_step_ms", second_backward)):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n = max(2, steps // 2)
        a.record()
        for _ in range(n):
            fn()
        b.record()
        torch.cuda.synchronize()
        out[name] = round(a.elapsed_time(b) / n, 3)
    return out


def step_parts(cfg):
    parts = ["norm-" + cfg["estimator"], "clip_scale"]
    if cfg["accumulate"]:
        parts.append("clip_accumulate")
    if cfg["noise_sigma"] is not None:
        parts.append("add_noise")
    return parts


if __name__ == "__main__":
    main()
