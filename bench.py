#!/usr/bin/env python3
"""Throughput of randomized per-sample norm estimation (DP-SGD-RC) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload q_proj|tiny|mlp|decoder|stack]
                    [--probe rademacher|gaussian]

One step is one pass of the workload's hot path over one batch already
resident in HBM: the norm estimates of every layer (Hutchinson, or Hutch++ for
``decoder``) summed per sample, the clip factors, and -- where the workload
has them -- the clipped accumulation of every layer and the Gaussian noise.
The default workload is one Llama-3.2-1B q_proj-shaped layer (B=4, T=2048,
d=p=2048, bf16, k=16 Rademacher probes, clip C=1).  Inputs are synthetic
(seeded) and several copies are rotated so that the 256 MB Infinity Cache
does not serve a step from a previous step's reads.

Prints one JSON line.  ``roofline`` covers the kernel that takes the most time
in the step, timed with HIP events around each launch on the launch stream;
``extra.accumulate`` times the clipped-accumulation GEMM on an mlp-shaped
layer against the bf16 matrix-core peak; ``cpu_baseline`` is the CPU oracle
timed on a bounded sample of the same workload.
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
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="q_proj")
    ap.add_argument("--probe", default="rademacher", choices=["rademacher", "gaussian"],
                    help="Hutchinson probe family (Gaussian: dense columns, k <= 32)")
    ap.add_argument("--rotate-bytes", type=float, default=1.2e9,
                    help="total bytes of rotated input copies (defeats the 256 MB Infinity Cache)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="skip the accumulation-GEMM measurement")
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
    C = cfg["C"]
    probe = probe_id(D, cfg)

    def step(layers, n2, c):
        if cfg["estimator"] == "hutch":       # norms and clip factors in the same launches
            D.dprc_norm_hutch_clip(layers, cfg["k"], 0, C, n2=n2, c=c, ws=ws_norm, probe=probe)
        else:
            D.dprc_norm_hutchpp(layers, cfg["s"], cfg["r"], 0, n2=n2, ws=ws_norm)
            D.dprc_clip_scale(n2, C, c=c)
        if cfg["accumulate"]:
            for (A, E, li), g in zip(layers, grads):
                D.dprc_clip_accumulate(A, E, c, grad=g, ws=ws_acc)
                if cfg["noise_sigma"] is not None:
                    D.dprc_add_noise(g, cfg["noise_sigma"], C, 0, li)
    return step


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
                   "accumulate": (("gemm_kernel",), "paper_2605_24879_amd/csrc/k_gemm.hip")}


def measured_traffic(workload, kernel):
    """HBM bytes per launch (read + write) from the committed rocprofv3 counter summary, or None
    when there is none for this workload or the kernel source changed since it was taken."""
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
    for rec in recs:
        if rec.get("source_sha256_16") != sha(src) or \
                rec.get("device_hpp_sha256_16") != sha("paper_2605_24879_amd/csrc/device.hpp"):
            return None
    # per launch, averaged over the dispatches of the kind's kernel families
    n = sum(rec.get("dispatches", 1) for rec in recs)
    return int(sum((rec["read_bytes"] + rec["write_bytes"]) * rec.get("dispatches", 1) for rec in recs) / n)


def cpu_baseline(cfg, sets, budget_s):
    """The oracle (fp64 numpy, explicit per-sample gradients) on a bounded sample of the workload."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import estimators as est
    from oracle import philox
    layers = sets[0]
    B, T = cfg["B"], cfg["T"]
    done_tokens = 0
    pairs = []
    t0 = time.perf_counter()
    # (layer, sample) pairs in order, cycled until the budget is spent (small workloads finish a
    # pass in well under a second)
    while time.perf_counter() - t0 <= budget_s:
        for (A, E, li) in layers:
            _, d, p = cfg["layers"][li]
            for i in range(B):
                Ai = A[i].float().cpu().numpy().astype(np.float64)
                Ei = E[i].float().cpu().numpy().astype(np.float64)
                if cfg["estimator"] == "hutch":
                    kind = cfg.get("probe", "rademacher")
                    Z = est.probe_matrix(kind, 0, li, 0, p, cfg["k"])
                    est.hutch_layer(Ai[None], Ei[None], cfg["k"], 0, li, probe=kind, Z=Z)
                else:
                    est.hutchpp_layer(Ai[None], Ei[None], cfg["s"], cfg["r"], 0, li)
                done_tokens += T
                pairs.append(f"{cfg['layers'][li][0]}[{i}]")
                if time.perf_counter() - t0 > budget_s:
                    break
            if time.perf_counter() - t0 > budget_s:
                break
    dt = time.perf_counter() - t0
    info = threadpool_info()
    threads = max([x.get("num_threads", 1) for x in info] or [1])
    # the oracle's norm stage over all layers: tokens/s per layer-sample pass, scaled to whole-step tokens
    layer_tokens = B * T * len(cfg["layers"])
    return {"value": done_tokens / dt * (B * T) / layer_tokens, "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"fp64 explicit per-sample gradients + Hutchinson for {len(pairs)} (layer, sample) pair "
                      f"evaluations ({', '.join(pairs[:6])}{'...' if len(pairs) > 6 else ''}; pairs cycled in "
                      f"order until the budget was spent) in {dt:.1f} s; "
                      f"blas={','.join(sorted(set(x.get('internal_api', '?') for x in info))) or 'unknown'}, "
                      f"os.cpu_count={os.cpu_count()}, affinity={len(os.sched_getaffinity(0))}"}


def accumulate_extra(D, torch, workloads, hip, steps):
    """Clipped accumulation GEMM on one mlp gate layer (d=2048, p=8192, B=2, T=8192)."""
    cfg = workloads.BY_NAME["mlp"]
    A, E = workloads.layer_inputs(cfg, 0, device="cuda")
    c = torch.tensor([0.37, 0.81], device="cuda")
    g = torch.empty(A.shape[2], E.shape[2], device="cuda")
    for _ in range(3):
        D.dprc_clip_accumulate(A, E, c, grad=g)
    recs = trace_kernels(hip, D, lambda: D.dprc_clip_accumulate(A, E, c, grad=g), steps)
    t = [ms for (k, ms) in recs if k == "accumulate"]
    avg_ms = sum(t) / len(t)
    flops = 2.0 * cfg["B"] * cfg["T"] * A.shape[2] * E.shape[2]
    tf = flops / (avg_ms * 1e-3) / 1e12
    # context only: the vendor bf16 GEMM (hipBLASLt through torch) on the same operands and layout
    # (both token-major, A^T E over B*T tokens), without the per-sample factors
    A2 = A.reshape(-1, A.shape[2])
    E2 = E.reshape(-1, E.shape[2])
    for _ in range(3):
        A2.t() @ E2
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        A2.t() @ E2
    ev1.record()
    torch.cuda.synchronize()
    vendor_tf = flops / (ev0.elapsed_time(ev1) / steps * 1e-3) / 1e12
    return {"workload": "mlp.gate B=2 T=8192 d=2048 p=8192", "kernel": "accumulate",
            "bound": "mfma", "achieved": round(tf, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": round(tf / BF16_PEAK_TFLOPS, 4), "avg_launch_us": round(avg_ms * 1e3, 2),
            "flops_per_launch": flops, "vendor_gemm_tflops_same_shape": round(vendor_tf, 1)}


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
          f"copies={copies}", file=sys.stderr, flush=True)
    sets = make_inputs(cfg, torch, workloads, copies)
    pairs0 = sets[0]
    if cfg["estimator"] == "hutch":
        ws_n = torch.empty(max(1, D.dprc_norm_hutch_workspace(pairs0, cfg["k"], probe=probe_id(D, cfg))), dtype=torch.uint8, device="cuda")
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

    for w in range(max(args.warmup, 1)):
        step(sets[w % copies], n2, c)
    torch.cuda.synchronize()
    run = lambda s: step(sets[s % copies], n2, c)
    if args.graph:
        # one captured graph per input copy; the library enqueues on torch's capture stream
        graphs = []
        for ci in range(copies):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                step(sets[ci], n2, c)
            graphs.append(gr)
        for w in range(args.warmup):
            graphs[w % copies].replay()
        torch.cuda.synchronize()
        run = lambda s: graphs[s % copies].replay()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record()
    for s in range(args.steps):
        run(s)
    t_end.record()
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_end) / args.steps
    print(f"[bench] timed {args.steps} steps ({'graph replay' if args.graph else 'eager'}): "
          f"{ms_per_step*1e3:.2f} us/step", file=sys.stderr, flush=True)
    # context only: the same steps on one input copy, which the 256 MB Infinity Cache may hold
    hot_ms = None
    if copies > 1:
        for _ in range(3):
            step(sets[0], n2, c)
        t_start.record()
        for _ in range(args.steps):
            step(sets[0], n2, c)
        t_end.record()
        torch.cuda.synchronize()
        hot_ms = t_start.elapsed_time(t_end) / args.steps

    # per-kernel durations over the same number of steps, with the launch hook on
    hip = Hip()
    it = iter(range(10 ** 9))
    # one traced step sizes the trace (the stack workload launches several hundred kernels per step)
    per_step = len(trace_kernels(hip, D, lambda: step(sets[0], n2, c), 1, capacity=1 << 14))
    recs = trace_kernels(hip, D, lambda: step(sets[next(it) % copies], n2, c), args.steps,
                         capacity=per_step * args.steps + 16)
    per_kind = {}
    for k, ms in recs:
        tot, cnt = per_kind.get(k, (0.0, 0))
        per_kind[k] = (tot + ms, cnt + 1)
    dom = max(per_kind, key=lambda k: per_kind[k][0])
    kb = kernel_bytes_per_step(cfg)
    tot_ms, cnt = per_kind[dom]
    launches_per_step = cnt / args.steps
    if dom in kb:
        bytes_per_launch = kb[dom] / launches_per_step
        achieved = kb[dom] * args.steps / (tot_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": measured_traffic(cfg["name"] + ("_gaussian" if cfg.get("probe") == "gaussian" else ""), dom),
                "kernel": dom,
                "bytes_per_launch": int(bytes_per_launch), "avg_launch_us": round(tot_ms / cnt * 1e3, 2)}
    elif dom == "accumulate":
        flops = sum(2 * B * T * d * p for (_, d, p) in cfg["layers"])
        tf = flops * args.steps / (tot_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(tf, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf / BF16_PEAK_TFLOPS, 4), "traffic": measured_traffic(cfg["name"], dom), "kernel": dom,
                "flops_per_launch": int(flops / launches_per_step), "avg_launch_us": round(tot_ms / cnt * 1e3, 2)}
    else:
        roof = {"bound": "hbm", "achieved": None, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": None,
                "traffic": None, "kernel": dom}
    norm_bytes = workloads.algorithmic_norm_bytes(cfg)
    norm_ms = sum(per_kind.get(k, (0.0, 0))[0] for k in ("project", "token_reduce", "qr", "hutchpp_final",
                                                          "project_f32", "token_reduce_f32", "sample_sq",
                                                          "probe_bits", "token_splits", "sample_sum", "qr_combine", "qr_expand",
                                                          "hutchpp_sum", "probe_gauss")) / args.steps
    kernels = {k: {"launches_per_step": v[1] / args.steps, "avg_launch_us": round(v[0] / v[1] * 1e3, 2),
                   "us_per_step": round(v[0] / args.steps * 1e3, 2)} for k, v in sorted(per_kind.items())}
    extra = {"norm_kernels_us_per_step": round(norm_ms * 1e3, 2),
             "norm_hbm_gbps_kernels": round(norm_bytes / (norm_ms * 1e-3) / 1e9, 1) if norm_ms else None,
             "step_hbm_gbps": round(norm_bytes / (ms_per_step * 1e-3) / 1e9, 1),
             "step_hbm_frac": round(norm_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
             "kernels": kernels, "input_copies_rotated": copies,
             "hot_cache_tokens_per_s": round(B * T / (hot_ms * 1e-3), 1) if hot_ms else None}
    if not args.no_extra:
        extra["accumulate"] = accumulate_extra(D, torch, workloads, hip, max(5, args.steps // 5))
        if len(cfg["layers"]) == 1 and copies > 1:
            extra["vendor_read_same_operand"] = read_reference(torch, sets, copies, args.steps)
    rec = {"metric": "per-sample norm-estimation tokens/s + HBM GB/s (% peak), Llama-3.2-1B shapes",
           "value": round(B * T / (ms_per_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg["dtype"],
           "data": "synthetic (seeded; Llama-3.2-1B layer shapes)",
           "config": workloads.describe(cfg) | {"C": cfg["C"], "steps_include": step_parts(cfg),
                                                "launch": "hip_graph_replay" if args.graph else "eager"},
           "roofline": roof, "extra": extra}
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(cfg, sets, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


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
        grads = [D.dprc_clip_accumulate(A, E, c, ws=drv._ws_acc) for (A, E, _) in pairs]
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
        for (A, E, j), m in zip(pairs, masters):
            g = D.dprc_clip_accumulate(A, E, c, ws=drv._ws_acc)
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
