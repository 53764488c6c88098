"""Benchmark of the fused ConvFirst block on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu] [--no-extra]

A step is one fused-block forward over one batch (N = 128, 56 x 56, C = 64,
E = 4, depth-wise 3 x 3, GELU(erf), fp16 NHWC) with inputs resident in HBM.
Steps rotate over several x/y buffer sets whose total exceeds the 256 MB
Infinity Cache, so a step never reads what the previous one wrote.  HIP
events on the launch stream bracket exactly K steps after W warm-up steps.

Prints ONE JSON line: images/s (value), ms per step, computational efficiency
(FLOPs of the block at the dense fp16 MFMA peak divided by the measured
latency), the roofline of the kernel, the fp64 CPU oracle timed on a bounded
sample on the host cores, and the other workloads (block C = 256 k = 7, the
four-stage stack, the layer-by-layer baseline, the N = 1 latency cases).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

import paper_2404_03617_amd as cf
from paper_2404_03617_amd import roofline as rl
from paper_2404_03617_amd import synth
from paper_2404_03617_amd.workloads import BENCH_WORKLOAD, WORKLOADS

MALL_BYTES = 256 << 20
HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "paper_2404_03617_amd", "csrc")
PROFILES = os.path.join(HERE, "profiles")
# sources of the C = 64 fp16 fused kernel; the counter-based traffic figure is
# reported only while they hash to the value recorded with the counters
FUSED_SOURCES = ("cf_block64.h", "cf_block64_k3.hip", "cf_fused_impl.h", "cf_device.h")


def fused_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in FUSED_SOURCES:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(name: str):
    """HBM bytes per launch of the fused kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, or None when it is absent or was taken
    on different kernel sources."""
    path = os.path.join(PROFILES, "fused_block_%s.md" % name)
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and line.startswith("- "):
                k, v = line[2:].split(":", 1)
                fields[k.strip()] = v.strip().strip("`")
    if fields.get("kernel source hash") != fused_source_hash():
        return None
    try:
        return int(fields["traffic bytes per launch"])
    except (KeyError, ValueError):
        return None


def calib_copy():
    """A plain elementwise kernel over a known size (256 MiB read, 256 MiB
    written) whose FETCH_SIZE / WRITE_SIZE calibrate the counters."""
    a = torch.ones(128 << 20, dtype=torch.float16, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        torch.neg(a, out=b)
    torch.cuda.synchronize()


def _sets_needed(bytes_per_set: int) -> int:
    return max(2, min(16, -(-2 * MALL_BYTES // max(bytes_per_set, 1))))


def _time(fn, steps: int, warmup: int, stream) -> float:
    """Seconds per step from HIP events on `stream`."""
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for i in range(steps):
        fn(warmup + i)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / 1e3 / steps


def _time_each(fn, steps: int, stream) -> float:
    """Average seconds of one launch, each bracketed by its own HIP events on
    `stream` (the per-kernel duration the roofline divides by)."""
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        starts[i].record(stream)
        fn(i)
        ends[i].record(stream)
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in zip(starts, ends)) / 1e3 / steps


def block_case(name: str, steps: int, warmup: int, act: str = "gelu", unfused: bool = False,
               per_launch: bool = False):
    w = WORKLOADS[name]
    N, H, W, C, E, k = w["N"], w["H"], w["W"], w["C"], w["E"], w["k"]
    eb = 2
    nsets = _sets_needed(2 * N * H * W * C * eb)
    xs = [synth.activations(w["seed"] + 100 * i, N, H, W, C, w["dtype"]).cuda() for i in range(nsets)]
    ys = [torch.empty_like(xs[0]) for _ in range(nsets)]
    p = {kk: (None if v is None else v.cuda()) for kk, v in
         synth.block_params(w["seed"], 0, C, E, k, w["dtype"]).items()}
    stream = torch.cuda.current_stream()
    if unfused:
        ws = torch.empty(cf.lib().cf_unfused_workspace_bytes(N, H, W, C, E, 0), dtype=torch.uint8,
                         device="cuda")
        fn = lambda i: cf.block_forward_unfused(xs[i % nsets], p, act=act, out=ys[i % nsets], ws=ws)
        cfg = None
    else:
        # as the paper's benchmark does, tune before the timed iterations: the
        # library times each kernel configuration of this shape and keeps the
        # fastest for the block_forward calls below
        cf.block_autotune(xs[0], p, act=act, out=ys[0])
        cfg = cf.block_tuned_config(xs[0].shape, C, E, k, xs[0].dtype, act)
        fn = lambda i: cf.block_forward(xs[i % nsets], p, act=act, out=ys[i % nsets])
    t = _time(fn, steps, warmup, stream)
    t_kernel = _time_each(fn, steps, stream) if per_launch else t
    flops = rl.block_flops(N, H, W, C, E, k)
    return dict(N=N, seconds=t, kernel_seconds=t_kernel, flops=flops, kernel_config=cfg,
                bytes=rl.block_bytes_fused(N, H, W, C, E, k, eb))


def split_case(name: str, steps: int, warmup: int):
    w = WORKLOADS[name]
    N, H, W, C, E, k = w["N"], w["H"], w["W"], w["C"], w["E"], w["k"]
    x = synth.activations(w["seed"], N, H, W, C, w["dtype"]).cuda()
    y = torch.empty_like(x)
    p = {kk: (None if v is None else v.cuda()) for kk, v in
         synth.block_params(w["seed"], 0, C, E, k, w["dtype"]).items()}
    ws = torch.empty(cf.lib().cf_split_workspace_bytes(N, H, W, C, E, 0), dtype=torch.uint8, device="cuda")
    t = _time(lambda i: cf.block_forward_split(x, p, out=y, ws=ws), steps, warmup, torch.cuda.current_stream())
    return dict(N=N, seconds=t, flops=rl.block_flops(N, H, W, C, E, k))


def stack_case(name: str, steps: int, warmup: int):
    w = WORKLOADS[name]
    N, H, W = w["N"], w["H"], w["W"]
    depths, widths, E, k = w["depths"], w["widths"], w["E"], w["k"]
    layers = [(kd, {kk: (None if v is None else v.cuda()) for kk, v in p.items()})
              for kd, p in synth.stack_layers(w["seed"], depths, widths, E, k, w["dtype"])]
    nsets = 2
    xs = [synth.activations(w["seed"] + 100 * i, N, H, W, widths[0], w["dtype"]).cuda() for i in range(nsets)]
    # one output buffer per stage / down-sampling step
    bufs = []
    h, ww = H, W
    for s, c in enumerate(widths):
        if s > 0:
            h, ww = h // 2, ww // 2
            bufs.append(torch.empty((N, h, ww, c), dtype=xs[0].dtype, device="cuda"))
        bufs.append(torch.empty((N, h, ww, c), dtype=xs[0].dtype, device="cuda"))
    eager = lambda i: cf.stack_forward(xs[i % nsets], layers, bufs=bufs)
    t_eager = _time(eager, steps, warmup, torch.cuda.current_stream())
    # the launch sequence replayed as one HIP graph per input set
    try:
        graphs = [cf.capture_stack(xs[i], layers, bufs) for i in range(nsets)]
        t = _time(lambda i: graphs[i % nsets].replay(), steps, warmup, torch.cuda.current_stream())
        mode = "hipGraph replay"
    except Exception as e:  # capture unavailable: the eager launches are the figure
        t, mode = t_eager, "eager launches (graph capture failed: %s)" % (str(e).splitlines() or ["?"])[0]
    kern = rl.stack_kernels(N, H, W, depths, widths, E, k)
    flops = sum(n for _, n, _ in kern)
    T, cmax = rl.waterline([(n, b) for _, n, b in kern])
    return dict(N=N, seconds=t, eager_seconds=t_eager, mode=mode, flops=flops, waterline_T_min_s=T,
                waterline_C_max=cmax)


def cpu_baseline(name: str, min_seconds: float = 12.0):
    """The fp64 oracle on the workload's full batch, all host cores, repeated
    until at least `min_seconds` of CPU work have been timed."""
    import oracle
    w = WORKLOADS[name]
    x = synth.activations(w["seed"], w["N"], w["H"], w["W"], w["C"], w["dtype"])
    p = synth.params_f64(synth.block_params(w["seed"], 0, w["C"], w["E"], w["k"], w["dtype"]))
    xd = synth.to_f64(x)
    passes, used = 0, 0
    t0 = time.perf_counter()
    while True:
        _, used = oracle.block_forward(xd, p, act="gelu", return_threads=True)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    images = passes * w["N"]
    return {"value": round(images / dt, 2), "unit": "images/s", "cores": int(used), "kind": "oracle",
            "sample": "%d passes over the %d-image batch of %s (fp64 C loops), %.1f s"
                      % (passes, w["N"], name, dt)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=BENCH_WORKLOAD)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-extra", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run a 256 MiB elementwise copy (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this library has no multi-GPU path; run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    cf.lib()
    name = args.workload
    w = WORKLOADS[name]
    res = block_case(name, args.steps, args.warmup, per_launch=True)
    t = res["seconds"]
    tk = res["kernel_seconds"]
    N = res["N"]
    ips = N / t
    eff = rl.comp_eff(res["flops"], t)
    gbps = res["bytes"] / tk / 1e9
    t_hbm = res["bytes"] / rl.PEAK_HBM_BPS
    t_mfma = res["flops"] / rl.PEAK_FP16_FLOPS
    bound = "hbm" if t_hbm >= t_mfma else "mfma"
    if bound == "hbm":
        roof = {"bound": "hbm", "achieved": round(gbps, 1), "peak": rl.PEAK_HBM_BPS / 1e9, "unit": "GB/s",
                "frac": round(gbps * 1e9 / rl.PEAK_HBM_BPS, 4), "traffic": measured_traffic(name)}
    else:
        tf = res["flops"] / tk / 1e12
        roof = {"bound": "mfma", "achieved": round(tf, 1), "peak": rl.PEAK_FP16_FLOPS / 1e12,
                "unit": "TFLOP/s", "frac": round(tf * 1e12 / rl.PEAK_FP16_FLOPS, 4),
                "traffic": measured_traffic(name)}
    out = {
        "metric": "images/sec and % of fp16 MFMA peak (computational efficiency), batch 128",
        "value": round(ips, 1),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded N(0,1) activations, N(0,1/fan_in) weights)",
        "config": {"workload": name, "N": w["N"], "H": w["H"], "W": w["W"], "C": w["C"], "E": w["E"],
                   "k": w["k"], "act": "gelu_erf", "kernel": "fused block (1 launch)",
                   "kernel_config": res["kernel_config"]},
        "comp_eff": round(eff, 4),
        "tflops": round(res["flops"] / t / 1e12, 1),
        "kernel_us": round(tk * 1e6, 2),
        "roofline": roof,
    }
    if not args.no_extra:
        extra = {}
        u = block_case(name, max(5, args.steps // 5), 2, unfused=True)
        extra["unfused_same_workload"] = {"ms": round(u["seconds"] * 1e3, 4),
                                          "images_per_s": round(u["N"] / u["seconds"], 1),
                                          "comp_eff": round(rl.comp_eff(u["flops"], u["seconds"]), 4),
                                          "fused_speedup": round(u["seconds"] / t, 2)}
        r = block_case(name, max(5, args.steps // 5), 2, act="relu")
        extra["relu_same_workload"] = {"ms": round(r["seconds"] * 1e3, 4),
                                       "comp_eff": round(rl.comp_eff(r["flops"], r["seconds"]), 4)}
        for nm in WORKLOADS:
            wk = WORKLOADS[nm]
            if nm == name:
                continue
            if wk["kind"] == "block":
                b = block_case(nm, max(5, args.steps // 2), 3)
                e = {"ms": round(b["seconds"] * 1e3, 4), "images_per_s": round(b["N"] / b["seconds"], 1),
                     "comp_eff": round(rl.comp_eff(b["flops"], b["seconds"]), 4)}
                if wk["N"] * wk["H"] * wk["W"] <= 256:
                    s = split_case(nm, max(5, args.steps // 2), 3)
                    e["split_ms"] = round(s["seconds"] * 1e3, 4)
                extra[nm] = e
            else:
                s = stack_case(nm, max(3, args.steps // 5), 2)
                extra[nm] = {"ms": round(s["seconds"] * 1e3, 4), "images_per_s": round(s["N"] / s["seconds"], 1),
                             "comp_eff": round(rl.comp_eff(s["flops"], s["seconds"]), 4),
                             "mode": s["mode"], "eager_ms": round(s["eager_seconds"] * 1e3, 4),
                             "waterline_C_max": round(s["waterline_C_max"], 4)}
        out["other_workloads"] = extra
    if args.calib_copy:
        calib_copy()
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(name, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
