#!/usr/bin/env python3
"""Benchmark of the fused WTConv forward + backward on one MI355X.

Workload: ConvNeXt-T stage-1 layer shape, B=64, C=96, H=W=56, k=5, L=3,
float32, seeded synthetic inputs (see paper_2608_10805_amd/inputs.py). One
step is the whole operator: wtconv_forward, then the two phases of
wtconv_backward (the fused pass writing dx and kernel-gradient partials, then
the finalize that reduces and unfolds them). Inputs are resident in HBM before
timing starts; steps rotate over several distinct buffer sets so that the
256 MB Infinity Cache cannot hold one step's tensors for the next.

Prints one JSON line. `value` is achieved GB/s: the single-pass algorithmic
bytes (x, y, dy, dx, each read or written once; parameters and gradients)
divided by the measured step time. `roofline` describes the dominant kernel,
timed with HIP events on the stream it runs on. `cpu_baseline` times the
float64 CPU oracle on the host cores.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fused WTConv fwd+bwd ms and achieved HBM GB/s (% of peak), ConvNeXt-T shapes"
WORKLOAD = {"workload": "wtconv_fwdbwd_convnext_t_stage1", "B": 64, "C": 96, "H": 56, "W": 56, "k": 5, "L": 3,
            "dtype": "f32", "pass": "fwd+bwd"}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--sets", type=int, default=4, help="distinct input/output buffer sets rotated over")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target duration of the oracle timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (profiler counter calibration)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "hbm_traffic_wtconv_convnext_t_stage1.txt"),
                    help="counter summary with the measured HBM bytes of the dominant kernel")
    return ap.parse_args()


def cpu_baseline(inp, work_bytes, seconds):
    import oracle

    planes = WORKLOAD["B"] * WORKLOAD["C"]
    log(f"cpu_baseline: float64 oracle fwd+bwd over the whole workload ({planes} planes), "
        f"{oracle.num_threads()} threads")
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.forward(inp.x, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
        oracle.backward(inp.x, inp.dy, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    return {"value": round(work_bytes * reps / el / 1e9, 4), "unit": "GB/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"the full workload ({planes} planes of 56x56, k=5, L=3), forward and backward, "
                      f"{reps} repetitions in {el:.1f} s, float64; {el / reps * 1e3:.1f} ms per step"}


def kernel_source_hash():
    """sha256 of the HIP sources the library is built from."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_10805_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def load_traffic(path, kernel):
    """Measured HBM bytes per launch of `kernel` from a counter summary under
    profiles/ ("key: value" lines), if it was taken on the current kernel
    sources and workload; else None."""
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("kernel_source_sha256") != kernel_source_hash() or rec.get("workload") != WORKLOAD["workload"]:
        return None
    key = f"{kernel}_hbm_bytes_per_launch"
    return float(rec[key]) if key in rec else None


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}, WORLD_SIZE {world}); this operator's "
              f"benchmark has no multi-GPU mode.", file=sys.stderr, flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_10805_amd import binding, iomodel
    from paper_2608_10805_amd.inputs import make_inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * 1024 * 1024 // 4
        a, b = torch.ones(n, device=dev), torch.empty(n, device=dev)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log(f"copy calibration: 3 copies of {args.copy_calibration_mib} MiB")
        return
    B, C, H, W, k, L = (WORKLOAD[n] for n in ("B", "C", "H", "W", "k", "L"))
    log(f"bench: {WORKLOAD['workload']} B={B} C={C} H={H} W={W} k={k} L={L} f32, steps={args.steps} "
        f"warmup={args.warmup} sets={args.sets}")
    inp = make_inputs(B, C, H, W, k, L, "f32", seed=0)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    bw, bs = t(inp.base_w), t(inp.base_scale)
    lw, ls = [t(a) for a in inp.level_w], [t(a) for a in inp.level_scale]
    x0, dy0 = t(inp.x), t(inp.dy)
    sets = []
    for s in range(args.sets):
        x = x0 if s == 0 else x0.clone()
        dy = dy0 if s == 0 else dy0.clone()
        sets.append((x, dy, torch.empty_like(x), torch.empty_like(x)))
    bk = binding.Backward(x0, bw, bs, lw, ls, need_dx=True)

    def step(i, ev=None):
        x, dy, y, dx = sets[i % len(sets)]
        if ev is not None:
            ev[0].record()
        binding.forward(x, bw, bs, lw, ls, out=y)
        if ev is not None:
            ev[1].record()
        bk.partials(x, dy, dx)
        if ev is not None:
            ev[2].record()
        bk.finalize()
        if ev is not None:
            ev[3].record()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    log("bench: warmup done")

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        step(i, evs[i])
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps
    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    bwd_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    fin_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    log(f"bench: {ms_step * 1e3:.1f} us/step (forward {fwd_ms * 1e3:.1f}, backward fused {bwd_ms * 1e3:.1f}, "
        f"finalize {fin_ms * 1e3:.1f})")

    work = iomodel.single_pass_work(B, C, H, W, k, L, "f32")
    value = work.bytes_fwdbwd / (ms_step * 1e-3) / 1e9
    if bwd_ms >= fwd_ms:
        dom, dom_ms, dom_fma, dom_bytes = "backward_fused", bwd_ms, work.fma_bwd, work.bytes_bwd
    else:
        dom, dom_ms, dom_fma, dom_bytes = "forward", fwd_ms, work.fma_fwd, work.bytes_fwd
    achieved = 2.0 * dom_fma / (dom_ms * 1e-3) / 1e12
    peak = iomodel.FP32_FLOPS / 1e12
    traffic = load_traffic(args.traffic, dom)
    roofline = {"bound": "alu", "achieved": round(achieved, 3), "peak": round(peak, 1), "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": traffic, "kernel": dom,
                "kernel_ms": round(dom_ms, 5),
                "hbm_view": {"algorithmic_bytes": dom_bytes,
                             "achieved_GBps": round(dom_bytes / (dom_ms * 1e-3) / 1e9, 1),
                             "frac": round(dom_bytes / (dom_ms * 1e-3) / 1e9 / iomodel.HBM_PEAK_GBPS, 4)}}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(inp, work.bytes_fwdbwd, args.cpu_seconds)
    N = B * C * H * W
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic (seeded; x, dy ~ N(0,1), weights U(-0.2,0.2))",
        "config": dict(WORKLOAD),
        "hbm_frac": round(value / iomodel.HBM_PEAK_GBPS, 4),
        "fwd_ms": round(fwd_ms, 5), "bwd_fused_ms": round(bwd_ms, 5), "bwd_finalize_ms": round(fin_ms, 5),
        "algorithmic_bytes_per_step": work.bytes_fwdbwd,
        "floors_us": {"hbm": round(iomodel.hbm_floor_s(work.bytes_fwdbwd) * 1e6, 2),
                      "fp32_fma": round(iomodel.fma_floor_s(work.fma_fwdbwd) * 1e6, 2)},
        "paper_io_model_elems_per_N": {"Q_ref": round(iomodel.q_ref(L), 3), "Q_fused": round(iomodel.q_fused(L), 3),
                                       "single_pass_fwd": 2, "single_pass_fwdbwd": 5},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "N": N,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
