#!/usr/bin/env python3
"""Benchmark of the fused WTConv forward + backward on one MI355X.

Workload: ConvNeXt-T stage-1 layer shape, B=64, C=96, H=W=56, k=5, L=3,
float32, seeded synthetic inputs (see paper_2608_10805_amd/inputs.py). One
step is the whole operator, forward and backward, as the library's entry
points run it for this shape: wtconv_forward (y), wtconv_backward_partials
without dx (the kernel-gradient pass), wtconv_backward_data (dx: the forward
pass on dy with rotated kernels) and wtconv_backward_finalize (fixed-order
reduction and unfold) -- exactly the kernels wtconv_backward launches here,
each bracketed by its own HIP events. Inputs are resident in HBM before timing
starts; steps rotate over several distinct buffer sets so that the 256 MB
Infinity Cache cannot hold one step's tensors for the next.

Prints one JSON line. `value` is achieved GB/s: the single-pass algorithmic
bytes (x, y, dy, dx, each read or written once; parameters and gradients)
divided by the measured step time. `roofline` describes the dominant kernel (the one
with the largest share of the step), timed with HIP events on the stream it
runs on; `kernels` lists every kernel of the step the same way. `cpu_baseline` times the
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
    ap.add_argument("--warmup", type=int, default=200,
                    help="untimed steps before the timed region (the GPU clock settles over tens of ms)")
    ap.add_argument("--sets", type=int, default=4, help="distinct input/output buffer sets rotated over")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target duration of the oracle timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (profiler counter calibration)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "hbm_traffic_wtconv_convnext_t_stage1.txt"),
                    help="counter summary with the measured HBM bytes of the dominant kernel")
    ap.add_argument("--no-config-table", action="store_true",
                    help="skip the per-configuration fwd / fwd+bwd timing table")
    ap.add_argument("--table-steps", type=int, default=10)
    ap.add_argument("--summarize-trace", metavar="DB",
                    help="write the kernel statistics of a rocprofv3 --kernel-trace database to --out and exit")
    ap.add_argument("--summarize-counters", metavar="DB",
                    help="write the SQ instruction counters of a rocprofv3 --pmc database to --out and exit")
    ap.add_argument("--summarize-traffic", nargs=4, metavar=("FETCH_DB", "WRITE_DB", "COPY_FETCH_DB", "COPY_WRITE_DB"),
                    help="write per-launch HBM bytes from rocprofv3 FETCH_SIZE / WRITE_SIZE databases of this "
                         "benchmark and of --copy-calibration-mib runs to --out and exit")
    ap.add_argument("--traffic-invariance-run", action="store_true",
                    help="run one forward of each traffic-invariance configuration and exit (for rocprofv3 --pmc)")
    ap.add_argument("--summarize-invariance", nargs=4, metavar=("FETCH_DB", "WRITE_DB", "COPY_FETCH_DB", "COPY_WRITE_DB"),
                    help="write the HBM traffic of each --traffic-invariance-run forward, in units of N, to --out and exit")
    ap.add_argument("--copy-mib", type=int, default=256, help="size of the calibration copy behind --summarize-traffic")
    ap.add_argument("--command", default="", help="the profiling command, recorded in the summary")
    ap.add_argument("--out", help="summary file for --summarize-trace / --summarize-traffic")
    return ap.parse_args()


# Every benchmarked configuration of the operator (fwd and fwd+bwd timed for each):
# (name, B, C, H, W, k, L, dtype)
def table_configs():
    out = [("small_fwd", 2, 16, 32, 32, 5, 1, "f32"),
           ("convnext_s1", 64, 96, 56, 56, 5, 3, "f32")]
    out += [(f"convnext_s2_L{L}", 64, 192, 28, 28, 5, L, "f32") for L in range(1, 6)]
    out += [("convnext_s1_bf16_L5", 128, 96, 56, 56, 5, 5, "bf16")]
    for (B, C, H, W) in [(128, 96, 56, 56), (128, 192, 28, 28), (128, 384, 14, 14), (128, 768, 7, 7),
                         (32, 128, 63, 95), (16, 64, 224, 224)]:
        for dt in ("f32", "bf16"):
            for L in (1, 3, 5):
                out.append((f"sweep_{H}x{W}_c{C}_L{L}_{dt}", B, C, H, W, 5, L, dt))
    # the paper's own layer sweep: B=8, C in {32, 64, 128}, H=W in {128, 256, 512},
    # L = 1..5, fp32 and fp16, k = 5 (its latency tables report the geometric
    # mean over the nine shapes)
    for k in (5, 3):
        for dt in ("f32", "f16"):
            for L in range(1, 6):
                for C in (32, 64, 128):
                    for H in (128, 256, 512):
                        out.append((f"paper_k{k}_{H}x{H}_c{C}_L{L}_{dt}", 8, C, H, H, k, L, dt))
    return out


# The paper's fused-kernel latencies on its RTX A6000 (geometric mean over its
# nine layer shapes, L = 1..5; absolute-latency tables for k = 5 and k = 3), for
# context next to the MI355X figures.
PAPER_A6000_MS = {
    5: {"f32": {"fwd": [2.312, 2.552, 2.634, 2.681, 2.703], "fwdbwd": [7.800, 8.693, 8.995, 9.154, 9.277]},
        "f16": {"fwd": [1.389, 1.592, 1.668, 1.710, 1.748], "fwdbwd": [5.365, 6.148, 6.442, 6.600, 6.733]}},
    3: {"f32": {"fwd": [1.667, 1.880, 1.945, 1.979, 2.001], "fwdbwd": [6.081, 6.891, 7.135, 7.248, 7.332]},
        "f16": {"fwd": [1.029, 1.155, 1.205, 1.234, 1.258], "fwdbwd": [3.908, 4.470, 4.665, 4.773, 4.870]}},
}


def paper_sweep_summary(rows):
    """Geometric means over the paper's nine layer shapes, per kernel size,
    dtype and L: {"k5": {"f32": [...], "f16": [...]}, "k3": {...}}."""
    import math
    out = {}
    for k in (5, 3):
        per_dt = {}
        for dt in ("f32", "f16"):
            per_l = []
            for L in range(1, 6):
                sel = [r for r in rows if r["name"].startswith("paper_") and r["k"] == k and r["dtype"] == dt
                       and r["L"] == L]
                if len(sel) != 9:
                    continue
                g = lambda key: math.exp(sum(math.log(r[key]) for r in sel) / len(sel))  # noqa: E731
                per_l.append({"L": L, "fwd_ms": round(g("fwd_ms"), 4), "fwdbwd_ms": round(g("fwdbwd_ms"), 4),
                              "paper_a6000_fwd_ms": PAPER_A6000_MS[k][dt]["fwd"][L - 1],
                              "paper_a6000_fwdbwd_ms": PAPER_A6000_MS[k][dt]["fwdbwd"][L - 1]})
            per_dt[dt] = per_l
        out[f"k{k}"] = per_dt
    return out


def config_table(steps, dev):
    """ms, algorithmic GB/s and roofline fractions of fwd and fwd+bwd for every
    configuration. Timing-only inputs are drawn on the device (seeded, with the
    distributions of the parity inputs); buffer sets rotate so that one step's
    tensors do not stay in the 256 MB Infinity Cache."""
    import torch

    from paper_2608_10805_amd import binding, iomodel

    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
    gen = torch.Generator(device=dev)
    rows = []
    for name, B, C, H, W, k, L, dt in table_configs():
        gen.manual_seed(0)
        f32 = dict(device=dev, dtype=torch.float32)
        bw = (torch.rand(C, k, k, generator=gen, **f32) * 0.4 - 0.2)
        bs = torch.rand(C, generator=gen, **f32) + 0.5
        lw = [torch.rand(4 * C, k, k, generator=gen, **f32) * 0.4 - 0.2 for _ in range(L)]
        ls = [torch.rand(4 * C, generator=gen, **f32) * 0.15 + 0.05 for _ in range(L)]
        act = B * C * H * W * iomodel.elem_bytes(dt)
        nsets = max(1, min(8, -(-600 * 2 ** 20 // (4 * act))))
        sets = []
        for _ in range(nsets):
            x = torch.randn(B, C, H, W, generator=gen, **f32).to(tdt[dt])
            dy = torch.randn(B, C, H, W, generator=gen, **f32).to(tdt[dt])
            sets.append((x, dy, torch.empty_like(x), torch.empty_like(x)))
        fws = torch.empty(max(1, binding.wtconv_forward_workspace_bytes(
            binding.make_desc(B, C, H, W, k, L, binding._dtype_code(sets[0][0])))), dtype=torch.uint8, device=dev)
        bk = binding.Backward(sets[0][0], bw, bs, lw, ls, need_dx=True)

        def run(n, with_bwd):
            for i in range(n):
                x, dy, y, dx = sets[i % nsets]
                binding.forward(x, bw, bs, lw, ls, out=y, workspace=fws)
                if with_bwd:
                    bk.partials(x, dy, dx)
                    bk.finalize()

        res = {}
        for with_bwd in (False, True):
            # untimed runs for at least 20 ms first: the GPU clock settles over
            # tens of ms, and a short configuration is otherwise timed cold
            t0 = time.perf_counter()
            while True:
                run(3, with_bwd)
                torch.cuda.synchronize()
                if time.perf_counter() - t0 >= 0.02:
                    break
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record()
            run(steps, with_bwd)
            b.record()
            torch.cuda.synchronize()
            res[with_bwd] = a.elapsed_time(b) / steps
        work = iomodel.single_pass_work(B, C, H, W, k, L, dt)
        fwd_ms, fb_ms = res[False], res[True]
        row = {"name": name, "B": B, "C": C, "H": H, "W": W, "k": k, "L": L, "dtype": dt,
               "fwd_ms": round(fwd_ms, 4), "fwdbwd_ms": round(fb_ms, 4),
               "fwd_GBps": round(work.bytes_fwd / (fwd_ms * 1e-3) / 1e9, 1),
               "fwdbwd_GBps": round(work.bytes_fwdbwd / (fb_ms * 1e-3) / 1e9, 1)}
        row["fwd_hbm_frac"] = round(row["fwd_GBps"] / iomodel.HBM_PEAK_GBPS, 4)
        row["fwdbwd_hbm_frac"] = round(row["fwdbwd_GBps"] / iomodel.HBM_PEAK_GBPS, 4)
        row["fwdbwd_fma_frac"] = round(iomodel.fma_floor_s(work.fma_fwdbwd) / (fb_ms * 1e-3), 4)
        log(f"table: {name:28s} fwd {fwd_ms * 1e3:8.1f} us  fwd+bwd {fb_ms * 1e3:8.1f} us  "
            f"{row['fwdbwd_GBps']:7.1f} GB/s  fma {row['fwdbwd_fma_frac']:.3f}")
        rows.append(row)
        del sets, bk, fws
        torch.cuda.empty_cache()
    return rows


def memory_table(dev):
    """Peak allocated device memory of the layer (`WTConv2d`) over one training
    step (forward, then backward from a given dy) and over one inference
    forward, for the paper's nine layer shapes, L = 1..5, fp32 and fp16.

    Each peak is divided by the compulsory footprint: inference x, y and the
    parameters; training x, y, dy, dx, the parameters and their gradients,
    which is about what a plain depthwise convolution of the same shape holds.
    Reported per dtype and L as the geometric mean and the maximum over the
    shapes, with the largest workspace (peak minus compulsory) in bytes."""
    import math

    import torch

    from paper_2608_10805_amd import iomodel
    from paper_2608_10805_amd.autograd import WTConv2d

    tdt = {"f32": torch.float32, "f16": torch.float16}
    gen = torch.Generator(device=dev)
    out = {}
    for dt in ("f32", "f16"):
        per_l = []
        for L in range(1, 6):
            train, infer, extra = [], [], 0
            for C in (32, 64, 128):
                for H in (128, 256, 512):
                    B, k = 8, 5
                    gen.manual_seed(0)
                    layer = WTConv2d(C, kernel_size=k, levels=L, device=dev)
                    nparam = sum(p.numel() for p in layer.parameters()) * 4
                    act = B * C * H * H * iomodel.elem_bytes(dt)
                    x = torch.randn(B, C, H, H, generator=gen, device=dev).to(tdt[dt])
                    dy = torch.randn(B, C, H, H, generator=gen, device=dev).to(tdt[dt])
                    torch.cuda.synchronize()
                    base = torch.cuda.memory_allocated(dev) - 2 * act - nparam
                    torch.cuda.reset_peak_memory_stats(dev)
                    with torch.no_grad():
                        y = layer(x)
                    torch.cuda.synchronize()
                    peak_inf = torch.cuda.max_memory_allocated(dev) - base - act  # dy is not part of inference
                    comp_inf = 2 * act + nparam
                    del y
                    x.requires_grad_(True)
                    torch.cuda.synchronize()
                    torch.cuda.reset_peak_memory_stats(dev)
                    y = layer(x)
                    y.backward(dy)
                    torch.cuda.synchronize()
                    peak_tr = torch.cuda.max_memory_allocated(dev) - base
                    comp_tr = 4 * act + 2 * nparam
                    infer.append(peak_inf / comp_inf)
                    train.append(peak_tr / comp_tr)
                    extra = max(extra, peak_tr - comp_tr, peak_inf - comp_inf)
                    del x, dy, y, layer
                    torch.cuda.empty_cache()
            gm = lambda v: math.exp(sum(math.log(t) for t in v) / len(v))  # noqa: E731
            per_l.append({"L": L, "train_peak_over_compulsory": round(gm(train), 4),
                          "train_max": round(max(train), 4),
                          "infer_peak_over_compulsory": round(gm(infer), 4), "infer_max": round(max(infer), 4),
                          "max_extra_bytes": int(extra)})
            log(f"memory: {dt} L{L} train {gm(train):.4f} (max {max(train):.4f})  "
                f"infer {gm(infer):.4f} (max {max(infer):.4f})  extra {extra / 2 ** 20:.1f} MiB")
        out[dt] = per_l
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inp, work_bytes, seconds):
    import oracle

    planes = WORKLOAD["B"] * WORKLOAD["C"]
    threads = oracle.num_threads()
    log(f"cpu_baseline: float64 oracle fwd+bwd over the whole workload ({planes} planes), {threads} threads")
    reps, t0 = 0, time.perf_counter()
    while True:
        y_ref = oracle.forward(inp.x, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
        g_ref = oracle.backward(inp.x, inp.dy, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    # single-thread forward on a 4-image slice of the same workload, scaled to the whole batch
    nb = 4
    oracle.set_num_threads(1)
    t1 = time.perf_counter()
    oracle.forward(inp.x[:nb], inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
    el1 = time.perf_counter() - t1
    oracle.set_num_threads(threads)
    fwd1_s = el1 * WORKLOAD["B"] / nb
    refs = {"y": y_ref, "dx": g_ref["dx"], "d_base_w": g_ref["d_base_w"], "d_base_scale": g_ref["d_base_scale"],
            "d_level_w": g_ref["d_level_w"], "d_level_scale": g_ref["d_level_scale"]}
    return refs, {"value": round(work_bytes * reps / el / 1e9, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"the full workload ({planes} planes of 56x56, k=5, L=3), forward and backward, "
                      f"{reps} repetitions in {el:.1f} s, float64; {el / reps * 1e3:.1f} ms per step",
            "fwd_1thread_s": round(fwd1_s, 3),
            "fwd_1thread_sample": f"forward of {nb} of {WORKLOAD['B']} images ({nb * WORKLOAD['C']} planes) on one "
                                  f"thread in {el1:.2f} s, scaled to the whole batch"}


def full_size_parity(refs, x, dy, bw, bs, lw, ls):
    """Every output of one forward and one backward of the library on the
    benchmark's own inputs against the float64 oracle's (the cpu_baseline run):
    max |got - ref| / max |ref| per tensor, against the fp32 tolerance 1e-5."""
    import numpy as np

    from paper_2608_10805_amd import binding
    y = binding.forward(x, bw, bs, lw, ls)
    dx, dbw, dbs, dlw, dls = binding.backward(x, dy, bw, bs, lw, ls, need_dx=True)
    got = {"y": [y], "dx": [dx], "d_base_w": [dbw], "d_base_scale": [dbs], "d_level_w": dlw, "d_level_scale": dls}
    errs = {}
    for name, ts in got.items():
        ref = refs[name] if isinstance(refs[name], list) else [refs[name]]
        g = np.concatenate([t.detach().cpu().double().numpy().ravel() for t in ts])
        r = np.concatenate([np.asarray(a, dtype=np.float64).ravel() for a in ref])
        errs[name] = float(np.max(np.abs(g - r)) / max(float(np.max(np.abs(r))), 1e-30))
    tol = 1e-5
    return {"vs": "float64 oracle, whole workload", "max_rel_err": {k: float(f"{v:.3g}") for k, v in errs.items()},
            "tol": tol, "pass": all(v < tol for v in errs.values())}


def copy_ceiling_gbps(dev, gib=1):
    """Device-to-device copy of `gib` GiB: bytes read + written per second."""
    import torch
    n = gib * (1 << 30) // 4
    a, b = torch.ones(n, device=dev), torch.empty(n, device=dev)
    for _ in range(2):
        b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    reps = 5
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    s = e0.elapsed_time(e1) * 1e-3 / reps
    del a, b
    torch.cuda.empty_cache()
    return 2.0 * n * 4 / s / 1e9


def valu_probe(dev):
    """Sustained non-packed fp32 FMA rate from the probe kernel (TFLOP/s and implied clock)."""
    import ctypes

    import torch
    from paper_2608_10805_amd import build

    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.valu_probe_fmas.restype = ctypes.c_longlong
    lib.valu_probe_fmas.argtypes = [ctypes.c_int, ctypes.c_int]
    lib.valu_probe_launch.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    blocks, iters = 8192, 256
    out = torch.empty(blocks * 256, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    for _ in range(2):
        assert lib.valu_probe_launch(out.data_ptr(), blocks, iters, stream) == 0
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    reps = 3
    for _ in range(reps):
        assert lib.valu_probe_launch(out.data_ptr(), blocks, iters, stream) == 0
    e1.record()
    torch.cuda.synchronize()
    s = e0.elapsed_time(e1) * 1e-3 / reps
    fma_s = lib.valu_probe_fmas(blocks, iters) / s
    return {"fp32_TFLOPs": round(2 * fma_s / 1e12, 2), "implied_clock_GHz": round(fma_s / (256 * 64) / 1e9, 3)}


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


# Kernels of the benchmark step, by the symbol prefix rocprofv3 reports.
STEP_KERNELS = {"forward": "fused_kernel<5, float, false, true, false>", "grad": "grad_kernel<5, float, false>",
                "finalize": "reduce_kernel"}


def _rocpd_rows(db, sql):
    import sqlite3
    con = sqlite3.connect(db)
    try:
        return con.execute(sql).fetchall()
    finally:
        con.close()


def summarize_trace(db, out, command):
    """Kernel statistics (calls, total and average duration) of a rocprofv3
    --kernel-trace database, one line per kernel."""
    rows = _rocpd_rows(db, "select name, count(*), sum(duration), avg(duration) from kernels group by name "
                           "order by sum(duration) desc")
    total = sum(r[2] for r in rows)
    lines = ["# rocprofv3 kernel trace statistics, fused WTConv fwd+bwd benchmark step",
             f"# workload: {WORKLOAD['workload']} B={WORKLOAD['B']} C={WORKLOAD['C']} H=W={WORKLOAD['H']} "
             f"k={WORKLOAD['k']} L={WORKLOAD['L']} fp32, MI355X",
             f"# command: {command}",
             f"kernel_source_sha256: {kernel_source_hash()}",
             "# kernel | calls | total_us | average_us | percent"]
    for name, n, tot, avg in rows:
        short = name.replace("void ", "").replace("wtc::(anonymous namespace)::", "").split("(wtc::")[0]
        lines.append(f"{short[:110]} | {n} | {tot / 1e3:.1f} | {avg / 1e3:.3f} | {100.0 * tot / total:.1f}")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def _counter_per_kernel(db, counter):
    """Mean value of `counter` per dispatch, by kernel name (rocprofv3 --pmc database)."""
    rows = _rocpd_rows(db, f"select kernel_name, dispatch_id, sum(value) from counters_collection where "
                           f"counter_name = '{counter}' group by kernel_name, dispatch_id")
    acc = {}
    for name, _, v in rows:
        acc.setdefault(name, []).append(v)
    return {k: sum(v) / len(v) for k, v in acc.items()}


def summarize_traffic(fetch_db, write_db, cfetch_db, cwrite_db, copy_mib, out, command):
    """Measured HBM bytes per launch of the step's kernels: FETCH_SIZE and
    WRITE_SIZE (KiB) scaled by what the same counters report for a plain device
    copy of known size."""
    copy_kib = copy_mib * 1024.0
    cf = max((v for k, v in _counter_per_kernel(cfetch_db, "FETCH_SIZE").items() if "copyBuffer" in k), default=0)
    cw = max((v for k, v in _counter_per_kernel(cwrite_db, "WRITE_SIZE").items() if "copyBuffer" in k), default=0)
    fscale, wscale = copy_kib / cf, copy_kib / cw
    fetch = _counter_per_kernel(fetch_db, "FETCH_SIZE")
    write = _counter_per_kernel(write_db, "WRITE_SIZE")
    B, C, H, W, k, L = (WORKLOAD[n] for n in ("B", "C", "H", "W", "k", "L"))
    from paper_2608_10805_amd import iomodel
    algo = 2.0 * B * C * H * W * 4 + 4.0 * iomodel.param_count(C, k, L)
    lines = ["# HBM traffic per kernel launch from rocprofv3 counters, fused WTConv fwd+bwd benchmark step",
             f"# workload: B={B} C={C} H=W={H} k={k} L={L} fp32 (ConvNeXt-T stage 1), MI355X",
             f"# commands (one counter per run): {command}",
             f"# calibration: a {copy_mib} MiB device copy reads and writes {copy_kib:.0f} KiB; FETCH_SIZE reports "
             f"{cf:.0f} KiB (scale x{fscale:.3f}), WRITE_SIZE reports {cw:.0f} KiB (scale x{wscale:.3f})",
             f"workload: {WORKLOAD['workload']}",
             f"kernel_source_sha256: {kernel_source_hash()}",
             f"fetch_scale: {fscale:.4f}",
             f"write_scale: {wscale:.4f}"]
    for key, prefix in STEP_KERNELS.items():
        fk = [v for n, v in fetch.items() if prefix in n]
        wk = [v for n, v in write.items() if prefix in n]
        if not fk or not wk:
            continue
        f_kib, w_kib = sum(fk) / len(fk), sum(wk) / len(wk)
        hbm = f_kib * 1024 * fscale + w_kib * 1024 * wscale
        note = f"; algorithmic {algo / 1e6:.2f} MB; ratio {hbm / algo:.3f}" if key != "finalize" else ""
        lines.append(f"# {key} = {prefix}: FETCH {f_kib:.1f} KiB, WRITE {w_kib:.1f} KiB -> {hbm / 1e6:.2f} MB{note}")
        lines.append(f"{key}_hbm_bytes_per_launch: {hbm:.0f}")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


# HBM traffic at L = 3, fp32, across tensor shapes (k = 5) and kernel sizes
# (C = 64, H = W = 256), B = 8: the paper's traffic-invariance measurement
# (appendix on traffic), whose fused design moves a predicted 8.25N elements.
INVARIANCE_CONFIGS = [(8, 32, 512, 512, 5, 3), (8, 64, 256, 256, 5, 3), (8, 128, 128, 128, 5, 3),
                      (8, 64, 256, 256, 3, 3), (8, 64, 256, 256, 7, 3)]


def traffic_invariance_run(dev):
    """One forward per configuration, each after its own input allocation, so
    that the library's dispatches of one configuration form one contiguous run
    between torch's own kernels."""
    import torch

    from paper_2608_10805_amd import binding

    gen = torch.Generator(device=dev)
    for B, C, H, W, k, L in INVARIANCE_CONFIGS:
        gen.manual_seed(0)
        f32 = dict(device=dev, dtype=torch.float32)
        bw = torch.rand(C, k, k, generator=gen, **f32) * 0.4 - 0.2
        bs = torch.rand(C, generator=gen, **f32) + 0.5
        lw = [torch.rand(4 * C, k, k, generator=gen, **f32) * 0.4 - 0.2 for _ in range(L)]
        ls = [torch.rand(4 * C, generator=gen, **f32) * 0.15 + 0.05 for _ in range(L)]
        x = torch.randn(B, C, H, W, generator=gen, **f32)
        y = torch.empty_like(x)
        nbytes = binding.wtconv_forward_workspace_bytes(binding.make_desc(B, C, H, W, k, L, binding._dtype_code(x)))
        ws = torch.empty(max(1, nbytes), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        binding.forward(x, bw, bs, lw, ls, out=y, workspace=ws)
        torch.cuda.synchronize()
        log(f"invariance: forward B={B} C={C} H=W={H} k={k} L={L} done")
        del x, y, ws
        torch.cuda.empty_cache()


def _library_dispatch_groups(db, counter):
    """Per-dispatch totals of `counter` for the library's kernels, grouped into
    runs of consecutive library dispatches (any other kernel ends a run)."""
    rows = _rocpd_rows(db, f"select kernel_name, dispatch_id, sum(value) from counters_collection where "
                           f"counter_name = '{counter}' group by kernel_name, dispatch_id order by dispatch_id")
    groups, cur = [], None
    for name, _, v in rows:
        if "wtc::" in name:
            if cur is None:
                cur = []
                groups.append(cur)
            cur.append(v)
        else:
            cur = None
    return groups


def summarize_invariance(fetch_db, write_db, cfetch_db, cwrite_db, copy_mib, out, command):
    """HBM traffic of each forward of --traffic-invariance-run, all of the
    library's kernels of that forward summed, in units of N fp32 elements."""
    copy_kib = copy_mib * 1024.0
    cf = max((v for k, v in _counter_per_kernel(cfetch_db, "FETCH_SIZE").items() if "copyBuffer" in k), default=0)
    cw = max((v for k, v in _counter_per_kernel(cwrite_db, "WRITE_SIZE").items() if "copyBuffer" in k), default=0)
    fscale, wscale = copy_kib / cf, copy_kib / cw
    fg = _library_dispatch_groups(fetch_db, "FETCH_SIZE")
    wg = _library_dispatch_groups(write_db, "WRITE_SIZE")
    if len(fg) != len(INVARIANCE_CONFIGS) or len(wg) != len(INVARIANCE_CONFIGS):
        raise SystemExit(f"expected {len(INVARIANCE_CONFIGS)} forwards, found {len(fg)} / {len(wg)}")
    lines = ["# HBM traffic of one forward at L = 3, fp32, across tensor shapes and kernel sizes (rocprofv3 counters)",
             f"# commands (one counter per run): {command}",
             f"# calibration: a {copy_mib} MiB device copy reads and writes {copy_kib:.0f} KiB; FETCH_SIZE reports "
             f"{cf:.0f} KiB (scale x{fscale:.3f}), WRITE_SIZE reports {cw:.0f} KiB (scale x{wscale:.3f})",
             "# the paper's fused design: 8.25N predicted; its measurements 8.17N-8.60N",
             f"kernel_source_sha256: {kernel_source_hash()}",
             "# B C H W k L | launches | fetch_N | write_N | total_N"]
    for (B, C, H, W, k, L), f, w in zip(INVARIANCE_CONFIGS, fg, wg):
        n_bytes = 4.0 * B * C * H * W
        fn = sum(f) * 1024 * fscale / n_bytes
        wn = sum(w) * 1024 * wscale / n_bytes
        lines.append(f"{B} {C} {H} {W} {k} {L} | {len(f)} | {fn:.3f} | {wn:.3f} | {fn + wn:.3f}")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")


SQ_COUNTERS = ("SQ_WAVES", "SQ_INSTS_VALU", "SQ_INSTS_LDS", "SQ_INSTS_SALU", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES",
               "SQ_ACTIVE_INST_VALU", "SQ_WAIT_INST_LDS")


def summarize_counters(db, out, command):
    """Instruction counters per launch of the step's forward and gradient
    kernels (one rocprofv3 --pmc run with the eight SQ counters above), set
    against the algorithmic FMA count: each full-lane wavefront FMA does 64 of
    them, and a SIMD issues one wavefront VALU instruction per 4 cycles."""
    from paper_2608_10805_amd import iomodel
    B, C, H, W, k, L = (WORKLOAD[n] for n in ("B", "C", "H", "W", "k", "L"))
    work = iomodel.single_pass_work(B, C, H, W, k, L, "f32")
    per = {name: _counter_per_kernel(db, name) for name in SQ_COUNTERS}
    lines = ["# SQ instruction counters per kernel launch, fused WTConv fwd+bwd benchmark step",
             f"# workload: B={B} C={C} H=W={H} k={k} L={L} fp32 (ConvNeXt-T stage 1), MI355X",
             f"# command: {command}",
             f"workload: {WORKLOAD['workload']}",
             f"kernel_source_sha256: {kernel_source_hash()}"]
    simds = 256 * 4
    for key in ("forward", "grad"):
        prefix = STEP_KERNELS[key]
        vals = {}
        for name in SQ_COUNTERS:
            v = [x for n, x in per[name].items() if prefix in n]
            if v:
                vals[name] = sum(v) / len(v)
        if "SQ_INSTS_VALU" not in vals:
            continue
        fma_wave = work.fma_fwd / 64.0
        issue_cycles = 4.0 * vals["SQ_INSTS_VALU"] / simds
        lines.append(f"# {key} = {prefix}")
        for name in SQ_COUNTERS:
            if name in vals:
                lines.append(f"{key}_{name}: {vals[name]:.0f}")
        lines.append(f"# {key}: algorithmic FMAs {work.fma_fwd:.4g} = {fma_wave:.4g} full-lane wavefront FMAs, "
                     f"{fma_wave / vals['SQ_INSTS_VALU']:.3f} of the VALU instructions issued; VALU issue per SIMD "
                     f"{issue_cycles:.4g} cycles = {issue_cycles / 2.2e3:.1f} us at 2.2 GHz")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    args = parse()
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.out, args.command)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.out, args.command)
        return
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic, args.copy_mib, args.out, args.command)
        return
    if args.summarize_invariance:
        summarize_invariance(*args.summarize_invariance, args.copy_mib, args.out, args.command)
        return
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
    if args.traffic_invariance_run:
        traffic_invariance_run(dev)
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
    bk = binding.Backward(x0, bw, bs, lw, ls, need_dx=False)

    def step(i, ev=None):
        x, dy, y, dx = sets[i % len(sets)]
        if ev is not None:
            ev[0].record()
        binding.forward(x, bw, bs, lw, ls, out=y)
        if ev is not None:
            ev[1].record()
        bk.partials(x, dy, None)
        if ev is not None:
            ev[2].record()
        bk.data(dy, dx)
        if ev is not None:
            ev[3].record()
        bk.finalize()
        if ev is not None:
            ev[4].record()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    log("bench: warmup done")

    # The timed region: K plain steps (no events between the calls).
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        step(i)
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps
    # The same K steps again with an event between every two calls, on the
    # library's stream, for each kernel's duration. The five event records add
    # a few microseconds per call, so this pass is not the step time.
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        step(i, evs[i])
    torch.cuda.synchronize()
    per_step = [e[0].elapsed_time(e[4]) for e in evs]
    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    grad_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    data_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    fin_ms = float(np.mean([e[3].elapsed_time(e[4]) for e in evs]))
    log(f"bench: {ms_step * 1e3:.1f} us/step; with events between the calls {np.mean(per_step) * 1e3:.1f} us = "
        f"forward {fwd_ms * 1e3:.1f}, kernel-gradient pass {grad_ms * 1e3:.1f}, dx pass {data_ms * 1e3:.1f}, "
        f"finalize {fin_ms * 1e3:.1f}")

    work = iomodel.single_pass_work(B, C, H, W, k, L, "f32")
    value = work.bytes_fwdbwd / (ms_step * 1e-3) / 1e9
    # Kernels of the step for this workload (each entry point is one launch
    # here): the fused forward kernel runs twice (y, and dx on dy with rotated
    # kernels), the kernel-gradient pass once. Algorithmic work per launch:
    # the forward k^2 (N + coefficient sites) FMAs, moving x (or dy) in and y
    # (or dx) out; the gradient pass the same FMA count, reading x and dy.
    N = B * C * H * W
    fwd_bytes = 2.0 * N * 4 + 4.0 * iomodel.param_count(C, k, L)
    kernels = {
        "forward": {"launches_per_step": 2, "ms": (fwd_ms + data_ms) / 2, "fma": work.fma_fwd, "bytes": fwd_bytes},
        "grad": {"launches_per_step": 1, "ms": grad_ms, "fma": work.fma_fwd, "bytes": fwd_bytes},
    }
    for kv in kernels.values():
        kv["TFLOPs"] = round(2.0 * kv["fma"] / (kv["ms"] * 1e-3) / 1e12, 3)
        kv["fma_frac"] = round(iomodel.fma_floor_s(kv["fma"]) / (kv["ms"] * 1e-3), 4)
        kv["GBps"] = round(kv["bytes"] / (kv["ms"] * 1e-3) / 1e9, 1)
        kv["ms"] = round(kv["ms"], 5)
    kernels["finalize"] = {"launches_per_step": 1, "ms": round(fin_ms, 5)}
    dom = max(("forward", "grad"), key=lambda n: kernels[n]["ms"] * kernels[n]["launches_per_step"])
    dom_ms, dom_fma, dom_bytes = kernels[dom]["ms"], kernels[dom]["fma"], kernels[dom]["bytes"]
    achieved = 2.0 * dom_fma / (dom_ms * 1e-3) / 1e12
    peak = iomodel.FP32_FLOPS / 1e12
    traffic = load_traffic(args.traffic, dom)
    copy_gbps = copy_ceiling_gbps(dev)
    probe = valu_probe(dev)
    log(f"bench: copy ceiling {copy_gbps:.0f} GB/s, VALU probe {probe}")
    roofline = {"bound": "alu", "achieved": round(achieved, 3), "peak": round(peak, 1), "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": traffic, "kernel": dom,
                "kernel_ms": round(dom_ms, 5),
                "hbm_view": {"algorithmic_bytes": dom_bytes,
                             "achieved_GBps": round(dom_bytes / (dom_ms * 1e-3) / 1e9, 1),
                             "frac": round(dom_bytes / (dom_ms * 1e-3) / 1e9 / iomodel.HBM_PEAK_GBPS, 4)}}
    table = None
    memory = None
    if not args.no_config_table:
        table = config_table(args.table_steps, dev)
        memory = memory_table(dev)
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        refs, cpu = cpu_baseline(inp, work.bytes_fwdbwd, args.cpu_seconds)
        parity = full_size_parity(refs, x0, dy0, bw, bs, lw, ls)
        log(f"parity vs the float64 oracle (whole workload): {parity}")
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic (seeded; x, dy ~ N(0,1), weights U(-0.2,0.2))",
        "config": dict(WORKLOAD),
        "hbm_frac": round(value / iomodel.HBM_PEAK_GBPS, 4),
        "ms_mean": round(ms_step, 5),
        "instrumented_step_ms": {"mean": round(float(np.mean(per_step)), 5),
                                 "median": round(float(np.median(per_step)), 5),
                                 "min": round(float(np.min(per_step)), 5)},
        "copy_ceiling_GBps": round(copy_gbps, 1), "hbm_frac_of_copy": round(value / copy_gbps, 4),
        "valu_probe": probe,
        "fma_frac": round(iomodel.fma_floor_s(work.fma_fwdbwd) / (ms_step * 1e-3), 4),
        "fwd_ms": round(fwd_ms, 5), "bwd_ms": round(grad_ms + data_ms + fin_ms, 5), "kernels": kernels,
        "algorithmic_bytes_per_step": work.bytes_fwdbwd,
        "floors_us": {"hbm": round(iomodel.hbm_floor_s(work.bytes_fwdbwd) * 1e6, 2),
                      "fp32_fma": round(iomodel.fma_floor_s(work.fma_fwdbwd) * 1e6, 2)},
        "paper_io_model_elems_per_N": {"Q_ref": round(iomodel.q_ref(L), 3), "Q_fused": round(iomodel.q_fused(L), 3),
                                       "single_pass_fwd": 2, "single_pass_fwdbwd": 5,
                                       "rocprof_dominant_kernel": (round(traffic / (N * 4), 3)
                                                                   if traffic is not None else None)},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "parity": parity,
        "N": N,
        "configs": table,
        "paper_layer_sweep_geomean": paper_sweep_summary(table) if table else None,
        "paper_layer_sweep_peak_memory": memory,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
