"""Host-side logic of bench.py (no GPU): the one-GPU guard, the rocprofv3
summaries and the traffic lookup that gates `roofline.traffic`."""
import os
import sqlite3
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

FWD = "void wtc::(anonymous namespace)::fused_kernel<5, float, false, true, false>(wtc::FusedArgs)"
GRAD = "void wtc::(anonymous namespace)::grad_kernel<5, float, false>(wtc::GradArgs)"
RED = "wtc::(anonymous namespace)::reduce_kernel(wtc::ReduceArgs)"
COPY = "__amd_rocclr_copyBuffer"


def _trace_db(path, rows):
    con = sqlite3.connect(path)
    con.execute("create table kernels (name text, duration integer)")
    con.executemany("insert into kernels values (?, ?)", rows)
    con.commit()
    con.close()
    return str(path)


def _counter_db(path, counter, per_kernel):
    """per_kernel: {kernel name: [value per dispatch]}; each dispatch's value is
    split over two rows (as per-XCD rows are) to exercise the summation."""
    con = sqlite3.connect(path)
    con.execute("create table counters_collection (kernel_name text, dispatch_id integer, counter_name text, "
                "value real)")
    disp = 0
    for name, values in per_kernel.items():
        for v in values:
            disp += 1
            con.execute("insert into counters_collection values (?, ?, ?, ?)", (name, disp, counter, v / 2))
            con.execute("insert into counters_collection values (?, ?, ?, ?)", (name, disp, counter, v / 2))
    con.commit()
    con.close()
    return str(path)


def _kv(path):
    rec = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    return rec


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


WL = bench.HEADLINE


def test_summarize_trace(tmp_path):
    db = _trace_db(tmp_path / "t.db", [(FWD, 70000), (FWD, 72000), (GRAD, 90000), (RED, 4000)])
    out = tmp_path / "trace.txt"
    bench.summarize_trace(db, str(out), "the command", WL, 1)
    text = out.read_text()
    assert "# command: the command" in text
    rec = _kv(out)
    assert rec["kernel_source_sha256"] == bench.kernel_source_hash()
    assert rec["workload"] == WL
    fwd_line = [ln for ln in text.splitlines() if ln.startswith("fused_kernel<5, float, false, true, false>")][0]
    name, calls, per_step, total, avg, pct = [f.strip() for f in fwd_line.split("|")]
    assert (calls, per_step, total, avg) == ("2", "2.00", "142.0", "71.000")
    assert abs(float(pct) - 100.0 * 142 / 236) < 0.06
    assert bench.load_trace_avg_us(str(out), WL, bench.STEP_KERNELS["forward"]) == pytest.approx(71.0)
    assert bench.load_trace_avg_us(str(out), "other", bench.STEP_KERNELS["forward"]) is None


def test_summarize_traffic_scales_by_the_copy(tmp_path):
    # the copy reads 256 MiB but FETCH_SIZE shows half of it; WRITE_SIZE all of it
    kib = 256 * 1024.0
    fetch = _counter_db(tmp_path / "f.db", "FETCH_SIZE", {FWD: [1000.0, 1000.0], GRAD: [3000.0], RED: [4.0]})
    write = _counter_db(tmp_path / "w.db", "WRITE_SIZE", {FWD: [500.0, 500.0], GRAD: [10.0], RED: [2.0]})
    cfetch = _counter_db(tmp_path / "cf.db", "FETCH_SIZE", {COPY: [kib / 2]})
    cwrite = _counter_db(tmp_path / "cw.db", "WRITE_SIZE", {COPY: [kib]})
    out = tmp_path / "traffic.txt"
    bench.summarize_traffic(fetch, write, cfetch, cwrite, 256, str(out), "cmd", WL, 1)
    rec = _kv(out)
    assert float(rec["fetch_scale"]) == pytest.approx(2.0)
    assert float(rec["write_scale"]) == pytest.approx(1.0)
    fwd = (2 * 1000 + 500) * 1024
    grad = (2 * 3000 + 10) * 1024
    red = (2 * 4 + 2) * 1024
    assert float(rec["bytes_per_launch fused_kernel<5, float, false, true, false>"]) == pytest.approx(fwd, rel=1e-9)
    assert float(rec["bytes_per_launch grad_kernel<5, float, false>"]) == pytest.approx(grad, rel=1e-9)
    # one profiled step: the forward kernel twice, the others once
    step = 2 * fwd + grad + red
    assert float(rec["step_hbm_bytes"]) == pytest.approx(step, rel=1e-6)
    B, C, H, W, k, L, dt = bench.WORKLOADS[WL]
    assert float(rec["step_hbm_elems_per_N"]) == pytest.approx(step / (4.0 * B * C * H * W), abs=1e-4)


def test_traffic_lookup_needs_current_sources(tmp_path):
    kib = 1024.0
    fetch = _counter_db(tmp_path / "f.db", "FETCH_SIZE", {FWD: [100.0]})
    write = _counter_db(tmp_path / "w.db", "WRITE_SIZE", {FWD: [100.0]})
    cfetch = _counter_db(tmp_path / "cf.db", "FETCH_SIZE", {COPY: [kib]})
    cwrite = _counter_db(tmp_path / "cw.db", "WRITE_SIZE", {COPY: [kib]})
    out = tmp_path / "traffic.txt"
    bench.summarize_traffic(fetch, write, cfetch, cwrite, 1, str(out), "cmd", WL, 1)
    fwd = bench.STEP_KERNELS["forward"]
    assert bench.load_traffic(str(out), WL, fwd) == pytest.approx(200 * 1024)
    assert bench.load_traffic(str(out), WL) == pytest.approx(200 * 1024)
    assert bench.load_traffic(str(out), WL, bench.STEP_KERNELS["grad"]) is None  # no counters for it
    assert bench.load_traffic(str(out), "another_workload", fwd) is None
    stale = out.read_text().replace(bench.kernel_source_hash(), "0" * 64)
    out.write_text(stale)
    assert bench.load_traffic(str(out), WL, fwd) is None
    assert bench.load_traffic(str(tmp_path / "missing.txt"), WL, fwd) is None


def test_summarize_counters(tmp_path):
    per = {n: {FWD: [v], GRAD: [2 * v]} for n, v in zip(bench.SQ_COUNTERS, range(1, 9))}
    con = sqlite3.connect(tmp_path / "sq.db")
    con.execute("create table counters_collection (kernel_name text, dispatch_id integer, counter_name text, "
                "value real)")
    disp = 0
    for name, kv in per.items():
        for kern, vals in kv.items():
            for v in vals:
                disp += 1
                con.execute("insert into counters_collection values (?, ?, ?, ?)", (kern, disp, name, float(v)))
    con.commit()
    con.close()
    out = tmp_path / "sq.txt"
    bench.summarize_counters(str(tmp_path / "sq.db"), str(out), "cmd", WL)
    rec = _kv(out)
    assert float(rec["SQ_INSTS_VALU fused_kernel<5, float, false, true, false>"]) == per["SQ_INSTS_VALU"][FWD][0]
    assert float(rec["SQ_INSTS_VALU grad_kernel<5, float, false>"]) == per["SQ_INSTS_VALU"][GRAD][0]
    assert rec["kernel_source_sha256"] == bench.kernel_source_hash()


def _fake_rows():
    rows = []
    for i, (name, B, C, H, W, k, L, dt) in enumerate(bench.table_configs()):
        rows.append({"name": name, "B": B, "C": C, "H": H, "W": W, "k": k, "L": L, "dtype": dt,
                     "fwd_ms": 0.1234 + i * 1e-4, "fwdbwd_ms": 0.4567 + i * 1e-4, "fwd_GBps": 1234.5,
                     "fwdbwd_GBps": 2345.6, "fwd_hbm_frac": 0.1543, "fwdbwd_hbm_frac": 0.2932,
                     "fwd_fma_frac": 0.4, "fwdbwd_fma_frac": 0.41})
    return rows


def test_configs_summary_covers_every_sweep_point_compactly():
    """The headline line carries every (shape, dtype, L = 1..5) point of the
    shape sweep and stays a few KB, so the whole line survives a tail of the
    benchmark's output."""
    import json
    memory = {dt: [{"L": L, "train_peak_over_compulsory": 1.2, "infer_peak_over_compulsory": 1.3}
                   for L in range(1, 6)] for dt in ("f32", "f16")}
    s = bench.configs_summary(_fake_rows(), memory)
    sweep = s["sweep_us_L1to5"]
    assert len(sweep) == 2 * len(bench.SWEEP_SHAPES)
    for v in sweep.values():
        assert len(v["fwd"]) == len(v["fb"]) == 5
    assert len(s["stage2_f32_fb_us_L1to5"]) == 5
    assert set(s["paper_sweep_geomean_us_L1to5"]) == {"k5_f32", "k5_f16", "k3_f32", "k3_f16"}
    assert len(json.dumps(s, separators=(",", ":"))) < 2000


def test_table_has_every_sweep_level():
    names = {c[0] for c in bench.table_configs()}
    for (B, C, H, W) in bench.SWEEP_SHAPES:
        for dt in ("f32", "bf16"):
            for L in range(1, 6):
                assert f"sweep_{H}x{W}_c{C}_L{L}_{dt}" in names


def test_summarize_invariance_groups_each_forward(tmp_path):
    """Library dispatches between torch kernels form one forward each; the
    summary divides their scaled bytes by 4N."""
    kib = 64 * 1024.0
    n_cfg = len(bench.INVARIANCE_CONFIGS)

    def db(path, counter, per_forward):
        con = sqlite3.connect(path)
        con.execute("create table counters_collection (kernel_name text, dispatch_id integer, counter_name text, "
                    "value real)")
        disp = 0
        for f in range(n_cfg):
            disp += 1
            con.execute("insert into counters_collection values (?, ?, ?, ?)", ("at::randn_kernel", disp, counter, 5.0))
            for v in per_forward[f]:
                disp += 1
                con.execute("insert into counters_collection values (?, ?, ?, ?)", (FWD, disp, counter, v))
        con.commit()
        con.close()
        return str(path)

    # forward f: two library launches (e.g. carrier + fused pass)
    fetch = db(tmp_path / "f.db", "FETCH_SIZE", [[100.0 * (f + 1), 50.0] for f in range(n_cfg)])
    write = db(tmp_path / "w.db", "WRITE_SIZE", [[10.0, 20.0 * (f + 1)] for f in range(n_cfg)])
    cfetch = _counter_db(tmp_path / "cf.db", "FETCH_SIZE", {COPY: [kib / 2]})
    cwrite = _counter_db(tmp_path / "cw.db", "WRITE_SIZE", {COPY: [kib]})
    out = tmp_path / "inv.txt"
    bench.summarize_invariance(fetch, write, cfetch, cwrite, 64, str(out), "cmd")
    rows = [ln for ln in out.read_text().splitlines() if ln and not ln.startswith("#") and "|" in ln]
    assert len(rows) == n_cfg
    for f, (row, cfg) in enumerate(zip(rows, bench.INVARIANCE_CONFIGS)):
        B, C, H, W, k, L = cfg
        fields = [x.strip() for x in row.split("|")]
        assert fields[0].split() == [str(v) for v in cfg]
        assert fields[1] == "2"
        n_bytes = 4.0 * B * C * H * W
        want_f = 2 * (100.0 * (f + 1) + 50.0) * 1024 / n_bytes
        want_w = (10.0 + 20.0 * (f + 1)) * 1024 / n_bytes
        assert float(fields[2]) == pytest.approx(want_f, abs=6e-4)
        assert float(fields[3]) == pytest.approx(want_w, abs=6e-4)


def test_summarize_invariance_rejects_a_missing_forward(tmp_path):
    con = sqlite3.connect(tmp_path / "f.db")
    con.execute("create table counters_collection (kernel_name text, dispatch_id integer, counter_name text, "
                "value real)")
    con.execute("insert into counters_collection values (?, ?, ?, ?)", (FWD, 1, "FETCH_SIZE", 1.0))
    con.commit()
    con.close()
    cf = _counter_db(tmp_path / "cf.db", "FETCH_SIZE", {COPY: [1.0]})
    cw = _counter_db(tmp_path / "cw.db", "WRITE_SIZE", {COPY: [1.0]})
    with pytest.raises(SystemExit):
        bench.summarize_invariance(str(tmp_path / "f.db"), str(tmp_path / "f.db"), cf, cw, 1,
                                   str(tmp_path / "o.txt"), "cmd")


def test_paper_sweep_summary_geomeans():
    rows = []
    for name, B, C, H, W, k, L, dt in bench.table_configs():
        if name.startswith("paper_"):
            rows.append({"name": name, "k": k, "dtype": dt, "L": L, "fwd_ms": float(C) / 32 * (H / 128),
                         "fwdbwd_ms": 2.0})
    s = bench.paper_sweep_summary(rows)
    # geometric mean of (C/32) * (H/128) over C in {32,64,128}, H in {128,256,512} = 2 * 2
    assert s["k3"]["f32"][0]["fwd_ms"] == pytest.approx(4.0)
    assert s["k5"]["f16"][4]["fwdbwd_ms"] == pytest.approx(2.0)
    assert s["k3"]["f16"][2]["paper_a6000_fwd_ms"] == 1.205
    assert len(s["k5"]["f32"]) == 5
