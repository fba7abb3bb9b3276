"""Host logic of bench.py (no GPU): the reducers that turn rocprofv3 kernel
traces and counter collections into the committed summaries, checked on
small synthetic CSV files, and the single-GPU guard."""
import argparse
import csv
import json
import os
import subprocess
import sys

import pytest

import bench

COUNTER_COLS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id",
                "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size",
                "VGPR_Count", "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value",
                "Start_Timestamp", "End_Timestamp"]
STAGE = "void ios::ios_stage_kernel<0, false>(HIP_vector_type<int, 4u> const*, int, ios::StageArgs)"


def args(config="tiny", batch=1):
    return argparse.Namespace(config=config, batch=batch, seed=0)


def counter_dir(tmp_path, name, rows, meta):
    """rows: (kernel, {counter: value}, workgroups, start, end) in dispatch order."""
    d = tmp_path / name
    d.mkdir()
    with open(d / "run_counter_collection.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(COUNTER_COLS)
        for i, (kern, counters, wg, t0, t1) in enumerate(rows, start=1):
            for c, v in counters.items():
                w.writerow([i, i, 1, 1, 1, 1, wg * 512, 1, kern, 512, 0, 0, 64, 0, 32, c, v, t0, t1])
    (d / "bench.json").write_text(json.dumps(meta))
    return str(d)


def test_trace_summary_takes_the_timed_loop_per_stage(tmp_path, capsys):
    d = tmp_path / "trace"
    d.mkdir()
    rows, t = [], 0
    # a tuning launch, then 2 steps of 3 stages; stage k lasts 100 (k + 1) + step ns
    for step, k in [(None, 0)] + [(s, k) for s in range(2) for k in range(3)]:
        dur = 5000 if step is None else 100 * (k + 1) + step
        rows.append((t, t + dur, 300 + k))
        t += dur + 10
    with open(d / "run_kernel_trace.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X"])
        for t0, t1, wg in rows:
            w.writerow([STAGE, t0, t1, wg * 512])
    sched = [{"units": u, "strategy": "concurrent"} for u in (["A"], ["B1"], ["B2"])]
    (d / "bench.json").write_text(json.dumps({"steps": 2, "stages": 3, "value": 1.0, "schedule": sched,
                                              "kernel_sha": "abc"}))
    bench.trace_summary(args(), str(d), out_dir=str(tmp_path))
    out = json.loads(capsys.readouterr().out)
    assert out["launches"] == 6
    assert [p["median_ns"] for p in out["per_stage"]] == [100.5, 200.5, 300.5]
    assert [p["workgroups"] for p in out["per_stage"]] == [300, 301, 302]
    assert [p["units"] for p in out["per_stage"]] == [["A"], ["B1"], ["B2"]]
    assert out["median_gap_ns"] == 10
    # mean duration 200.5 ns; period = (last end - first start) / 6 = (1261 - 50) / 6... from the rows
    t_first, t_last = rows[1][0], rows[-1][1]
    assert out["mean_period_ns"] == round((t_last - t_first) / 6, 1)
    alg = bench.unit_work(bench_spec_tiny(), 1)
    mfma = sum(v[0] for v in alg.values())
    assert out["frac_from_trace"] == round(mfma / 3 / 200.5 / 1e3 / bench.PEAK_FP32_TFLOPS, 5)
    assert json.load(open(tmp_path / "trace_tiny_bs1.json"))["kernel_sha"] == "abc"


def bench_spec_tiny():
    import workloads as W
    return W.make("tiny")[0]


def test_write_traffic_scales_by_the_copy(tmp_path):
    sched = [{"units": ["A"], "strategy": "concurrent"}, {"units": ["B"], "strategy": "concurrent"}]
    meta = {"steps": 2, "stages": 2, "copy_mb": 1, "schedule": sched}
    dirs = []
    for c, base in (("FETCH_SIZE", 100.0), ("WRITE_SIZE", 10.0)):
        rows = [(STAGE, {c: 999.0}, 10, 0, 1)]                       # warm-up, not timed
        rows += [(STAGE, {c: base * (k + 1)}, 10, 0, 1) for _ in range(2) for k in range(2)]
        rows += [("__amd_rocclr_copyBuffer", {c: 512.0}, 10, 0, 1)]  # 1 MiB copy read as 512 KiB
        dirs.append(counter_dir(tmp_path, c, rows, meta))
    bench.write_traffic(args(), *dirs, out_dir=str(tmp_path))
    out = json.load(open(tmp_path / "traffic_tiny_bs1.json"))
    assert out["fetch"]["scale"] == pytest.approx(2.0)
    assert out["fetch"]["bytes_per_launch"] == pytest.approx(150.0 * 1024 * 2)
    assert out["traffic_bytes_per_launch"] == pytest.approx(165.0 * 1024 * 2)
    assert [p["fetch_bytes"] for p in out["per_stage"]] == [100 * 2048, 200 * 2048]
    assert [p["write_bytes"] for p in out["per_stage"]] == [10 * 2048, 20 * 2048]


def test_write_occupancy_weights_by_active_cycles(tmp_path):
    def run(name, stages, occ, act):
        meta = {"steps": 2, "stages": stages,
                "schedule": [{"units": [f"s{k}"], "strategy": "concurrent"} for k in range(stages)]}
        rows = [(STAGE, {"MeanOccupancyPerCU": 50.0, "GRBM_GUI_ACTIVE": 1.0}, 7, 0, 1)]   # not timed
        rows += [(STAGE, {"MeanOccupancyPerCU": occ[k], "GRBM_GUI_ACTIVE": act[k]}, 100 + k, 0, 1000)
                 for _ in range(2) for k in range(stages)]
        return counter_dir(tmp_path, name, rows, meta)
    ios = run("ios", 2, [6.0, 3.0], [100.0, 300.0])
    seq = run("seq", 3, [2.0, 2.0, 2.0], [50.0, 60.0, 70.0])
    bench.write_occupancy(args(), ios, seq, out_dir=str(tmp_path))
    out = json.load(open(tmp_path / "occupancy_tiny_bs1.json"))
    assert out["ios"]["mean_waves_per_cu"] == pytest.approx((6 * 100 + 3 * 300) / 400)
    assert out["sequential"]["mean_waves_per_cu"] == pytest.approx(2.0)
    assert out["ios_over_sequential"] == pytest.approx(3.75 / 2.0, abs=1e-3)
    assert [p["workgroups"] for p in out["ios"]["per_stage"]] == [100, 101]
    assert out["ios"]["per_stage"][0]["dispatch_us"] == pytest.approx(1.0)


def test_write_mfma_compares_with_the_algorithmic_flops(tmp_path):
    # tiny block: A = 1x1 16->16, B1 = 1x1 16->8, B2 = 3x3 8->16, all on 8x8
    alg = {"A": 2 * 64 * 16 * 16, "B1": 2 * 64 * 8 * 16, "B2": 2 * 64 * 16 * 72}
    sched = [{"units": ["A", "B1"], "strategy": "merge"}, {"units": ["B2"], "strategy": "concurrent"}]
    counted = [(alg["A"] + alg["B1"]) * 1.5, alg["B2"]]
    rows = [(STAGE, {"SQ_INSTS_VALU_MFMA_MOPS_F32": c / 512, "SQ_INSTS_VALU_MFMA_F32": c / 2048}, 4, 0, 1)
            for _ in range(3) for c in counted]
    d = counter_dir(tmp_path, "mfma", rows, {"steps": 3, "stages": 2, "schedule": sched})
    bench.write_mfma(args(), d, out_dir=str(tmp_path))
    out = json.load(open(tmp_path / "mfma_tiny_bs1.json"))
    assert [p["algorithmic_flop"] for p in out["per_stage"]] == [alg["A"] + alg["B1"], alg["B2"]]
    assert [p["counted_over_algorithmic"] for p in out["per_stage"]] == [1.5, 1.0]
    assert out["per_stage"][1]["mfma_instructions"] == pytest.approx(alg["B2"] / 2048)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(bench.ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
