"""Benchmark: batch-1 latency of IOS-scheduled multi-branch CNN blocks on one
MI355X, with achieved fp32 TFLOP/s of the stage kernel against the MFMA peak.

One *step* is one ``ios_run`` of the whole workload (every stage of the
schedule found by Algorithm 1 with on-device profiling) on inputs already
resident in HBM.  Default workload: the SqueezeNet-style stack of eight fire
modules (96x55x55 -> 512x13x13), batch 1, seed 0 -- the largest of the
batch-1 configurations (1.14 GFLOP); the other four batch-1 configurations
are measured the same way and reported beside it.

Printed as one JSON line (N = 1 only):
  value        median over 5 equal windows of the K timed steps (HIP events
               on the launch stream), microseconds per step
  roofline     the stage kernel: algorithmic MFMA flops per launch / the
               mean launch duration over the timed region (step time /
               launches per step), vs the fp32 MFMA peak
  baselines    the same kernels under the sequential (one unit per launch)
               and greedy schedules, timed the same way
  cpu_baseline the oracle (plain fp64 C loops, one thread) on the host
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_TFLOPS = 157.3          # MI355X dense fp32 MFMA (256 CU x 2.4 GHz x 256 flop/clk)
PEAK_HBM_GBS = 8000.0
KERNEL_SOURCES = ["paper_2011_01302_amd/csrc/" + f for f in (
    "stage_kernel.h", "stage_kernel_full.hip", "stage_kernel_full_persist.hip", "stage_kernel_sep.hip",
    "stage_kernel_sep_persist.hip", "stage_kernel_seprow.hip", "stage_kernel_seprow_persist.hip",
    "stage_kernel_pipe.hip", "stage_kernel_pipe_persist.hip", "stage_kernel_light.hip",
    "stage_kernel_light_persist.hip",
    "stage_launch.cpp", "exec.cpp", "ios_internal.h")]


def kernel_sha() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


# ------------------------------------------------------------------ algorithmic work

def unit_work(spec, batch):
    """Per unit: (MFMA flops, VALU flops, weight bytes) — algorithmic, i.e.
    2 x MAC of the operator as defined, no padding of merged kernels."""
    import workloads as W
    shp = W.infer_shapes(spec)
    out = {}
    for op in W.unit_ops(spec):
        c, h, w = shp[op["in"][0]]
        co, ho, wo = shp[op["name"]]
        px = batch * ho * wo
        k = op["kind"]
        if k == "conv":
            out[op["name"]] = (2 * px * co * c * op["kh"] * op["kw"], 0, 4 * (co * c * op["kh"] * op["kw"] + co))
        elif k == "sepconv":
            out[op["name"]] = (2 * px * co * c, 2 * px * c * op["kh"] * op["kw"] + px * c * (len(op["in"]) - 1),
                               4 * (c * op["kh"] * op["kw"] + co * c + co))
        elif k in ("maxpool", "avgpool"):
            out[op["name"]] = (0, px * co * op["kh"] * op["kw"], 0)
        else:
            out[op["name"]] = (0, px * co * len(op["in"]), 0)
    return out


def stage_bytes(spec, batch, names):
    """Compulsory HBM bytes of a stage: inputs from outside it read once,
    every unit output written once, weights read once."""
    import workloads as W
    shp = W.infer_shapes(spec)
    units = {op["name"]: op for op in W.unit_ops(spec)}
    views = {op["name"]: op for op in spec["ops"] if op["kind"] in ("concat", "identity")}

    def sources(t):
        if t in views:
            s = []
            for i in views[t]["in"]:
                s += sources(i)
            return s
        return [t]
    ext = set()
    for n in names:
        for t in units[n]["in"]:
            for s in sources(t):
                if s not in names:
                    ext.add(s)
    by = sum(4 * batch * shp[t][0] * shp[t][1] * shp[t][2] for t in ext)
    by += sum(4 * batch * shp[n][0] * shp[n][1] * shp[n][2] for n in names)
    return by


# ------------------------------------------------------------------ timing

def conv_tiles(I, g):
    """The graph's current conv tile shapes, {unit id: shape}."""
    return {g.tid[op["name"]]: I.ios_get_conv_tile(g.handle, g.tid[op["name"]])
            for op in g.spec["ops"] if op["kind"] == "conv"}


def tune_for(I, g, q, iso):
    """Start from the shapes each conv chose alone (iso), then pick shapes per
    stage of q; returns the stages' summed measured latency (ns)."""
    for u, t in iso.items():
        I.ios_set_conv_tile(g.handle, u, t)
    return I.ios_schedule_tune_tiles(g.handle, q)


def time_steps(I, g, q, ins, outs, stream, warmup, steps, torch):
    return statistics.mean(timed_repeats(I, g, q, ins, outs, stream, warmup, steps, torch, 1))


def timed_repeats(I, g, q, ins, outs, stream, warmup, steps, torch, repeats=5):
    """`warmup` untimed runs, then `steps` back-to-back ios_runs split into
    `repeats` equal windows between HIP events recorded on the launch stream
    (torch's current stream, which ios_run is given); us per step of each
    window."""
    ip = [t.data_ptr() for t in ins]
    op = [t.data_ptr() for t in outs]
    for _ in range(warmup):
        I.ios_run(g.handle, q, ip, op, stream)
    torch.cuda.synchronize()
    per = steps // repeats
    assert per * repeats == steps and per > 0, "steps must be a positive multiple of repeats"
    s = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(repeats + 1)]
    ev[0].record(s)
    for r in range(repeats):
        for _ in range(per):
            I.ios_run(g.handle, q, ip, op, stream)
        ev[r + 1].record(s)
    torch.cuda.synchronize()
    return [ev[r].elapsed_time(ev[r + 1]) * 1e3 / per for r in range(repeats)]


def unit_tiling(I, g):
    """Every unit's tuning choices, {name: [tile, xcd_lg]} (for replays)."""
    return {op["name"]: list(I.ios_get_unit_tiling(g.handle, g.tid[op["name"]]))
            for op in g.spec["ops"] if op["kind"] not in ("concat", "identity")}


def set_unit_tiling(I, g, tiling):
    for name, (tile, lg) in tiling.items():
        I.ios_set_unit_tiling(g.handle, g.tid[name], tile, lg)


def stage_times(I, g, q, ins, outs, stream, reps):
    """Per-stage GPU ns (median over reps) from HIP events recorded around
    each stage launch on the launch stream."""
    ip = [t.data_ptr() for t in ins]
    op = [t.data_ptr() for t in outs]
    n = len(I.ios_schedule_get(q))
    rows = [I.ios_run_timed(g.handle, q, ip, op, stream, n) for _ in range(reps)]
    return [statistics.median(r[k] for r in rows) for k in range(n)], rows


def host_cpu():
    """CPU model and logical CPU count of the host the oracle ran on."""
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"model": model, "logical_cpus": os.cpu_count()}


def cpu_oracle(spec, ten, budget_s):
    from oracle import evaluator as E
    E.build()
    E.outputs(spec, ten)                                 # warm (loads the library)
    n, t0 = 0, time.perf_counter()
    while True:
        E.outputs(spec, ten)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s or n >= 50:
            break
    return el / n * 1e6, n


def load_traffic(workload, sha):
    p = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(p):
        return None
    d = json.load(open(p))
    if d.get("kernel_sha") != sha:
        return None
    return d.get("traffic_bytes_per_launch")


def recorded_plan(config, batch):
    """The plan recorded under profiles/ for this configuration (schedule and
    tuning choices of a DP search on an MI355X, with the kernel sources it
    was taken with), or (None, None) when there is none for the current
    sources."""
    p = os.path.join(ROOT, "profiles", f"plan_{config}_bs{batch}.json")
    if not os.path.exists(p):
        return None, None
    plan = [json.loads(l) for l in open(p) if l.startswith("{") and '"tiling"' in l][-1]
    if plan.get("kernel_sha") != kernel_sha():
        return None, None
    return plan, p


def load_trace(workload, sha):
    """Kernel-trace summary of the same plan (profiles/trace_<workload>.json)
    when it was taken from the current kernel sources."""
    p = os.path.join(ROOT, "profiles", f"trace_{workload}.json")
    if not os.path.exists(p):
        return None
    d = json.load(open(p))
    if d.get("kernel_sha") != sha:
        return None
    return {k: d.get(k) for k in ("mean_ns", "mean_period_ns", "median_gap_ns", "frac_from_trace")}


def _pmc_rows(d, counter):
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r.get("Counter_Name") == counter:
                rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    rows.sort()
    return rows


def write_traffic(args, fetch_dir, write_dir, out_dir=None):
    """HBM bytes per stage launch of the timed loop, from rocprofv3 --pmc
    FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by what the
    same counter reads for the plain copy of --copy-mb MiB at the end of the
    run.  The timed loop is the last steps x stages stage-kernel dispatches
    before that copy."""
    res = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _pmc_rows(d, counter)
        copy = [v for _, k, v in rows if "ios_stage_kernel" not in k][-1]
        stage = [v for _, k, v in rows if "ios_stage_kernel" in k]
        meta = json.load(open(os.path.join(d, "bench.json")))
        n = meta["steps"] * meta["stages"]
        timed = stage[-n:]
        copy_bytes = meta["copy_mb"] << 20
        scale = copy_bytes / (copy * 1024.0)
        ns = meta["stages"]
        res[counter] = {"kib_per_launch_raw": sum(timed) / len(timed), "copy_kib_raw": copy,
                        "scale": scale, "bytes_per_launch": sum(timed) / len(timed) * 1024.0 * scale,
                        "per_stage_bytes": [statistics.mean(timed[k::ns]) * 1024.0 * scale for k in range(ns)]}
    out = {"workload": f"{args.config}_bs{args.batch}", "kernel_sha": kernel_sha(),
           "fetch": res["FETCH_SIZE"], "write": res["WRITE_SIZE"],
           "traffic_bytes_per_launch": res["FETCH_SIZE"]["bytes_per_launch"] + res["WRITE_SIZE"]["bytes_per_launch"]}
    sched = json.load(open(os.path.join(fetch_dir, "bench.json"))).get("schedule")
    if sched:
        out["per_stage"] = [{"units": st["units"], "strategy": st["strategy"],
                             "fetch_bytes": round(f), "write_bytes": round(w)}
                            for st, f, w in zip(sched, res["FETCH_SIZE"]["per_stage_bytes"],
                                                res["WRITE_SIZE"]["per_stage_bytes"])]
    path = os.path.join(out_dir or os.path.join(ROOT, "profiles"), f"traffic_{args.config}_bs{args.batch}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def write_mfma(args, d, out_dir=None):
    """fp32 MFMA work the hardware counted per stage launch of the timed loop
    (rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_INSTS_VALU_MFMA_F32: add
    and mul ops / 512, and MFMA instructions) against the stages' algorithmic
    MFMA flops (2 x MAC of the convolutions as defined).  The excess is the
    padding the kernel multiplies by zero: output channels to multiples of 16,
    input channels to multiples of 4 and the reduction to multiples of 16,
    pixel rows of the last M-tile, and the zero taps of merged kernels."""
    import workloads as W
    meta = json.load(open(os.path.join(d, "bench.json")))
    ns, steps = meta["stages"], meta["steps"]
    mops = [v for _, k, v in _pmc_rows(d, "SQ_INSTS_VALU_MFMA_MOPS_F32") if "ios_stage_kernel" in k][-steps * ns:]
    inst = [v for _, k, v in _pmc_rows(d, "SQ_INSTS_VALU_MFMA_F32") if "ios_stage_kernel" in k][-steps * ns:]
    spec, _ = W.make(args.config, args.batch, args.seed)
    work = unit_work(spec, args.batch)
    rows = []
    for k in range(ns):
        units = meta["schedule"][k]["units"]
        alg = sum(work[n][0] for n in units)
        counted = statistics.mean(mops[k::ns]) * 512
        rows.append({"units": units, "strategy": meta["schedule"][k]["strategy"],
                     "algorithmic_flop": alg, "counted_flop": counted,
                     "mfma_instructions": statistics.mean(inst[k::ns]),
                     "counted_over_algorithmic": round(counted / alg, 4) if alg else None})
    out = {"workload": f"{args.config}_bs{args.batch}", "kernel_sha": kernel_sha(), "per_stage": rows,
           "counted_over_algorithmic": round(sum(r["counted_flop"] for r in rows) /
                                             sum(r["algorithmic_flop"] for r in rows), 4)}
    path = os.path.join(out_dir or os.path.join(ROOT, "profiles"), f"mfma_{args.config}_bs{args.batch}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out, indent=1))


def write_occupancy(args, ios_dir, seq_dir, out_dir=None):
    """Mean resident waves per CU while the stage kernels run, for the IOS
    schedule and for the sequential one-unit-per-launch schedule of the same
    kernels (Sec. 6.3 compares active warps the same way).  From two
    rocprofv3 --pmc MeanOccupancyPerCU GRBM_GUI_ACTIVE runs: the derived
    counter is SQ_LEVEL_WAVES accumulated over the dispatch / the GPU-active
    cycles of the dispatch / CUs, so launch and drain count as empty time.
    The timed loop is the last steps x stages stage-kernel dispatches; each
    is weighted by its GPU-active cycles."""
    out = {"workload": f"{args.config}_bs{args.batch}", "kernel_sha": kernel_sha(),
           "counter": "MeanOccupancyPerCU (waves per CU over the dispatch's GPU-active cycles; "
                      "a CU holds at most 32 wave64, this kernel at most 16)"}
    for name, d in (("ios", ios_dir), ("sequential", seq_dir)):
        occ = _pmc_rows(d, "MeanOccupancyPerCU")
        act = {i: v for i, _, v in _pmc_rows(d, "GRBM_GUI_ACTIVE")}
        info = _pmc_info(d)
        meta = json.load(open(os.path.join(d, "bench.json")))
        ns = meta["stages"]
        timed = [(i, v) for i, k, v in occ if "ios_stage_kernel" in k][-meta["steps"] * ns:]
        w = sum(act[i] for i, _ in timed)
        stages = []
        for k in range(ns):
            rows = timed[k::ns]
            wk = sum(act[i] for i, _ in rows)
            stages.append({"units": meta["schedule"][k]["units"], "strategy": meta["schedule"][k]["strategy"],
                           "workgroups": info[rows[0][0]][0],
                           "mean_waves_per_cu": round(sum(v * act[i] for i, v in rows) / wk, 3),
                           "dispatch_us": round(statistics.median(info[i][1] for i, _ in rows) / 1e3, 2)})
        out[name] = {"stages": ns, "mean_waves_per_cu": round(sum(v * act[i] for i, v in timed) / w, 3),
                     "per_stage": stages}
    out["ios_over_sequential"] = round(out["ios"]["mean_waves_per_cu"] / out["sequential"]["mean_waves_per_cu"], 3)
    path = os.path.join(out_dir or os.path.join(ROOT, "profiles"), f"occupancy_{args.config}_bs{args.batch}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out, indent=1))


def _pmc_info(d):
    """Dispatch id -> (workgroups, dispatch ns under counter collection)."""
    import csv
    import glob
    info = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            wg = int(r["Grid_Size"]) // max(1, int(r["Workgroup_Size"]))
            info[int(r["Dispatch_Id"])] = (wg, int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    return info


def trace_summary(args, trace_dir, out_dir=None):
    """Stage-kernel launch durations of the timed loop from a rocprofv3
    --kernel-trace run of this benchmark (run with --no-stage-times, so the
    timed loop is the last steps x stages stage-kernel dispatches; bench.json
    in the directory holds that run's JSON line).  Also the mean launch
    period (first start to last end / launches, which includes the gaps the
    event-based figure of the benchmark line includes) and the fraction of
    the fp32 MFMA peak the kernel durations give.  Written to
    profiles/trace_<workload>.json (or out_dir)."""
    import csv
    import glob
    import workloads as W
    rows = []
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if "ios_stage_kernel" in r["Kernel_Name"]:
                rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), int(r.get("Grid_Size_X") or r.get("Grid_Size")) // 512))
    rows.sort()
    meta = json.load(open(os.path.join(trace_dir, "bench.json")))
    n = meta["steps"] * meta["stages"]
    timed = rows[-n:]
    dur = [e - b for b, e, _ in timed]
    by_grid = {}
    for (b, e, wg) in timed:
        by_grid.setdefault(wg, []).append(e - b)
    gaps = [timed[i + 1][0] - timed[i][1] for i in range(len(timed) - 1)]
    ns = meta["stages"]
    sched = meta.get("schedule") or [{}] * ns
    spec, _ = W.make(args.config, args.batch, args.seed)
    work = unit_work(spec, args.batch)
    per_stage = []
    for k in range(ns):
        units = sched[k].get("units")
        f_m = sum(work[u][0] for u in units) if units else None
        med = statistics.median(dur[k::ns])
        per_stage.append({"units": units, "workgroups": timed[k][2], "median_ns": med,
                          "tflops": round(f_m / med / 1e3, 3) if f_m is not None else None})
    mean = statistics.mean(dur)
    period = (timed[-1][1] - timed[0][0]) / len(timed)
    mfma_step = sum(w[0] for w in work.values())
    out = {"workload": f"{args.config}_bs{args.batch}", "kernel_sha": meta.get("kernel_sha"),
           "launches": len(timed), "mean_ns": mean, "median_ns": statistics.median(dur),
           "mean_period_ns": round(period, 1),
           "median_gap_ns": statistics.median(gaps) if gaps else None,
           "frac_from_trace": round(mfma_step / ns / mean / 1e3 / PEAK_FP32_TFLOPS, 5),
           "frac_from_period": round(mfma_step / ns / period / 1e3 / PEAK_FP32_TFLOPS, 5),
           "per_stage": per_stage,
           "by_workgroups": {str(k): {"launches": len(v), "median_ns": statistics.median(v)}
                             for k, v in sorted(by_grid.items())},
           "step_us_of_that_run": meta["value"]}
    path = os.path.join(out_dir or os.path.join(ROOT, "profiles"), f"trace_{args.config}_bs{args.batch}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out, indent=1))


# NASNet at batch 32 is left out: its ~56k candidate stages at that batch take
# longer to profile than a benchmark run should.
SUITE = [("tiny", 1), ("inception", 1), ("inception", 16), ("randwire", 1), ("nasnet", 1),
         ("squeeze", 1), ("squeeze", 32), ("squeeze", 128)]


def run_suite(args):
    """Every configuration and batch size of the benchmark list: the DP
    schedule (on-device profiling), the sequential and greedy schedules, all
    on the same kernels and timed the same way."""
    import numpy as np
    import torch

    import paper_2011_01302_amd as I
    import workloads as W
    report = []
    for config, batch in SUITE:
        spec, ten = W.make(config, batch, args.seed)
        g = I.Graph(spec, ten)
        dev = "cuda:0"
        ins = [torch.from_numpy(np.ascontiguousarray(ten[t["name"]])).to(dev) for t in spec["inputs"]]
        shp = W.infer_shapes(spec)
        outs = [torch.empty((batch,) + shp[o], device=dev) for o in spec["outputs"]]
        stream = torch.cuda.current_stream().cuda_stream
        row = {"config": config, "batch": batch}
        iso = conv_tiles(I, g)
        work = unit_work(spec, batch)
        row["gflop"] = round(sum(w[0] + w[1] for w in work.values()) / 1e9, 4)
        for name, mode in (("ios", I.IOS_SCHED_DP), ("sequential", I.IOS_SCHED_SEQUENTIAL),
                           ("greedy", I.IOS_SCHED_GREEDY)):
            o = I.ios_sched_opts_default()
            o.mode = mode
            if config in ("randwire", "nasnet"):      # tens of thousands of candidate stages
                o.warmup, o.reps, o.repeats = 1, 3, 1
                o.verify_reps = 20                     # the picked stages measured in full
            print(f"[suite] {config} bs{batch} {name}: scheduling", file=sys.stderr, flush=True)
            t0 = time.perf_counter()
            for u, t in iso.items():
                I.ios_set_conv_tile(g.handle, u, t)
            q, pred = I.ios_schedule(g.handle, o)
            search = time.perf_counter() - t0
            tune_for(I, g, q, iso)
            steps = max(20, min(args.steps, int(2e5 / max(1.0, row["gflop"] * 1e3))))
            us = time_steps(I, g, q, ins, outs, stream, 10, steps, torch)
            assert I.ios_device_status(g.handle, stream) == 0
            sched = I.ios_schedule_get(q)
            entry = {"us": round(us, 2), "stages": len(sched), "predicted_us": round(pred / 1e3, 2),
                     "search_s": round(search, 2)}
            if mode == I.IOS_SCHED_DP:
                st, tr, ms = I.ios_schedule_stats(q)
                entry.update({"states": st, "transitions": tr, "stages_measured": ms,
                              "schedule": [(g.names(ids), "merge" if t else "concurrent") for ids, t in sched]})
            row[name] = entry
            I.ios_schedule_destroy(q)
        row["speedup_vs_sequential"] = round(row["sequential"]["us"] / row["ios"]["us"], 3)
        row["speedup_vs_greedy"] = round(row["greedy"]["us"] / row["ios"]["us"], 3)
        row["tflops"] = round(row["gflop"] / row["ios"]["us"] * 1e3, 2)
        print(f"[suite] {config:9s} bs{batch:<4d} IOS {row['ios']['us']:9.2f} us ({row['ios']['stages']} stages)"
              f"  seq {row['sequential']['us']:9.2f}  greedy {row['greedy']['us']:9.2f}"
              f"  x{row['speedup_vs_sequential']:.2f} vs seq  {row['tflops']} TFLOP/s", file=sys.stderr, flush=True)
        report.append(row)
        g.close()
        del ins, outs
        torch.cuda.empty_cache()
    with open(args.suite, "w") as f:
        json.dump(report, f, indent=1)


def _setup(I, W, torch, config, batch, seed):
    import numpy as np
    spec, ten = W.make(config, batch, seed)
    g = I.Graph(spec, ten)
    dev = "cuda:0"
    ins = [torch.from_numpy(np.ascontiguousarray(ten[t["name"]])).to(dev) for t in spec["inputs"]]
    shp = W.infer_shapes(spec)
    outs = [torch.empty((batch,) + shp[o], device=dev) for o in spec["outputs"]]
    return spec, g, ins, outs


def _cost_table(I, g):
    """The graph's last search's stage latencies: {(block, mask): {strategy: ns}}."""
    import tempfile
    with tempfile.NamedTemporaryFile("r", suffix=".jsonl") as f:
        I.ios_schedule_dump_costs(g.handle, f.name)
        rows = [json.loads(x) for x in open(f.name)]
    tab = {}
    for r in rows:
        tab[(r["block"], r["mask"])] = {I.IOS_CONCURRENT: r["concurrent_ns"], I.IOS_MERGE: r["merge_ns"]}
    return tab


def run_next(args):
    """Follow-up experiments on the same calls (written to args.next as JSON):
    (1) strategy ablation -- IOS-Both, IOS-Parallel (no merge), IOS-Merge (no
        concurrency), sequential and greedy, on every configuration at batch
        1; the variants replay IOS-Both's measured stage latencies so that all
        DP runs see the same costs (Sec. 6.1);
    (2) batch specialisation -- schedules optimised at one batch size run at
        the others (Inception block at 1 / 16, SqueezeNet stack at 1 / 32 /
        128; Sec. 7.2);
    (3) pruning -- r in {1, 2, 3}, s in {3, 8}: search time, stages measured,
        latency of the schedule found (Sec. 4.3, Sec. 7.1)."""
    import torch

    import paper_2011_01302_amd as I
    import workloads as W
    stream = torch.cuda.current_stream().cuda_stream
    out = {"ablation": [], "batch": [], "pruning": [], "fig10": []}
    parts = set(args.next_parts.split(",")) if args.next_parts else {"ablation", "batch", "pruning", "fig10"}

    def fast(o, config):
        if config in ("randwire", "nasnet"):       # tens of thousands of candidate stages
            o.warmup, o.reps, o.repeats = 1, 3, 1
            o.verify_reps = 20                      # the picked stages measured in full
        return o

    def timed(g, q, ins, outs, gflop):
        if not hasattr(g, "iso_tiles"):             # the isolated choice of this graph
            g.iso_tiles = conv_tiles(I, g)
        iso = g.iso_tiles
        tune_for(I, g, q, iso)
        steps = max(20, min(args.steps, int(2e5 / max(1.0, gflop * 1e3))))
        us = time_steps(I, g, q, ins, outs, stream, 10, steps, torch)
        assert I.ios_device_status(g.handle, stream) == 0
        for u, t in iso.items():                    # searches start from the isolated choice
            I.ios_set_conv_tile(g.handle, u, t)
        return round(us, 2)

    # (1) strategy ablation
    for config in (W.CONFIG_NAMES if "ablation" in parts else []):
        spec, g, ins, outs = _setup(I, W, torch, config, 1, args.seed)
        gflop = sum(w[0] + w[1] for w in unit_work(spec, 1).values()) / 1e9
        row = {"config": config}
        o = fast(I.ios_sched_opts_default(), config)
        t0 = time.perf_counter()
        q, pred = I.ios_schedule(g.handle, o)
        row["search_s"] = round(time.perf_counter() - t0, 2)
        tab = _cost_table(I, g)
        row["ios_both"] = {"us": timed(g, q, ins, outs, gflop), "stages": len(I.ios_schedule_get(q)),
                           "predicted_us": pred / 1e3}
        I.ios_schedule_destroy(q)
        for name, strat in (("ios_parallel", 1), ("ios_merge", 2)):
            o = I.ios_sched_opts_default()
            o.strategies = strat
            q, pred = I.ios_schedule(g.handle, o, cost=lambda b, m, ids, t: tab[(b, m)][t])
            row[name] = {"us": timed(g, q, ins, outs, gflop), "stages": len(I.ios_schedule_get(q)),
                         "predicted_us": pred / 1e3}
            I.ios_schedule_destroy(q)
        for name, mode in (("sequential", I.IOS_SCHED_SEQUENTIAL), ("greedy", I.IOS_SCHED_GREEDY)):
            o = I.ios_sched_opts_default()
            o.mode = mode
            q, pred = I.ios_schedule(g.handle, o)
            row[name] = {"us": timed(g, q, ins, outs, gflop), "stages": len(I.ios_schedule_get(q))}
            I.ios_schedule_destroy(q)
        print(f"[next] ablation {config}: " + json.dumps({k: v["us"] for k, v in row.items() if isinstance(v, dict)}),
              file=sys.stderr, flush=True)
        out["ablation"].append(row)
        g.close()

    # (2) batch specialisation
    for config, batches in ((("inception", (1, 16)), ("squeeze", (1, 32, 128))) if "batch" in parts else ()):
        scheds = {}
        for b in batches:
            spec, g, ins, outs = _setup(I, W, torch, config, b, args.seed)
            q, _ = I.ios_schedule(g.handle, I.ios_sched_opts_default())
            scheds[b] = [(ids, t) for ids, t in I.ios_schedule_get(q)]
            I.ios_schedule_destroy(q)
            g.close()
            del ins, outs
        for run_b in batches:
            spec, g, ins, outs = _setup(I, W, torch, config, run_b, args.seed)
            gflop = sum(w[0] + w[1] for w in unit_work(spec, run_b).values()) / 1e9
            row = {"config": config, "run_batch": run_b}
            for opt_b in batches:
                q = I.ios_schedule_from_stages(g.handle, [ids for ids, _ in scheds[opt_b]],
                                               [t for _, t in scheds[opt_b]])
                row[f"optimised_for_bs{opt_b}"] = timed(g, q, ins, outs, gflop)
                I.ios_schedule_destroy(q)
            print(f"[next] batch {config} run at bs{run_b}: " + json.dumps(row), file=sys.stderr, flush=True)
            out["batch"].append(row)
            g.close()
            del ins, outs
            torch.cuda.empty_cache()

    # (4) the last Inception-V3 module at batch 1 and 32 (Sec. 7.2, Fig. 10):
    # schedules searched at each batch size, which pairs they merge, and each
    # schedule run at both batch sizes
    if "fig10" in parts:
        scheds = {}
        for b in (1, 32):
            spec, g, ins, outs = _setup(I, W, torch, "inception_7c", b, args.seed)
            q, pred = I.ios_schedule(g.handle, I.ios_sched_opts_default())
            st = I.ios_schedule_get(q)
            scheds[b] = [(ids, t) for ids, t in st]
            gflop = sum(w[0] + w[1] for w in unit_work(spec, b).values()) / 1e9
            row = {"optimised_for": b, "stages": [(g.names(ids), "merge" if t else "concurrent") for ids, t in st],
                   "merged_pairs": [g.names(ids) for ids, t in st if t == I.IOS_MERGE],
                   "predicted_us": pred / 1e3, "gflop": round(gflop, 3)}
            I.ios_schedule_destroy(q)
            out["fig10"].append(row)
            print(f"[next] fig10 optimised for bs{b}: " + json.dumps(row), file=sys.stderr, flush=True)
            g.close()
            del ins, outs
        for run_b in (1, 32):
            spec, g, ins, outs = _setup(I, W, torch, "inception_7c", run_b, args.seed)
            gflop = sum(w[0] + w[1] for w in unit_work(spec, run_b).values()) / 1e9
            row = {"run_batch": run_b}
            for opt_b in (1, 32):
                q = I.ios_schedule_from_stages(g.handle, [ids for ids, _ in scheds[opt_b]], [t for _, t in scheds[opt_b]])
                row[f"optimised_for_bs{opt_b}"] = timed(g, q, ins, outs, gflop)
                I.ios_schedule_destroy(q)
            out["fig10"].append(row)
            print(f"[next] fig10 run at bs{run_b}: " + json.dumps(row), file=sys.stderr, flush=True)
            g.close()
            del ins, outs
            torch.cuda.empty_cache()

    # (3) pruning
    for config in (("inception", "randwire", "nasnet") if "pruning" in parts else ()):
        spec, g, ins, outs = _setup(I, W, torch, config, 1, args.seed)
        gflop = sum(w[0] + w[1] for w in unit_work(spec, 1).values()) / 1e9
        for r in (1, 2, 3):
            for s_ in (3, 8):
                o = fast(I.ios_sched_opts_default(), config)
                o.r, o.s = r, s_
                t0 = time.perf_counter()
                q, pred = I.ios_schedule(g.handle, o)
                search = time.perf_counter() - t0
                st, tr, ms = I.ios_schedule_stats(q)
                row = {"config": config, "r": r, "s": s_, "search_s": round(search, 2), "states": st,
                       "transitions": tr, "stages_measured": ms, "predicted_us": pred / 1e3,
                       "us": timed(g, q, ins, outs, gflop), "stages": len(I.ios_schedule_get(q))}
                I.ios_schedule_destroy(q)
                print(f"[next] pruning " + json.dumps(row), file=sys.stderr, flush=True)
                out["pruning"].append(row)
        g.close()
    with open(args.next, "w") as f:
        json.dump(out, f, indent=1)


def run_network(args):
    """Whole networks scheduled block by block (the block-wise speed-up
    appendix): for every network, the DP runs on each block with on-device
    profiling; the whole network is then timed end to end under the IOS,
    sequential and greedy schedules, and per block from HIP events around each
    stage launch (sum of the block's stage medians).  Written to args.network
    as JSON."""
    import torch

    import paper_2011_01302_amd as I
    import workloads as W
    stream = torch.cuda.current_stream().cuda_stream
    report = []
    nets = args.networks.split(",") if args.networks else W.NETWORK_NAMES
    for net in nets:
        print(f"[network] {net} bs{args.batch}: graph", file=sys.stderr, flush=True)
        spec, g, ins, outs = _setup(I, W, torch, net, args.batch, args.seed)
        work = unit_work(spec, args.batch)
        gflop = sum(w[0] + w[1] for w in work.values()) / 1e9
        block_of = {}
        for b in range(I.ios_graph_blocks(g.handle)):
            for u in I.ios_block_units(g.handle, b):
                block_of[u] = b
        names = spec.get("block_names") or [str(b) for b in range(len(set(block_of.values())))]
        row = {"network": net, "batch": args.batch, "units": len(block_of), "blocks": len(names),
               "gflop": round(gflop, 3)}
        per_block = {n: {} for n in names}
        iso = conv_tiles(I, g)
        for name, mode in (("ios", I.IOS_SCHED_DP), ("sequential", I.IOS_SCHED_SEQUENTIAL),
                           ("greedy", I.IOS_SCHED_GREEDY)):
            o = I.ios_sched_opts_default()
            o.mode = mode
            o.r, o.s = args.r, args.s
            if net in ("randwire_net", "nasnet_net"):
                # tens of thousands of candidate stages per block at r = 3:
                # r = 1 (the paper's Sec. 7.1 finds it close to the full
                # search; so do the single-block sweeps here) and light
                # profiling, the picked stages then measured in full
                o.r = 1
                o.warmup, o.reps, o.repeats = 1, 3, 1
                o.verify_reps = 20
            print(f"[network] {net}: {name} schedule", file=sys.stderr, flush=True)
            for u, t in iso.items():
                I.ios_set_conv_tile(g.handle, u, t)
            t0 = time.perf_counter()
            q, pred = I.ios_schedule(g.handle, o)
            search = time.perf_counter() - t0
            tuned = tune_for(I, g, q, iso)
            sched = I.ios_schedule_get(q)
            us = time_steps(I, g, q, ins, outs, stream, 10, max(20, min(args.steps, 100)), torch)
            assert I.ios_device_status(g.handle, stream) == 0
            entry = {"us": round(us, 2), "stages": len(sched), "predicted_us": round(pred / 1e3, 2),
                     "tuned_us": round(tuned / 1e3, 2), "search_s": round(search, 2)}
            if mode == I.IOS_SCHED_DP:
                st, tr, ms = I.ios_schedule_stats(q)
                entry.update({"states": st, "transitions": tr, "stages_measured": ms,
                              "schedule": [(g.names(ids), "merge" if t else "concurrent") for ids, t in sched]})
            if mode != I.IOS_SCHED_GREEDY:
                st_ns, _ = stage_times(I, g, q, ins, outs, stream, 20)
                for (ids, _t), ns in zip(sched, st_ns):
                    pb = per_block[names[block_of[ids[0]]]]
                    pb[name + "_us"] = round(pb.get(name + "_us", 0.0) + ns / 1e3, 2)
                    pb[name + "_stages"] = pb.get(name + "_stages", 0) + 1
            row[name] = entry
            I.ios_schedule_destroy(q)
            print(f"[network] {net} {name}: {us:.2f} us, {len(sched)} stages, search {search:.1f} s",
                  file=sys.stderr, flush=True)
        for n, pb in per_block.items():
            pb["speedup"] = round(pb["sequential_us"] / pb["ios_us"], 3)
        row["per_block"] = per_block
        row["speedup_vs_sequential"] = round(row["sequential"]["us"] / row["ios"]["us"], 3)
        row["speedup_vs_greedy"] = round(row["greedy"]["us"] / row["ios"]["us"], 3)
        row["tflops"] = round(gflop / row["ios"]["us"] * 1e3, 2)
        report.append(row)
        g.close()
        del ins, outs
        torch.cuda.empty_cache()
    with open(args.network, "w") as f:
        json.dump(report, f, indent=1)


# ------------------------------------------------------------------ main

BATCH1 = ["tiny", "inception", "randwire", "nasnet", "squeeze"]
LARGE_SEARCH = ("randwire", "nasnet")      # tens of thousands of candidate stages


def search_opts(I, config, r=3, s=8):
    o = I.ios_sched_opts_default()
    o.r, o.s = r, s
    if config in LARGE_SEARCH:
        o.warmup, o.reps, o.repeats = 1, 3, 1
        o.verify_reps = 20                      # the picked stages measured in full
    return o


def stage_rows(I, g, spec, batch, stages):
    """Per stage: its launch period when launched back to back alone (the
    stage profiler's own measurement, with the schedule's tile choices),
    algorithmic MFMA / VALU flops, compulsory bytes and their roofline."""
    work = unit_work(spec, batch)
    rows = []
    for ids, strat in stages:
        names = g.names(ids)
        ns = I.ios_profile_stage(g.handle, ids, strat, 3, 20, 3)
        f_m = sum(work[n][0] for n in names)
        f_v = sum(work[n][1] for n in names)
        by = stage_bytes(spec, batch, set(names)) + sum(work[n][2] for n in names)
        t_roof = max(f_m / (PEAK_FP32_TFLOPS * 1e12), f_v / (PEAK_FP32_TFLOPS * 1e12),
                     by / (PEAK_HBM_GBS * 1e9)) * 1e9
        rows.append({"units": names, "strategy": "merge" if strat else "concurrent", "ns": ns,
                     "mfma_flop": f_m, "valu_flop": f_v, "bytes": by,
                     "tflops": round(f_m / ns / 1e3, 3) if ns else None,
                     "frac_of_roofline": round(t_roof / ns, 5) if ns else None})
    return rows


def measure_config(I, W, torch, config, batch, seed, steps, warmup, args, plan=None, baselines=True):
    """Search (or replay `plan`), tune, time; the same for the baselines."""
    spec, g, ins, outs = _setup(I, W, torch, config, batch, seed)
    stream = torch.cuda.current_stream().cuda_stream
    work = unit_work(spec, batch)
    mfma = sum(w[0] for w in work.values())
    iso = conv_tiles(I, g)
    res = {"config": config, "batch": batch, "gflop": round(sum(w[0] + w[1] for w in work.values()) / 1e9, 4)}
    tuned_ns = None
    if plan:
        set_unit_tiling(I, g, plan["tiling"])
        q = I.ios_schedule_from_stages(g.handle, [[g.tid[n] for n in st["units"]] for st in plan["schedule"]],
                                       [I.IOS_MERGE if st["strategy"] == "merge" else I.IOS_CONCURRENT
                                        for st in plan["schedule"]])
        search_s, pred_ns, stats = 0.0, plan["search"]["predicted_ns"], (0, 0, 0)
    else:
        o = search_opts(I, config, args.r, args.s)
        t0 = time.perf_counter()
        q, pred_ns = I.ios_schedule(g.handle, o)
        search_s = time.perf_counter() - t0
        stats = I.ios_schedule_stats(q)
        tuned_ns = I.ios_schedule_tune_tiles(g.handle, q)
    stages = I.ios_schedule_get(q)
    res["schedule"] = [{"units": g.names(ids), "strategy": "merge" if t else "concurrent"} for ids, t in stages]
    res["tiling"] = unit_tiling(I, g)
    res["search"] = {"seconds": round(search_s, 3), "states": stats[0], "transitions": stats[1],
                     "stages_measured": stats[2], "predicted_ns": pred_ns, "tuned_ns": tuned_ns}
    rep = timed_repeats(I, g, q, ins, outs, stream, warmup, steps, torch)
    assert I.ios_device_status(g.handle, stream) == 0
    us = statistics.median(rep)
    res["us"] = round(us, 3)
    res["launches"] = len(stages)
    res["repeats"] = {"n": len(rep), "steps_each": steps // len(rep), "median_us": round(us, 3),
                      "min_us": round(min(rep), 3), "max_us": round(max(rep), 3)}
    res["mfma_flop_per_step"] = mfma
    res["tflops"] = round(mfma / us / 1e6, 3)
    res["frac_of_fp32_mfma_peak"] = round(mfma / us / 1e6 / PEAK_FP32_TFLOPS, 5)
    print(f"[bench] {config} bs{batch}: IOS {us:.2f} us/step, {len(stages)} stages, search {search_s:.1f} s",
          file=sys.stderr, flush=True)
    if not args.no_stage_times:
        res["stages"] = stage_rows(I, g, spec, batch, stages)
    if baselines:
        base = {}
        for name, mode in (("sequential", I.IOS_SCHED_SEQUENTIAL), ("greedy", I.IOS_SCHED_GREEDY)):
            o = I.ios_sched_opts_default()
            o.mode = mode
            for u, t in iso.items():
                I.ios_set_conv_tile(g.handle, u, t)
            qb, _ = I.ios_schedule(g.handle, o)
            tune_for(I, g, qb, iso)
            ub = statistics.median(timed_repeats(I, g, qb, ins, outs, stream, warmup, steps, torch))
            base[name] = {"us": round(ub, 3), "launches": len(I.ios_schedule_get(qb)),
                          "speedup_of_ios": round(ub / us, 3)}
            I.ios_schedule_destroy(qb)
            print(f"[bench] {config} bs{batch}: {name} {ub:.2f} us/step", file=sys.stderr, flush=True)
        res["gpu_baselines"] = base
    return spec, g, q, ins, outs, res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500,
                    help="timed steps of the headline, split into 5 equal windows (median reported)")
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="squeeze")
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--r", type=int, default=3)
    ap.add_argument("--s", type=int, default=8)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-baselines", action="store_true")
    ap.add_argument("--headline-only", action="store_true",
                    help="skip the other batch-1 configurations")
    ap.add_argument("--report", default="", help="also write the full report (JSON) here")
    ap.add_argument("--dump-costs", default="", help="write the search's stage-latency table here")
    ap.add_argument("--no-stage-times", action="store_true",
                    help="profiler runs: time the headline only and print a short line (the timed "
                         "loop is then the last launches of the run)")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="finish with one plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--suite", default="",
                    help="instead of the headline line, measure every configuration and batch "
                         "(IOS vs sequential vs greedy) and write a JSON report to this path")
    ap.add_argument("--next", default="",
                    help="run the follow-up experiments (strategy ablation, batch specialisation, "
                         "pruning sweep) and write a JSON report to this path")
    ap.add_argument("--network", default="",
                    help="schedule whole networks block by block (IOS vs sequential vs greedy, "
                         "end to end and per block) and write a JSON report to this path")
    ap.add_argument("--networks", default="", help="with --network: comma-separated subset of the networks")
    ap.add_argument("--next-parts", default="", help="with --next: comma-separated subset of "
                                                      "ablation,batch,pruning,fig10")
    ap.add_argument("--trace-summary", default="", metavar="TRACE_DIR",
                    help="summarise the timed loop of a rocprofv3 --kernel-trace run of this "
                         "benchmark and exit")
    ap.add_argument("--plan-from", default="", metavar="PLAN_JSON",
                    help="replay the schedule and tuning choices recorded in this file (the last "
                         "JSON line holding a plan) instead of searching: for profiler runs, whose "
                         "added per-launch cost would change the search's choices")
    ap.add_argument("--save-plan", default="", metavar="PLAN_JSON",
                    help="write the headline's schedule and tuning choices here (for --plan-from)")
    ap.add_argument("--search", action="store_true",
                    help="always search: by default a configuration whose plan was recorded under "
                         "profiles/ (plan_<config>_bs<batch>.json, from a search on an MI355X with "
                         "the current kernel sources) replays that plan, so that the number and the "
                         "committed profiles describe the same schedule")
    ap.add_argument("--mode", choices=("dp", "sequential", "greedy"), default="dp",
                    help="schedule of the timed step: the DP search (default) or a baseline "
                         "(with --plan-from: that run's tile shapes, this mode's schedule)")
    ap.add_argument("--occupancy-from", nargs=2, metavar=("IOS_DIR", "SEQ_DIR"),
                    help="turn two rocprofv3 --pmc MeanOccupancyPerCU GRBM_GUI_ACTIVE runs (IOS "
                         "schedule, --mode sequential) into profiles/occupancy_<workload>.json and exit")
    ap.add_argument("--mfma-from", default="", metavar="PMC_DIR",
                    help="turn a rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_INSTS_VALU_MFMA_F32 run "
                         "into profiles/mfma_<workload>.json and exit")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this benchmark "
                         "into profiles/traffic_<workload>.json and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the stage executor runs on a single MI355X and this "
              "build has no multi-GPU path (batch sharding is a design note only).", file=sys.stderr)
        sys.exit(2)

    if args.trace_summary:
        trace_summary(args, args.trace_summary)
        return
    if args.traffic_from:
        write_traffic(args, *args.traffic_from)
        return
    if args.occupancy_from:
        write_occupancy(args, *args.occupancy_from)
        return
    if args.mfma_from:
        write_mfma(args, args.mfma_from)
        return

    lib = os.path.join(ROOT, "paper_2011_01302_amd", "libios.so")
    if not os.path.exists(lib):
        import __graft_entry__
        __graft_entry__._load_build_module().build()
    if args.suite:
        run_suite(args)
        return
    if args.next:
        run_next(args)
        return
    if args.network:
        run_network(args)
        return
    import torch

    import paper_2011_01302_amd as I
    import workloads as W

    print(f"[bench] config={args.config} batch={args.batch} seed={args.seed}", file=sys.stderr, flush=True)
    plan, plan_src = None, None
    if not args.plan_from and not args.search:
        plan, plan_src = recorded_plan(args.config, args.batch)
    if args.plan_from:
        plan = [json.loads(l) for l in open(args.plan_from) if l.startswith("{") and '"tiling"' in l][-1]
        plan_src = args.plan_from
    if plan is not None:
        if args.mode != "dp":
            # a baseline schedule of the same kernels, with the plan's tile choices
            spec, g, ins, outs = _setup(I, W, torch, args.config, args.batch, args.seed)
            set_unit_tiling(I, g, plan["tiling"])
            o = I.ios_sched_opts_default()
            o.mode = I.IOS_SCHED_SEQUENTIAL if args.mode == "sequential" else I.IOS_SCHED_GREEDY
            q, _ = I.ios_schedule(g.handle, o, cost=lambda b, m, ids, t: 1000)
            stream = torch.cuda.current_stream().cuda_stream
            us = statistics.median(timed_repeats(I, g, q, ins, outs, stream, args.warmup, args.steps, torch))
            stages = I.ios_schedule_get(q)
            print(json.dumps({"value": round(us, 3), "unit": "us", "stages": len(stages), "steps": args.steps,
                              "mode": args.mode,
                              "schedule": [{"units": g.names(ids), "strategy": "merge" if t else "concurrent"}
                                           for ids, t in stages]}), flush=True)
            return
    spec, g, q, ins, outs, head = measure_config(
        I, W, torch, args.config, args.batch, args.seed, args.steps, args.warmup, args, plan=plan,
        baselines=not (args.no_baselines or args.no_stage_times))
    if args.dump_costs and not plan:
        I.ios_schedule_dump_costs(g.handle, args.dump_costs)
    if args.save_plan:
        with open(args.save_plan, "w") as f:
            rec = {k: head[k] for k in ("config", "batch", "schedule", "tiling", "search")}
            rec["kernel_sha"] = kernel_sha()
            rec["us_when_searched"] = head["us"]
            f.write(json.dumps(rec) + "\n")
    us = head["us"]
    n_launch = head["launches"]

    if args.no_stage_times:
        if args.copy_mb:
            src = torch.ones(args.copy_mb << 18, device="cuda:0")
            dst = torch.empty_like(src)
            dst.copy_(src)
            torch.cuda.synchronize()
        print(json.dumps({"value": us, "unit": "us", "stages": n_launch, "steps": args.steps,
                          "copy_mb": args.copy_mb, "mode": args.mode, "schedule": head["schedule"],
                          "kernel_sha": kernel_sha()}), flush=True)
        return

    workload = f"{args.config}_bs{args.batch}"
    sha = kernel_sha()
    mfma = head["mfma_flop_per_step"]
    roof = {"bound": "mfma", "achieved": head["tflops"], "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
            "frac": head["frac_of_fp32_mfma_peak"], "traffic": load_traffic(workload, sha),
            "kernel": "ios_stage_kernel", "launches_per_step": n_launch,
            "mean_launch_ns": round(us * 1e3 / n_launch, 1),
            "mfma_flop_per_launch": mfma / n_launch, "kernel_sha": sha,
            "duration_basis": "HIP events over the timed region on the launch stream: step time / launches "
                              "per step (inter-kernel dispatch gaps included)"}
    tr = load_trace(workload, sha)
    if tr:
        roof["trace"] = tr
    result = {
        "metric": "batch-1 network latency (us) + achieved fp32 TFLOP/s per stage vs MFMA peak",
        "value": us, "unit": "us", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(us / 1e3, 6), "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{args.config} (seeded synthetic inputs, random-init weights; "
                               f"{head['gflop']} GFLOP per image)",
                   "batch": args.batch, "seed": args.seed, "pruning": {"r": args.r, "s": args.s},
                   "parallelism": "single GPU, inter-operator (IOS stages)"},
        "roofline": roof,
        "schedule": head.get("stages", head["schedule"]),
        "tiling": head["tiling"],
        "search": head["search"],
        "plan": ("replayed from " + os.path.relpath(plan_src, ROOT)) if plan else
                "searched in this run (DP with on-device stage profiling, then per-stage tile tuning)",
        "repeats": head["repeats"],
        "throughput_img_per_s": round(args.batch / us * 1e6, 1),
    }
    if "gpu_baselines" in head:
        result["gpu_baselines"] = head["gpu_baselines"]
    I.ios_schedule_destroy(q)
    g.close()
    del ins, outs
    torch.cuda.empty_cache()
    if not args.headline_only and args.batch == 1:
        others = {}
        for config in BATCH1:
            if config == args.config:
                continue
            steps = 100 if config in LARGE_SEARCH else 500
            p2, src2 = (None, None) if args.search else recorded_plan(config, 1)
            _, g2, q2, i2, o2, r2 = measure_config(I, W, torch, config, 1, args.seed, steps, args.warmup, args,
                                                   plan=p2, baselines=not args.no_baselines)
            r2["plan"] = ("replayed from " + os.path.relpath(src2, ROOT)) if p2 else "searched in this run"
            keep = ("us", "launches", "gflop", "tflops", "frac_of_fp32_mfma_peak", "repeats", "gpu_baselines",
                    "schedule", "search", "plan")
            others[config] = {k: r2[k] for k in keep if k in r2}
            I.ios_schedule_destroy(q2)
            g2.close()
            del i2, o2
            torch.cuda.empty_cache()
        result["other_batch1_configs"] = others
    if not args.no_cpu:
        cpu_us, n = cpu_oracle(spec, W.make(args.config, args.batch, args.seed)[1], args.cpu_seconds)
        result["cpu_baseline"] = {"value": round(cpu_us, 1), "unit": "us", "cores": 1, "kind": "oracle",
                                  "sample": f"{n} full evaluations of the {args.config} workload at batch "
                                            f"{args.batch} (fp64 direct loops, single thread)",
                                  "host": host_cpu()}
        print(f"[bench] cpu oracle {cpu_us:.0f} us/eval", file=sys.stderr, flush=True)
    line = json.dumps(result)
    if args.report:
        with open(args.report, "w") as f:
            f.write(line + "\n")
    print(line, flush=True)


if __name__ == "__main__":
    main()
