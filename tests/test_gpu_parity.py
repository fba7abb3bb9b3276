"""GPU parity: the library's stage kernels against the fp64 oracle, through
the C ABI, on the seeded workloads.  Activations must satisfy
max|gpu - oracle| / max|oracle| <= 1e-4 per output tensor (fp32 path vs fp64
reference); schedules found on the device must equal the oracle DP replayed
on the dumped cost table, bit for bit."""
import functools
import json
import os

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu
TOL = 1e-4

torch = pytest.importorskip("torch")
I = pytest.importorskip("paper_2011_01302_amd")
from oracle import evaluator as E          # noqa: E402
from oracle import schedule as O           # noqa: E402

DEV = "cuda:0"


@functools.lru_cache(maxsize=None)
def case(config, batch=1, seed=0):
    spec, ten = W.make(config, batch, seed)
    return spec, ten


@functools.lru_cache(maxsize=None)
def reference(config, batch=1, seed=0):
    spec, ten = case(config, batch, seed)
    return E.outputs(spec, ten)


def device_input(a, offset=0):
    """`a` on the device, starting `offset` floats into its allocation (so
    that offset 1..3 gives a base address off a 16-byte boundary)."""
    flat = torch.from_numpy(np.ascontiguousarray(a)).reshape(-1)
    buf = torch.empty(flat.numel() + offset, dtype=torch.float32, device=DEV)
    buf[offset:].copy_(flat.to(DEV))
    return buf[offset:].view(a.shape)


def run(g, q, spec, ten, stream=0, offset=0):
    ins = [device_input(ten[t["name"]], offset) for t in spec["inputs"]]
    shp = W.infer_shapes(spec)
    outs = [torch.full((g.batch,) + shp[o], float("nan"), device=DEV) for o in spec["outputs"]]
    I.ios_run(g.handle, q, [t.data_ptr() for t in ins], [o.data_ptr() for o in outs], stream)
    torch.cuda.synchronize()
    assert I.ios_device_status(g.handle, stream) == 0
    return [o.cpu().numpy() for o in outs]


def rel_err(got, ref):
    return float(np.abs(got.astype(np.float64) - ref).max() / np.abs(ref).max())


# Element-wise diagnostic: the largest |gpu - oracle| / |oracle| over the
# elements with |oracle| > 1e-3 max|oracle|.  The tensor bound (TOL) alone
# would allow up to TOL / 1e-3 = 0.1 there; fp32 accumulation over K <= 1200
# terms typically errs by ~sqrt(K) * 2^-24 ~ 2e-6 of the terms' magnitude,
# i.e. ~1e-3 relative at 1e-3 of the maximum, so 1e-2 is a tight-enough
# bound that still leaves room for the order in which a tile sums.
ELT_FLOOR, ELT_TOL = 1e-3, 1e-2


def elt_err(got, ref):
    a = np.abs(ref)
    sel = a > ELT_FLOOR * a.max()
    return float((np.abs(got.astype(np.float64) - ref)[sel] / a[sel]).max())


def check(outs, refs, what=""):
    worst = 0.0
    for got, ref in zip(outs, refs):
        assert got.shape == ref.shape
        assert np.isfinite(got).all(), what
        e = rel_err(got, ref)
        assert e <= TOL, f"{what}: relative error {e:.3e}"
        el = elt_err(got, ref)
        worst = max(worst, el)
        assert el <= ELT_TOL, f"{what}: element-wise relative error {el:.3e}"
    print(f"[parity] {what}: element-wise max {worst:.2e}", flush=True)


def sched(g, mode, cost=lambda b, m, ids, t: 1000):
    o = I.ios_sched_opts_default()
    o.mode = mode
    q, _ = I.ios_schedule(g.handle, o, cost)
    return q


def block_stages(g):
    """One concurrent stage holding a whole block (chains run inside it)."""
    blocks = g.blocks()
    return I.ios_schedule_from_stages(g.handle, blocks, [I.IOS_CONCURRENT] * len(blocks))


@pytest.fixture(autouse=True)
def _print_case(request):
    print(f"\n[gpu-case] {request.node.name}", flush=True)
    yield


# ------------------------------------------------------------------ schedules x configs

@pytest.mark.parametrize("config", W.CONFIG_NAMES)
@pytest.mark.parametrize("kind", ["sequential", "greedy", "block_stage"])
def test_parity_schedules(config, kind):
    spec, ten = case(config)
    g = I.Graph(spec, ten)
    if kind == "sequential":
        q = sched(g, I.IOS_SCHED_SEQUENTIAL)
    elif kind == "greedy":
        q = sched(g, I.IOS_SCHED_GREEDY)
    else:
        q = block_stages(g)
    check(run(g, q, spec, ten), reference(config), f"{config}/{kind}")
    I.ios_schedule_destroy(q)
    g.close()


def merge_schedule(g, spec, groups):
    """Stages: each listed group (names) as a merge stage, every other unit
    alone, in a valid order."""
    names = [u["name"] for u in W.unit_ops(spec)]
    grouped = {n for grp in groups for n in grp}
    stages, strat, done = [], [], set()
    for n in names:
        if n in done:
            continue
        grp = next((gr for gr in groups if n in gr), None)
        if grp:
            stages.append([g.tid[x] for x in grp])
            strat.append(I.IOS_MERGE)
            done |= set(grp)
        elif n not in grouped:
            stages.append([g.tid[n]])
            strat.append(I.IOS_CONCURRENT)
            done.add(n)
    return I.ios_schedule_from_stages(g.handle, stages, strat)


@pytest.mark.parametrize("config,groups", [
    ("tiny", [["A", "B1"]]),
    ("inception", [["b1", "b2a", "b3a"]]),
    ("inception", [["b1", "b3a"]]),
    ("squeeze", [[f"m{m}e1", f"m{m}e3"] for m in range(1, 9)]),
])
def test_parity_operator_merge(config, groups):
    spec, ten = case(config)
    g = I.Graph(spec, ten)
    q = merge_schedule(g, spec, groups)
    check(run(g, q, spec, ten), reference(config), f"{config}/merge")
    I.ios_schedule_destroy(q)
    g.close()


@pytest.mark.parametrize("tile", [str(t) for t in range(12)])
def test_parity_every_conv_tile_shape(tile, monkeypatch):
    monkeypatch.setenv("IOS_CONV_TILE", tile)
    for config in ["tiny", "inception", "squeeze"]:
        spec, ten = case(config)
        g = I.Graph(spec, ten)
        q = sched(g, I.IOS_SCHED_GREEDY)
        check(run(g, q, spec, ten), reference(config), f"{config}/tile{tile}")
        I.ios_schedule_destroy(q)
        q = merge_schedule(g, spec, [["A", "B1"]] if config == "tiny" else
                           [["b1", "b2a", "b3a"]] if config == "inception" else
                           [[f"m{m}e1", f"m{m}e3"] for m in range(1, 9)])
        check(run(g, q, spec, ten), reference(config), f"{config}/merge/tile{tile}")
        I.ios_schedule_destroy(q)
        g.close()


@pytest.mark.parametrize("config,seed", [("randwire", 1), ("nasnet", 1), ("nasnet", 2)])
def test_parity_other_seeds(config, seed):
    spec, ten = case(config, 1, seed)
    g = I.Graph(spec, ten)
    for q in (sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
        check(run(g, q, spec, ten), reference(config, 1, seed), f"{config}/seed{seed}")
        I.ios_schedule_destroy(q)
    g.close()


# ------------------------------------------------------------------ DP on the device

@pytest.mark.parametrize("config", ["tiny", "inception", "squeeze"])
def test_device_dp_schedule_replays_in_oracle(config, tmp_path):
    spec, ten = case(config)
    g = I.Graph(spec, ten)
    o = I.ios_sched_opts_default()
    o.warmup, o.reps, o.repeats = 2, 5, 3
    q, cost = I.ios_schedule(g.handle, o)
    assert cost > 0
    check(run(g, q, spec, ten), reference(config), f"{config}/dp")
    path = tmp_path / "costs.jsonl"
    I.ios_schedule_dump_costs(g.handle, str(path))
    table = {}
    for line in open(path):
        r = json.loads(line)
        table[(r["block"], r["mask"], 0)] = r["concurrent_ns"]
        if r["merge_ns"] is not None:
            table[(r["block"], r["mask"], 1)] = r["merge_ns"]
    total, stages = 0, []
    for b, blk in enumerate(O.blocks_of(spec)):
        res = O.ios_dp(blk, lambda m, t: table[(b, m, t)], 3, 8)
        total += res.cost
        stages += [(sorted(blk.units[i]["name"] for i in O.bits(m)), t) for m, t in res.schedule]
    lib = [(sorted(g.names(ids)), t) for ids, t in I.ios_schedule_get(q)]
    assert lib == stages
    assert total == cost
    I.ios_schedule_destroy(q)
    g.close()


@pytest.mark.parametrize("config,verify", [("randwire", 0), ("nasnet", 0), ("randwire", 10), ("nasnet", 10)])
def test_device_dp_large_blocks_replay_in_oracle(config, verify, tmp_path):
    """RandWire (33 units, ~31k candidate stages) and NASNet (17 units, ~56k):
    the search runs on the device with light profiling (and, with verify, the
    picked stages measured again until the search keeps its choice); the
    schedule must be the oracle's on the final dumped table and the outputs
    must match."""
    spec, ten = case(config)
    g = I.Graph(spec, ten)
    o = I.ios_sched_opts_default()
    o.warmup, o.reps, o.repeats = 1, 2, 1
    o.verify_reps = verify
    q, cost = I.ios_schedule(g.handle, o)
    check(run(g, q, spec, ten), reference(config), f"{config}/dp")
    path = tmp_path / "costs.jsonl"
    I.ios_schedule_dump_costs(g.handle, str(path))
    table = {}
    for line in open(path):
        r = json.loads(line)
        table[(r["mask"], 0)] = r["concurrent_ns"]
        if r["merge_ns"] is not None:
            table[(r["mask"], 1)] = r["merge_ns"]
    blk = O.blocks_of(spec)[0]
    res = O.ios_dp(blk, lambda m, t: table[(m, t)], 3, 8)
    lib = [(sorted(g.names(ids)), t) for ids, t in I.ios_schedule_get(q)]
    assert lib == [(sorted(blk.units[i]["name"] for i in O.bits(m)), t) for m, t in res.schedule]
    assert res.cost == cost
    states, transitions, _ = I.ios_schedule_stats(q)
    assert (states, transitions) == (res.states, res.transitions)
    I.ios_schedule_destroy(q)
    g.close()


def test_profile_stage_and_errors():
    spec, ten = case("inception")
    g = I.Graph(spec, ten)
    for u in W.unit_ops(spec):
        assert I.ios_profile_stage(g.handle, [g.tid[u["name"]]], 0, 1, 3, 1) > 0
    ids = [g.tid[n] for n in ("b1", "b2a", "b3a")]
    assert I.ios_profile_stage(g.handle, ids, I.IOS_MERGE, 1, 3, 1) > 0
    with pytest.raises(I.IosError) as e:
        I.ios_profile_stage(g.handle, [g.tid["b1"], g.tid["b4"]], I.IOS_MERGE)
    assert e.value.name == "IOS_E_NOT_MERGEABLE"
    g.close()


def test_conv_tile_shapes_read_and_replayed():
    """The tuned shape of every conv can be read back and replaced; stages
    compiled afterwards use the new shapes (results still match the oracle)."""
    spec, ten = case("inception")
    g = I.Graph(spec, ten)
    convs = [u["name"] for u in W.unit_ops(spec) if u["kind"] == "conv"]
    tuned = {n: I.ios_get_conv_tile(g.handle, g.tid[n]) for n in convs}
    assert all(0 <= v < I.IOS_CONV_TILE_SHAPES for v in tuned.values())
    with pytest.raises(I.IosError) as e:
        I.ios_get_conv_tile(g.handle, g.tid["pool"])
    assert e.value.name == "IOS_E_ARG"
    for k, n in enumerate(convs):
        I.ios_set_conv_tile(g.handle, g.tid[n], k % I.IOS_CONV_TILE_SHAPES)
    assert [I.ios_get_conv_tile(g.handle, g.tid[n]) for n in convs] == \
        [k % I.IOS_CONV_TILE_SHAPES for k in range(len(convs))]
    for mode in (I.IOS_SCHED_SEQUENTIAL, I.IOS_SCHED_GREEDY):
        q = sched(g, mode)
        check(run(g, q, spec, ten), reference("inception"), f"inception/replayed tiles/mode{mode}")
        I.ios_schedule_destroy(q)
    g.close()


@pytest.mark.parametrize("lg", ["0", "2", "4"])
def test_parity_every_xcd_tile_order(lg, monkeypatch):
    """Each run length of the XCD tile order (forced for every stage; the
    per-stage choice picks among these): ragged shapes with chained stages
    (persistent launches) and the Inception block in one and several
    stages."""
    monkeypatch.setenv("IOS_XCD_RUNS", lg)
    spec = ragged_spec(2)
    ten = W.make_tensors(spec, 3)
    ref = E.outputs(spec, ten)
    g = I.Graph(spec, ten)
    for q in (sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
        check(run(g, q, spec, ten), ref, f"ragged/xcd {lg}")
        I.ios_schedule_destroy(q)
    g.close()
    spec, ten = case("inception")
    g = I.Graph(spec, ten)
    for q in (sched(g, I.IOS_SCHED_SEQUENTIAL), sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
        check(run(g, q, spec, ten), reference("inception"), f"inception/xcd {lg}")
        I.ios_schedule_destroy(q)
    g.close()


def test_schedule_tune_tiles_per_stage(monkeypatch):
    """Per-stage conv tile shapes: the call measures every stage, leaves the
    chosen shapes on the graph and the schedule runs with them (results still
    match); with IOS_CONV_TILE set the shapes stay as they are."""
    spec, ten = case("inception")
    g = I.Graph(spec, ten)
    convs = [u["name"] for u in W.unit_ops(spec) if u["kind"] == "conv"]
    o = I.ios_sched_opts_default()
    o.warmup, o.reps, o.repeats = 2, 5, 3
    q, _ = I.ios_schedule(g.handle, o)
    check(run(g, q, spec, ten), reference("inception"), "inception/dp")
    total = I.ios_schedule_tune_tiles(g.handle, q, o)
    assert total > 0
    tiles = {n: I.ios_get_conv_tile(g.handle, g.tid[n]) for n in convs}
    assert all(0 <= v < I.IOS_CONV_TILE_SHAPES for v in tiles.values())
    for st_ids, strat in I.ios_schedule_get(q):
        if strat == I.IOS_MERGE:                       # a merged conv takes one shape
            assert len({tiles[n] for n in g.names(st_ids)}) == 1
    check(run(g, q, spec, ten), reference("inception"), "inception/dp/tuned tiles")
    monkeypatch.setenv("IOS_CONV_TILE", "2")
    assert I.ios_schedule_tune_tiles(g.handle, q, o) > 0
    assert {n: I.ios_get_conv_tile(g.handle, g.tid[n]) for n in convs} == tiles
    I.ios_schedule_destroy(q)
    g.close()


def test_schedule_tune_sepconv_blocks():
    """Per-stage choice on stages with SEPCONVs (blocks per tile), convs and
    pools, including a stage whose groups are chains: results still match."""
    spec = ragged_spec(2)
    ten = W.make_tensors(spec, 3)
    ref = E.outputs(spec, ten)
    g = I.Graph(spec, ten)
    o = I.ios_sched_opts_default()
    o.warmup, o.reps, o.repeats = 1, 3, 1
    for q in (sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
        assert I.ios_schedule_tune_tiles(g.handle, q, o) > 0
        check(run(g, q, spec, ten), ref, "ragged/tuned")
        I.ios_schedule_destroy(q)
    g.close()


def test_run_timed_and_determinism():
    spec, ten = case("inception")
    g = I.Graph(spec, ten)
    q = block_stages(g)
    a = run(g, q, spec, ten)
    b = run(g, q, spec, ten)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    ins = [torch.from_numpy(ten["x"]).to(DEV)]
    out = torch.empty((1, 256, 35, 35), device=DEV)
    ns = I.ios_run_timed(g.handle, q, [ins[0].data_ptr()], [out.data_ptr()])
    assert len(ns) == 1 and ns[0] > 0
    I.ios_schedule_destroy(q)
    g.close()


# ------------------------------------------------------------------ batches

def batched_reference(config, batch, seed=0):
    """The oracle on every image of a batch: images are independent, so each
    is evaluated as a batch-1 graph, several at a time (the oracle's C loops
    run without the interpreter lock)."""
    from concurrent.futures import ThreadPoolExecutor
    spec, ten = case(config, batch, seed)
    s1 = W.with_batch(spec, 1)

    def one(i):
        t1 = dict(ten)
        for t in spec["inputs"]:
            t1[t["name"]] = ten[t["name"]][i:i + 1]
        return E.outputs(s1, t1)
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        per = list(ex.map(one, range(batch)))
    return spec, ten, [np.concatenate([p[k] for p in per], axis=0) for k in range(len(spec["outputs"]))]


@pytest.mark.parametrize("config,batch,kinds", [
    ("inception", 16, ("dp", "sequential", "dp_tuned")),
    ("squeeze", 32, ("dp", "greedy")),
    ("squeeze", 128, ("dp", "greedy")),
    ("nasnet", 32, ("block_stage", "greedy", "greedy_tuned")),
])
def test_parity_batched_every_image(config, batch, kinds):
    """Every image of the batched configurations against the oracle, under
    the DP's schedule (on-device profiling, light) where the search is
    affordable, a one-stage chained schedule for NASNet and a baseline; the
    "_tuned" kinds then choose every stage's tiles in its company
    (ios_schedule_tune_tiles: pipelined conv shapes, the GEMM SEPCONV tile)."""
    spec, ten, refs = batched_reference(config, batch)
    g = I.Graph(spec, ten)
    for kind in kinds:
        if kind.startswith("dp"):
            o = I.ios_sched_opts_default()
            o.warmup, o.reps, o.repeats = 1, 3, 1
            q, _ = I.ios_schedule(g.handle, o)
        elif kind == "block_stage":
            q = block_stages(g)
        else:
            q = sched(g, I.IOS_SCHED_SEQUENTIAL if kind == "sequential" else I.IOS_SCHED_GREEDY)
        if kind.endswith("_tuned"):
            o = I.ios_sched_opts_default()
            o.warmup, o.reps, o.repeats = 1, 3, 1
            assert I.ios_schedule_tune_tiles(g.handle, q, o) > 0
        check(run(g, q, spec, ten), refs, f"{config}/bs{batch}/{kind}")
        I.ios_schedule_destroy(q)
    g.close()


def sepg_spec(batch):
    """SEPCONVs the 64-column GEMM tile applies to (planes up to 32 wide):
    21x21 planes (3 output rows per tile, the last tile of an image short),
    40 input channels (a short last chunk), 100 output channels (a short
    channel tile), 3x3 and 5x5 windows, chained."""
    sep = lambda n, i, co, k: {"name": n, "kind": "sepconv", "in": [i], "cout": co, "kh": k, "kw": k, "sh": 1,
                               "sw": 1, "ph": k // 2, "pw": k // 2, "pre_relu": 1, "post_relu": 0}
    ops = [sep("g1", "x", 100, 3), sep("g2", "x", 36, 5), sep("g3", "g1", 40, 5)]
    return {"name": "sepg", "batch": batch, "inputs": [{"name": "x", "c": 40, "h": 20, "w": 21}],
            "ops": ops, "outputs": ["g2", "g3"]}


@pytest.mark.parametrize("tile", ["7", "8"])
def test_parity_sepconv_gemm_batched(tile, monkeypatch):
    """The GEMM SEPCONV tile forced on every unit of a NASNet cell (128
    columns: 42-wide planes) or of sepg_spec (64 columns), over three images
    (row blocks of every image, halo rows at image borders), under greedy
    stages and one chained stage."""
    monkeypatch.setenv("IOS_SEP_TILE", tile)
    if tile == "7":
        spec, ten, refs = batched_reference("nasnet", 3)
    else:
        spec = sepg_spec(3)
        ten = W.make_tensors(spec, 5)
        refs = E.outputs(spec, ten)
    g = I.Graph(spec, ten)
    seps = [u["name"] for u in W.unit_ops(spec) if u["kind"] == "sepconv"]
    assert all(I.ios_get_unit_tiling(g.handle, g.tid[n])[0] == int(tile) for n in seps)
    for q in (sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
        check(run(g, q, spec, ten), refs, f"{spec['name']}/bs3/sep tile {tile}")
        I.ios_schedule_destroy(q)
    g.close()


def test_parity_inception_7c_merged_pairs_bs32():
    """The last Inception-V3 module at batch 32 with its two parallel
    1x3 / 3x1 pairs each run as one merged 3x3 conv (Sec. 7.2: the schedule
    the paper finds best at large batch), and with the three 1x1 convs on the
    input merged: every image against the oracle."""
    spec, ten, refs = batched_reference("inception_7c", 32)
    g = I.Graph(spec, ten)
    q = merge_schedule(g, spec, [["7c_1x1", "7c_3a", "7c_d3a"], ["7c_3b1", "7c_3b2"], ["7c_d3c1", "7c_d3c2"]])
    st = I.ios_schedule_get(q)
    assert sum(t == I.IOS_MERGE for _, t in st) == 3
    check(run(g, q, spec, ten), refs, "inception_7c/bs32/merged pairs")
    I.ios_schedule_destroy(q)
    g.close()


def test_device_dp_batched_replays_in_oracle(tmp_path):
    """A search at batch 16 (Sec. 7.2: schedules are specialised per batch
    size) replays bit for bit in the oracle DP on the dumped table."""
    spec, ten, refs = batched_reference("inception", 16)
    g = I.Graph(spec, ten)
    o = I.ios_sched_opts_default()
    o.warmup, o.reps, o.repeats = 1, 3, 3
    q, cost = I.ios_schedule(g.handle, o)
    check(run(g, q, spec, ten), refs, "inception/bs16/dp")
    path = tmp_path / "costs.jsonl"
    I.ios_schedule_dump_costs(g.handle, str(path))
    table = {}
    for line in open(path):
        r = json.loads(line)
        table[(r["mask"], 0)] = r["concurrent_ns"]
        if r["merge_ns"] is not None:
            table[(r["mask"], 1)] = r["merge_ns"]
    blk = O.blocks_of(spec)[0]
    res = O.ios_dp(blk, lambda m, t: table[(m, t)], 3, 8)
    lib = [(sorted(g.names(ids)), t) for ids, t in I.ios_schedule_get(q)]
    assert lib == [(sorted(blk.units[i]["name"] for i in O.bits(m)), t) for m, t in res.schedule]
    assert res.cost == cost
    I.ios_schedule_destroy(q)
    g.close()


def test_parity_batched_full_small():
    spec, ten = case("inception", 3)
    ref = E.outputs(spec, ten)
    g = I.Graph(spec, ten)
    q = block_stages(g)
    check(run(g, q, spec, ten), ref, "inception/bs3")
    I.ios_schedule_destroy(q)
    g.close()


def test_chained_stage_back_to_back_on_different_inputs():
    """A stage with in-stage dependencies (persistent launch, per-op
    counters reset by its last workgroup) run twice back to back, without a
    host wait between, on two different seeded inputs: each output must be
    its own input's oracle result (a counter left non-zero by the first run
    would let a consumer tile of the second read the first run's
    intermediates)."""
    spec = ragged_spec(2)
    ten_a = W.make_tensors(spec, 3)
    ten_b = dict(ten_a)
    other = W.make_tensors(spec, 4)
    for t in spec["inputs"]:
        ten_b[t["name"]] = other[t["name"]]
    refs = [E.outputs(spec, ten_a), E.outputs(spec, ten_b)]
    g = I.Graph(spec, ten_a)
    q = block_stages(g)
    shp = W.infer_shapes(spec)
    outs = []
    keep = []
    for ten in (ten_a, ten_b, ten_a, ten_b):
        ins = [device_input(ten[t["name"]]) for t in spec["inputs"]]
        o = [torch.full((g.batch,) + shp[n], float("nan"), device=DEV) for n in spec["outputs"]]
        I.ios_run(g.handle, q, [t.data_ptr() for t in ins], [x.data_ptr() for x in o], 0)
        keep.append(ins)
        outs.append(o)
    torch.cuda.synchronize()
    assert I.ios_device_status(g.handle, 0) == 0
    for k, o in enumerate(outs):
        check([x.cpu().numpy() for x in o], refs[k % 2], f"ragged/back-to-back run {k}")
    I.ios_schedule_destroy(q)
    g.close()


# ------------------------------------------------------------------ ragged shapes

def ragged_spec(batch, cin=13):
    conv = lambda n, i, co, k, s, p, post=1: {"name": n, "kind": "conv", "in": [i], "cout": co,
                                             "kh": k[0], "kw": k[1], "sh": s, "sw": s, "ph": p[0],
                                             "pw": p[1], "pre_relu": 0, "post_relu": post}
    ops = [conv("c1", "x", 20, (3, 3), 1, (1, 1)),
           conv("c2", "x", 7, (5, 5), 1, (2, 2)),
           conv("c3", "x", 9, (3, 1), 1, (1, 0)),
           conv("c4", "x", 5, (1, 3), 1, (0, 1)),
           conv("c5", "x", 11, (3, 3), 2, (1, 1), post=0),
           {"name": "s1", "kind": "sepconv", "in": ["c1", "c1"], "cout": 21, "kh": 3, "kw": 3,
            "sh": 1, "sw": 1, "ph": 1, "pw": 1, "pre_relu": 1, "post_relu": 0},
           {"name": "s2", "kind": "sepconv", "in": ["s1"], "cout": 13, "kh": 5, "kw": 5,
            "sh": 1, "sw": 1, "ph": 2, "pw": 2, "pre_relu": 1, "post_relu": 0},
           {"name": "s3", "kind": "sepconv", "in": ["x"], "cout": 6, "kh": 1, "kw": 3,
            "sh": 1, "sw": 1, "ph": 0, "pw": 1, "pre_relu": 1, "post_relu": 0},
           {"name": "s4", "kind": "sepconv", "in": ["x", "x", "x"], "cout": 17, "kh": 5, "kw": 5,
            "sh": 1, "sw": 1, "ph": 1, "pw": 1, "pre_relu": 1, "post_relu": 0},
           {"name": "mp", "kind": "maxpool", "in": ["x"], "kh": 3, "kw": 3, "sh": 2, "sw": 2,
            "ph": 1, "pw": 1},
           {"name": "ap", "kind": "avgpool", "in": ["s2"], "kh": 3, "kw": 3, "sh": 1, "sw": 1,
            "ph": 1, "pw": 1},
           {"name": "ad", "kind": "add", "in": ["ap", "s2", "s2"]},
           {"name": "mn", "kind": "mean", "in": ["c2", "c2", "c2"]},
           {"name": "cat", "kind": "concat", "in": ["c3", "c4"]},
           {"name": "cat2", "kind": "concat", "in": ["c5", "mp"]}]
    return {"name": "ragged", "batch": batch, "inputs": [{"name": "x", "c": cin, "h": 9, "w": 11}],
            "ops": ops, "outputs": ["ad", "mn", "cat", "cat2", "s3", "s4"]}


# tile None: shapes chosen by measurement, else forced; offset: inputs start
# 1 or 3 floats past a 16-byte boundary; the pipelined shapes (6 .. 11) need
# input channels in multiples of 16, so their cases take 32
@pytest.mark.parametrize("batch,tile,offset", [(1, None, 0), (2, None, 0), (1, "1", 1), (1, "0", 3),
                                               (2, "4", 1), (2, "6", 1), (3, "7", 0), (1, "8", 3),
                                               (2, "9", 3), (3, "10", 1), (1, "11", 0)])
def test_parity_ragged_shapes(batch, tile, offset, monkeypatch):
    if tile is not None:
        monkeypatch.setenv("IOS_CONV_TILE", tile)
    spec = ragged_spec(batch, 32 if tile is not None and int(tile) >= 6 else 13)
    ten = W.make_tensors(spec, 3)
    ref = E.outputs(spec, ten)
    g = I.Graph(spec, ten)
    for q in (sched(g, I.IOS_SCHED_SEQUENTIAL), sched(g, I.IOS_SCHED_GREEDY), block_stages(g),
              I.ios_schedule_from_stages(g.handle, [[g.tid[n] for n in ("c1", "c2", "c3", "c4")],
                                                    [g.tid[n] for n in ("c5", "s1", "s2", "s3", "s4", "mp",
                                                                        "ap", "ad", "mn")]],
                                         [I.IOS_MERGE, I.IOS_CONCURRENT])):
        check(run(g, q, spec, ten, offset=offset), ref, "ragged")
        I.ios_schedule_destroy(q)
    g.close()


def pool_planes_spec(batch):
    """Pools over many small planes (several whole planes per tile from 512
    planes up): inputs read from concat slices, outputs written into one,
    a global average pool, planes of a tile crossing an image boundary and
    a last tile with fewer planes."""
    conv = lambda n, co: {"name": n, "kind": "conv", "in": ["x"], "cout": co, "kh": 1, "kw": 1, "sh": 1,
                          "sw": 1, "ph": 0, "pw": 0, "pre_relu": 0, "post_relu": 0}
    pool = lambda n, kind, i, kh, kw, s, p: {"name": n, "kind": kind, "in": [i], "kh": kh, "kw": kw,
                                            "sh": s, "sw": s, "ph": p, "pw": p}
    ops = [conv("c1", 400), conv("c2", 400),
           {"name": "cat", "kind": "concat", "in": ["c1", "c2"]},
           pool("mp", "maxpool", "c2", 3, 3, 2, 1),
           pool("ap", "avgpool", "c1", 3, 3, 1, 1),
           pool("gp", "avgpool", "c2", 7, 7, 1, 0),
           pool("m2", "maxpool", "c1", 3, 3, 2, 1),
           {"name": "outc", "kind": "concat", "in": ["mp", "m2"]}]
    return {"name": "pool_planes", "batch": batch, "inputs": [{"name": "x", "c": 5, "h": 7, "w": 7}],
            "ops": ops, "outputs": ["cat", "ap", "gp", "outc"]}


@pytest.mark.parametrize("batch", [1, 2, 3])
def test_parity_pool_planes(batch):
    spec = pool_planes_spec(batch)
    ten = W.make_tensors(spec, 5)
    ref = E.outputs(spec, ten)
    g = I.Graph(spec, ten)
    for q in (sched(g, I.IOS_SCHED_SEQUENTIAL), sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
        check(run(g, q, spec, ten), ref, f"pool planes bs{batch}")
        I.ios_schedule_destroy(q)
    g.close()


@pytest.mark.parametrize("tile", ["0", "1", "4", "6", "7", "8", "9", "10", "11"])
def test_parity_conv_tiles_batched_small(tile, monkeypatch):
    """Forced conv tile shapes over several small images (the 16-pixel
    blocks of an 8x8 plane never span two images)."""
    monkeypatch.setenv("IOS_CONV_TILE", tile)
    spec, ten = case("tiny", 3)
    ref = E.outputs(spec, ten)
    g = I.Graph(spec, ten)
    for q in (sched(g, I.IOS_SCHED_SEQUENTIAL), block_stages(g)):
        check(run(g, q, spec, ten), ref, f"tiny/bs3/tile{tile}")
        I.ios_schedule_destroy(q)
    g.close()


@pytest.mark.parametrize("tile", [str(t) for t in range(11)])
def test_parity_every_sepconv_tile(tile, monkeypatch):
    # SEPCONV tile choice (staged: 16, 32 or 64 output pixels per tile; row:
    # 1 to 4 channel blocks; GEMM: whole rows in 128 or 64 columns; line:
    # 32 / W whole rows x 32 or 64 channels, RandWire's 28-wide nodes), forced
    # instead of measured (a unit a choice does not apply to falls back to
    # the staged tile: the wide 7x7 unit and multi-input sums for the row and
    # GEMM tiles; the 3x3 unit over 280 channels, ragged's 5x5 unit over 21
    # channels on a 9x11 plane and the NASNet / RandWire single-input units
    # run on the GEMM tile)
    monkeypatch.setenv("IOS_SEP_TILE", tile)
    for config in ["randwire", "nasnet"]:
        spec, ten = case(config)
        g = I.Graph(spec, ten)
        for q in (sched(g, I.IOS_SCHED_SEQUENTIAL), sched(g, I.IOS_SCHED_GREEDY)):
            check(run(g, q, spec, ten), reference(config), f"{config}/sep tile {tile}")
            I.ios_schedule_destroy(q)
        g.close()
    for spec in (ragged_spec(2), wide_sep_spec(2)):
        ten = W.make_tensors(spec, 4)
        g = I.Graph(spec, ten)
        for q in (sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
            check(run(g, q, spec, ten), E.outputs(spec, ten), f"{spec['name']}/sep tile {tile}")
            I.ios_schedule_destroy(q)
        g.close()


def line_spec(batch):
    """SEPCONVs the line tile applies to: 28-wide planes (one output row per
    tile) of 77 channels (an odd channel padded to a k-step), a six-input sum
    (two rounds of loads), chained; 16-wide planes of 15 rows (two output rows
    per tile, the last tile half past the image) and 33 channels; 8-wide
    planes of 96 channels (four rows per tile, the most channels); 32-wide
    planes (four loads per thread); l1 and l6 written into one concat (the
    graph output), read back as slices by l2 (channel offset 0 of 117) and l7
    (offset 77).  Output channels 77, 50, 40, 20, 64, 40 and 24: short and
    whole last blocks of 32 and 64 channels."""
    sep = lambda n, ins, co: {"name": n, "kind": "sepconv", "in": ins, "cout": co, "kh": 3, "kw": 3, "sh": 1,
                              "sw": 1, "ph": 1, "pw": 1, "pre_relu": 1, "post_relu": 0}
    ops = [sep("l1", ["x"], 77),
           sep("l2", ["x", "y", "l1", "x", "y", "l1"], 50),
           sep("l3", ["z"], 40),
           sep("l4", ["u", "u"], 20),
           sep("l5", ["v"], 64),
           sep("l6", ["y"], 40),
           {"name": "cat", "kind": "concat", "in": ["l1", "l6"]},
           sep("l7", ["l6"], 24)]
    return {"name": "line", "batch": batch,
            "inputs": [{"name": "x", "c": 77, "h": 28, "w": 28}, {"name": "y", "c": 77, "h": 28, "w": 28},
                       {"name": "z", "c": 33, "h": 15, "w": 16}, {"name": "u", "c": 96, "h": 10, "w": 8},
                       {"name": "v", "c": 70, "h": 6, "w": 32}],
            "ops": ops, "outputs": ["l2", "l3", "l4", "l5", "cat", "l7"]}


@pytest.mark.parametrize("tile", ["9", "10"])
def test_parity_sepconv_line_tile(tile, monkeypatch):
    """The line SEPCONV tile forced on every unit of line_spec over two
    images (sequential, greedy and chained stages) and of the RandWire block
    at batch 1 and 2, every image against the oracle."""
    monkeypatch.setenv("IOS_SEP_TILE", tile)
    spec = line_spec(2)
    ten = W.make_tensors(spec, 6)
    refs = E.outputs(spec, ten)
    g = I.Graph(spec, ten)
    # the two-block choice needs more than 32 output channels: not l4's 20 or l7's 24
    units = ("l1", "l2", "l3", "l4", "l5", "l6", "l7") if tile == "9" else ("l1", "l2", "l3", "l5", "l6")
    assert all(I.ios_get_unit_tiling(g.handle, g.tid[n])[0] == int(tile) for n in units)
    for q in (sched(g, I.IOS_SCHED_SEQUENTIAL), sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
        check(run(g, q, spec, ten), refs, f"line/bs2/sep tile {tile}")
        I.ios_schedule_destroy(q)
    g.close()
    for batch in (1, 2):
        spec, ten, refs = batched_reference("randwire", batch)
        g = I.Graph(spec, ten)
        seps = [u["name"] for u in W.unit_ops(spec) if u["kind"] == "sepconv"]
        assert all(I.ios_get_unit_tiling(g.handle, g.tid[n])[0] == int(tile) for n in seps)
        for q in (sched(g, I.IOS_SCHED_GREEDY), block_stages(g)):
            check(run(g, q, spec, ten), refs, f"randwire/bs{batch}/sep tile {tile}")
            I.ios_schedule_destroy(q)
        g.close()


def wide_sep_spec(batch):
    """SEPCONVs past the old limits: 280 input channels (18 chunks of 16 or 9
    of 32, a short last group), 7x7 and 1x5 windows, 180 output channels
    (12 channel blocks, several channel groups per pixel run), an odd 19x23
    plane, a chain of two and a three-input sum."""
    sep = lambda n, ins, co, kh, kw: {"name": n, "kind": "sepconv", "in": ins, "cout": co, "kh": kh, "kw": kw,
                                      "sh": 1, "sw": 1, "ph": kh // 2, "pw": kw // 2, "pre_relu": 1,
                                      "post_relu": 0}
    ops = [sep("w1", ["x"], 180, 7, 7),
           sep("w2", ["w1", "x2", "w1"], 36, 1, 5),
           sep("w3", ["x"], 20, 3, 3)]
    return {"name": "wide_sep", "batch": batch,
            "inputs": [{"name": "x", "c": 280, "h": 19, "w": 23}, {"name": "x2", "c": 180, "h": 19, "w": 23}],
            "ops": ops, "outputs": ["w2", "w3"]}
