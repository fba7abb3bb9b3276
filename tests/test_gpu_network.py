"""GPU parity on whole networks: Inception-V3 (3x299x299 -> 1000 logits,
13 blocks, 109 schedule units), SqueezeNet v1.0 (3x227x227 -> 1000, 12
blocks, 28 units), the RandWire stack (3 random-graph stages and 2
transitions, 101 units) and the NASNet stack (6 cells and a strided conv,
121 units), random weights, through the C ABI against the fp64 oracle
(max|gpu - oracle| / max|oracle| <= 1e-4 on the outputs), under the baseline
schedules and under the DP run block by block on the device, whose schedule
must equal the oracle DP replayed on the dumped cost table."""
import functools
import json

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
def case(net, batch=1):
    return W.make(net, batch, 0)


@functools.lru_cache(maxsize=None)
def reference(net, batch=1):
    spec, ten = case(net, batch)
    print(f"[gpu-case] oracle evaluation of {net} at batch {batch}", flush=True)
    return E.outputs(spec, ten)


def run(g, q, spec, ten):
    ins = [torch.from_numpy(np.ascontiguousarray(ten[t["name"]])).to(DEV) for t in spec["inputs"]]
    shp = W.infer_shapes(spec)
    outs = [torch.full((g.batch,) + shp[o], float("nan"), device=DEV) for o in spec["outputs"]]
    I.ios_run(g.handle, q, [t.data_ptr() for t in ins], [o.data_ptr() for o in outs], 0)
    torch.cuda.synchronize()
    assert I.ios_device_status(g.handle, 0) == 0
    return [o.cpu().numpy() for o in outs]


def check(outs, refs, what):
    for got, ref in zip(outs, refs):
        assert got.shape == ref.shape
        assert np.isfinite(got).all(), what
        e = float(np.abs(got.astype(np.float64) - ref).max() / np.abs(ref).max())
        assert e <= TOL, f"{what}: relative error {e:.3e}"


@pytest.fixture(autouse=True)
def _print_case(request):
    print(f"\n[gpu-case] {request.node.name}", flush=True)
    yield


@pytest.mark.parametrize("net,batch", [(n, 1) for n in W.NETWORK_NAMES] + [("squeezenet", 3)])
def test_network_parity_baseline_schedules(net, batch):
    """Sequential (one unit per launch), greedy (every ready unit per launch)
    and one stage per block (branches chained inside the launch, chains of up
    to five convs)."""
    spec, ten = case(net, batch)
    ref = reference(net, batch)
    g = I.Graph(spec, ten)
    assert len(g.blocks()) == len(spec["block_names"])
    for mode in (I.IOS_SCHED_SEQUENTIAL, I.IOS_SCHED_GREEDY):
        o = I.ios_sched_opts_default()
        o.mode = mode
        q, _ = I.ios_schedule(g.handle, o, lambda b, m, ids, t: 1000)
        check(run(g, q, spec, ten), ref, f"mode {mode}")
        I.ios_schedule_destroy(q)
    blocks = g.blocks()
    q = I.ios_schedule_from_stages(g.handle, blocks, [I.IOS_CONCURRENT] * len(blocks))
    check(run(g, q, spec, ten), ref, "one stage per block")
    I.ios_schedule_destroy(q)
    g.close()


# pruning per network: the random-graph stages and the NASNet cells search
# with r = 1 (the paper's fast setting, Sec. 7.1), which keeps the test short
PRUNING = {"inception_v3": (3, 8), "squeezenet": (3, 8), "randwire_net": (1, 8), "nasnet_net": (1, 8)}


@pytest.mark.parametrize("net", W.NETWORK_NAMES)
def test_network_device_dp_replays_in_oracle(net, tmp_path):
    """Algorithm 1 on each block with on-device stage profiling
    (light protocol); the outputs must match and the schedule must be the
    oracle DP's on the dumped cost table, block by block."""
    spec, ten = case(net)
    g = I.Graph(spec, ten)
    pr, ps = PRUNING[net]
    o = I.ios_sched_opts_default()
    o.warmup, o.reps, o.repeats = 1, 3, 1
    o.r, o.s = pr, ps
    q, cost = I.ios_schedule(g.handle, o)
    check(run(g, q, spec, ten), reference(net), "dp")
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
        res = O.ios_dp(blk, lambda m, t: table[(b, m, t)], pr, ps)
        total += res.cost
        stages += [(sorted(blk.units[i]["name"] for i in O.bits(m)), t) for m, t in res.schedule]
    lib = [(sorted(g.names(ids)), t) for ids, t in I.ios_schedule_get(q)]
    assert lib == stages
    assert total == cost
    # conv tile shapes chosen per stage, then the same schedule again
    assert I.ios_schedule_tune_tiles(g.handle, q, o) > 0
    check(run(g, q, spec, ten), reference(net), "dp, per-stage tiles")
    I.ios_schedule_destroy(q)
    g.close()
