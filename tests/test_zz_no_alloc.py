"""ios_run_noalloc (no allocation of any kind; intermediates and in-stage
counters in the library's fixed device array) against ios_run through the C
ABI: the same outputs on two calls in a row, the second on a smaller graph,
each also within the oracle tolerance; its error paths."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
I = pytest.importorskip("paper_2011_01302_amd")
from oracle import evaluator as E          # noqa: E402

DEV = "cuda:0"
TOL = 1e-4


def chained_spec(batch):
    """Two branches, one a chain of convs and a SEPCONV (so that a one-stage
    schedule has in-stage dependencies and uses the counters), a pool and an
    add; ragged sizes."""
    conv = lambda n, i, co, k, p: {"name": n, "kind": "conv", "in": [i], "cout": co, "kh": k, "kw": k,
                                   "sh": 1, "sw": 1, "ph": p, "pw": p, "pre_relu": 0, "post_relu": 1}
    ops = [conv("c1", "x", 24, 3, 1), conv("c2", "c1", 20, 1, 0),
           {"name": "s1", "kind": "sepconv", "in": ["c2", "c2"], "cout": 12, "kh": 3, "kw": 3, "sh": 1, "sw": 1,
            "ph": 1, "pw": 1, "pre_relu": 1, "post_relu": 0},
           conv("c3", "x", 12, 5, 2),
           {"name": "mp", "kind": "maxpool", "in": ["c3"], "kh": 3, "kw": 3, "sh": 1, "sw": 1, "ph": 1, "pw": 1},
           {"name": "ad", "kind": "add", "in": ["s1", "mp"]},
           {"name": "cat", "kind": "concat", "in": ["c2", "c3"]}]
    return {"name": "chained", "batch": batch, "inputs": [{"name": "x", "c": 10, "h": 13, "w": 11}],
            "ops": ops, "outputs": ["ad", "cat"]}


def rel_err(got, ref):
    return float(np.abs(got.astype(np.float64) - ref).max() / np.abs(ref).max())


def run_both(spec, ten, make_q):
    g = I.Graph(spec, ten)
    q = make_q(g)
    shp = W.infer_shapes(spec)
    ins = [torch.from_numpy(np.ascontiguousarray(ten[t["name"]])).to(DEV) for t in spec["inputs"]]
    ref_out = [torch.full((g.batch,) + shp[o], float("nan"), device=DEV) for o in spec["outputs"]]
    na_out = [torch.full((g.batch,) + shp[o], float("nan"), device=DEV) for o in spec["outputs"]]
    ip = [t.data_ptr() for t in ins]
    I.ios_run(g.handle, q, ip, [o.data_ptr() for o in ref_out])
    torch.cuda.synchronize()
    I.ios_run_noalloc(g.handle, q, ip, [o.data_ptr() for o in na_out])
    torch.cuda.synchronize()
    assert I.ios_device_status(g.handle) == 0
    res = ([o.cpu().numpy() for o in ref_out], [o.cpu().numpy() for o in na_out])
    I.ios_schedule_destroy(q)
    g.close()
    return res


def one_stage(g):
    blocks = g.blocks()
    return I.ios_schedule_from_stages(g.handle, blocks, [I.IOS_CONCURRENT] * len(blocks))


def greedy(g):
    o = I.ios_sched_opts_default()
    o.mode = I.IOS_SCHED_GREEDY
    return I.ios_schedule(g.handle, o, cost=lambda b, m, ids, t: 1000)[0]


@pytest.mark.parametrize("make_q", [one_stage, greedy], ids=["one_stage", "greedy"])
def test_noalloc_matches_ios_run_two_calls(make_q):
    print("\n[gpu-case] noalloc two calls", make_q.__name__, flush=True)
    cases = [("inception", W.make("inception", 2, 0)), ("chained", None)]
    spec_c = chained_spec(1)
    cases[1] = ("chained", (spec_c, W.make_tensors(spec_c, 5)))
    for name, (spec, ten) in cases:       # the second graph is the smaller one
        ref = E.outputs(spec, ten)
        lib, na = run_both(spec, ten, make_q)
        for a, b, r in zip(lib, na, ref):
            assert np.isfinite(b).all()
            assert np.array_equal(a, b), name
            assert rel_err(b, r) <= TOL, name


def test_noalloc_errors(monkeypatch):
    print("\n[gpu-case] noalloc errors", flush=True)
    monkeypatch.setenv("IOS_CONV_TILE", "1")      # no tile measurement at set-up
    monkeypatch.setenv("IOS_SEP_TILE", "1")
    spec = chained_spec(1)
    ten = W.make_tensors(spec, 5)
    g = I.Graph(spec, ten)
    q = one_stage(g)
    x = torch.zeros((1, 10, 13, 11), device=DEV)
    outs = [torch.zeros((1, 12, 13, 11), device=DEV), torch.zeros((1, 32, 13, 11), device=DEV)]
    with pytest.raises(I.IosError) as e:          # before any ios_run: not set up
        I.ios_run_noalloc(g.handle, q, [x.data_ptr()], [o.data_ptr() for o in outs])
    assert e.value.name == "IOS_E_STATE"
    I.ios_get_conv_tile(g.handle, g.tid["c1"])    # device set up, schedule not compiled yet
    with pytest.raises(I.IosError) as e:
        I.ios_run_noalloc(g.handle, q, [x.data_ptr()], [o.data_ptr() for o in outs])
    assert e.value.name == "IOS_E_STATE"
    with pytest.raises(I.IosError) as e:
        I.ios_run_noalloc(g.handle, q, [x.data_ptr()], [0, outs[1].data_ptr()])
    assert e.value.name in ("IOS_E_STATE", "IOS_E_ARG")
    I.ios_schedule_destroy(q)
    g.close()
    # intermediates larger than the array: the SqueezeNet stack at batch 32
    spec, ten = W.make("squeeze", 32, 0)
    g = I.Graph(spec, ten)
    I.ios_get_conv_tile(g.handle, g.tid["m1sq"])
    q = one_stage(g)
    with pytest.raises(I.IosError) as e:
        I.ios_run_noalloc(g.handle, q, [0], [0])
    assert e.value.name == "IOS_E_UNSUPPORTED"
    assert "64 MiB" in I.ios_last_error()
    I.ios_schedule_destroy(q)
    g.close()
