"""Pins for the oracle evaluator against facts that do not come from it:
textbook special cases, closed forms, hand-computed values and (for
cross-checks only) PyTorch CPU float64 routines."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import evaluator as E
import workloads as W


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_conv1x1_is_matmul():
    x = rnd((2, 7, 5, 6), 0)
    w = rnd((9, 7, 1, 1), 1)
    b = rnd((9,), 2)
    y = E.conv2d(x, w, b)
    ref = np.einsum("oc,nchw->nohw", w[:, :, 0, 0], x) + b[None, :, None, None]
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


def test_conv_hand_values():
    # 1 channel 3x3 input, 2x2 kernel, no pad: each output is a 4-term dot.
    x = np.arange(9, dtype=np.float64).reshape(1, 1, 3, 3)
    w = np.array([[[[1.0, 2.0], [3.0, 4.0]]]])
    y = E.conv2d(x, w)
    # y[0,0] = 0*1+1*2+3*3+4*4 = 27 ; y[0,1] = 1+4+12+20 = 37 ; y[1,0] = 3+8+18+28=57 ; y[1,1]=67
    np.testing.assert_array_equal(y[0, 0], [[27.0, 37.0], [57.0, 67.0]])
    # stride 2 pad 1: output 2x2 taking windows centred at corners
    y2 = E.conv2d(x, w, stride=(2, 2), pad=(1, 1))
    # (0,0): only tap (1,1) inside -> x[0,0]*4 = 0 ; (0,1): taps (1,0),(1,1) -> x[0,1]*3 + x[0,2]*4 = 3+8
    assert y2[0, 0, 0, 0] == 0.0 and y2[0, 0, 0, 1] == 11.0
    # (1,0): taps (0,1),(1,1) -> x[1,0]*2 + x[2,0]*4 = 6+24 ; (1,1): full window at rows1-2 cols1-2
    assert y2[0, 0, 1, 0] == 30.0 and y2[0, 0, 1, 1] == 4 * 1 + 5 * 2 + 7 * 3 + 8 * 4


def test_conv_centred_delta_is_identity_and_relu():
    x = rnd((1, 4, 6, 6), 3)
    w = np.zeros((4, 4, 3, 3))
    for c in range(4):
        w[c, c, 1, 1] = 1.0
    y = E.conv2d(x, w, pad=(1, 1))
    np.testing.assert_array_equal(y, x)
    y = E.conv2d(x, w, pad=(1, 1), post_relu=True)
    np.testing.assert_array_equal(y, np.maximum(x, 0))
    y = E.conv2d(x, -w, pad=(1, 1), pre_relu=True)
    np.testing.assert_array_equal(y, -np.maximum(x, 0))


def test_conv_constant_input_counts_in_bounds_taps():
    x = np.ones((1, 2, 5, 5))
    w = np.ones((1, 2, 3, 3))
    y = E.conv2d(x, w, pad=(1, 1))[0, 0]
    # corner: 2x2 taps in bounds per channel -> 8 ; edge: 2x3 -> 12 ; interior: 18
    assert y[0, 0] == 8 and y[0, 2] == 12 and y[2, 2] == 18 and y[4, 4] == 8


@pytest.mark.parametrize("k,s,p", [(1, 1, 0), (3, 1, 1), (5, 1, 2), (3, 2, 0), (3, 2, 1)])
def test_conv_matches_torch_cpu_float64(k, s, p):
    x = rnd((2, 5, 11, 9), 4)
    w = rnd((6, 5, k, k), 5)
    b = rnd((6,), 6)
    y = E.conv2d(x, w, b, (s, s), (p, p), post_relu=True)
    ref = torch.relu(F.conv2d(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b),
                              stride=s, padding=p)).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_asymmetric_kernel_matches_torch():
    x = rnd((1, 3, 8, 8), 7)
    w = rnd((4, 3, 3, 1), 8)
    y = E.conv2d(x, w, None, (1, 1), (1, 0))
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(w), padding=(1, 0)).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k", [3, 5])
def test_depthwise_matches_grouped_conv(k):
    x = rnd((2, 6, 9, 10), 9)
    w = rnd((6, 1, k, k), 10)
    y = E.depthwise(x, w, (k // 2, k // 2))
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(w), padding=k // 2, groups=6).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_avgpool_border_factors():
    x = np.ones((1, 1, 5, 5))
    y = E.pool(x, 3, 1, 1, is_max=False)[0, 0]
    assert y[0, 0] == 4 / 9 and y[0, 2] == 6 / 9 and y[2, 2] == 1.0


def test_pools_match_torch():
    x = rnd((2, 3, 11, 11), 11)
    t = torch.from_numpy(x)
    np.testing.assert_allclose(E.pool(x, 3, 1, 1, False),
                               F.avg_pool2d(t, 3, 1, 1, count_include_pad=True).numpy(), rtol=1e-12)
    np.testing.assert_array_equal(E.pool(x, 3, 1, 1, True), F.max_pool2d(t, 3, 1, 1).numpy())
    np.testing.assert_array_equal(E.pool(x, 3, 2, 0, True), F.max_pool2d(t, 3, 2, 0).numpy())


def test_maxpool_negative_input_ignores_padding():
    x = -np.ones((1, 1, 4, 4)) - np.arange(16).reshape(1, 1, 4, 4)
    y = E.pool(x, 3, 1, 1, True)
    assert y.max() < 0          # zero padding would have produced 0
    assert y[0, 0, 0, 0] == -1.0


def test_maxpool_s2_sizes():
    x = rnd((1, 2, 55, 55), 12)
    assert E.pool(x, 3, 2, 0, True).shape[-1] == 27
    assert E.pool(rnd((1, 2, 27, 27), 1), 3, 2, 0, True).shape[-1] == 13


def test_sepconv_unit_definition():
    a, b = rnd((1, 4, 7, 7), 13), rnd((1, 4, 7, 7), 14)
    dw, pw = rnd((4, 1, 3, 3), 15), rnd((5, 4, 1, 1), 16)
    y = E.sepconv([a, b], dw, pw, None, (1, 1))
    t = torch.relu(torch.from_numpy(a + b))
    t = F.conv2d(t, torch.from_numpy(dw), padding=1, groups=4)
    ref = F.conv2d(t, torch.from_numpy(pw)).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("kinds", [[(1, 0), (3, 1)], [(1, 0), (5, 2), (3, 1)], [(1, 0), (1, 0)]])
def test_merged_conv_equals_separate(kinds):
    x = rnd((2, 6, 9, 9), 17)
    convs = []
    for i, (k, p) in enumerate(kinds):
        convs.append({"w": rnd((3 + i, 6, k, k), 20 + i), "b": rnd((3 + i,), 30 + i),
                      "pad": (p, p), "post_relu": 1})
    parts = E.merged_conv(x, convs)
    for c, part in zip(convs, parts):
        ref = E.conv2d(x, c["w"], c["b"], (1, 1), c["pad"], post_relu=True)
        np.testing.assert_array_equal(part, ref)


def test_merged_asymmetric_3x1_1x3():
    # the 3x1 / 1x3 pair padded to 3x3 (Sec. 7.2, last Inception block)
    x = rnd((1, 4, 8, 8), 40)
    convs = [{"w": rnd((2, 4, 3, 1), 41), "b": None, "pad": (1, 0), "post_relu": 1},
             {"w": rnd((3, 4, 1, 3), 42), "b": None, "pad": (0, 1), "post_relu": 1}]
    parts = E.merged_conv(x, convs)
    for c, part in zip(convs, parts):
        np.testing.assert_array_equal(part, E.conv2d(x, c["w"], None, (1, 1), c["pad"], post_relu=True))


def test_config_shapes_and_concat_widths():
    shp = W.infer_shapes(W.make("tiny")[0])
    assert shp["out"] == (32, 8, 8)
    assert W.infer_shapes(W.make("inception")[0])["out"] == (256, 35, 35)
    assert W.infer_shapes(W.make("nasnet")[0])["out"] == (840, 42, 42)
    sq = W.infer_shapes(W.make("squeeze")[0])
    assert sq["pool3"] == (256, 27, 27) and sq["pool7"] == (512, 13, 13) and sq["m8"] == (512, 13, 13)
    rw = W.make("randwire")[0]
    assert len(W.unit_ops(rw)) == 33


def test_evaluate_inception_against_torch_float64():
    spec, ten = W.make("inception")
    out = E.outputs(spec, ten)[0]
    T = {k: torch.from_numpy(v.astype(np.float64)) for k, v in ten.items()}
    x = T["x"]
    c = lambda t, n, p: torch.relu(F.conv2d(t, T[n + ".w"], T[n + ".b"], padding=p))
    b1 = c(x, "b1", 0)
    b2 = c(c(x, "b2a", 0), "b2b", 2)
    b3 = c(c(c(x, "b3a", 0), "b3b", 1), "b3c", 1)
    b4 = c(F.avg_pool2d(x, 3, 1, 1, count_include_pad=True), "b4", 0)
    ref = torch.cat([b1, b2, b3, b4], 1).numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-11, atol=1e-11)


def _elt_spec(kind, n_in, c=3, h=4, w=5):
    ins = [{"name": f"x{i}", "c": c, "h": h, "w": w} for i in range(n_in)]
    return {"name": "elt", "batch": 1, "inputs": ins,
            "ops": [{"name": "y", "kind": kind, "in": [f"x{i}" for i in range(n_in)]}],
            "outputs": ["y"]}


def test_add_and_mean_closed_forms():
    """ADD / MEAN (sink mean of RandWire, NASNet's add) pinned by facts that
    hold whatever the summation order: x + (-x) = 0; k copies of x add to
    k x and average to x (inputs are 24-bit uniforms, so k x is exact in
    float64); hand values on small integers."""
    u = W.make("tiny")[1]["x"][:, :3, :4, :5].astype(np.float64)
    env = E.evaluate(_elt_spec("add", 2), {"x0": u, "x1": -u})
    assert np.array_equal(env["y"], np.zeros_like(u))
    for k in (1, 2, 3, 5):
        ten = {f"x{i}": u for i in range(k)}
        assert np.array_equal(E.evaluate(_elt_spec("add", k), ten)["y"], k * u)
        assert np.array_equal(E.evaluate(_elt_spec("mean", k), ten)["y"], u)
    a = np.arange(60, dtype=np.float64).reshape(1, 3, 4, 5)
    b = np.full((1, 3, 4, 5), 7.0)
    c = 2 * np.ones((1, 3, 4, 5))
    y = E.evaluate(_elt_spec("add", 3), {"x0": a, "x1": b, "x2": c})["y"]
    assert y[0, 0, 0, 0] == 9.0 and y[0, 2, 3, 4] == 68.0
    y = E.evaluate(_elt_spec("mean", 3), {"x0": a, "x1": b, "x2": c})["y"]
    assert y[0, 0, 0, 0] == 3.0 and y[0, 0, 3, 3] == 9.0 and y[0, 2, 3, 4] == 68.0 / 3.0
    y = E.evaluate(_elt_spec("mean", 2), {"x0": a, "x1": -a})["y"]
    assert np.array_equal(y, np.zeros_like(a))


def test_evaluate_mean_and_add_wiring():
    """The workloads wire ADD / MEAN as their descriptions say: RandWire's
    output is the mean of its sinks, NASNet's concat holds the five adds."""
    spec, ten = W.make("randwire")
    env = E.evaluate(spec, ten)
    sinks = spec["ops"][-1]["in"]
    assert spec["ops"][-1]["kind"] == "mean" and len(sinks) >= 1
    spec, ten = W.make("nasnet")
    env = E.evaluate(spec, ten)
    for b in range(5):
        np.testing.assert_array_equal(env["out"][:, 168 * b:168 * (b + 1)], env[f"add{b}"])


# ------------------------------------------------------------------ schedule invariance

def evaluate_schedule(spec, ten, blocks, stages):
    """Evaluate a block stage by stage (Sec. 3): each stage's units in
    ascending order (a group's chain in order), a merge stage as ONE
    convolution with the stacked, centred kernels, split back per unit; views
    as soon as their inputs exist."""
    from oracle import schedule as O
    env = {t["name"]: ten[t["name"]].astype(np.float64) for t in spec["inputs"]}
    views = [op for op in spec["ops"] if op["kind"] in ("concat", "identity")]

    def settle():
        for op in views:
            if op["name"] not in env and all(i in env for i in op["in"]):
                env[op["name"]] = E.eval_op(op, env, ten)
                settle()
                return
    for b, (mask, strat) in stages:
        us = [blocks[b].units[i] for i in O.bits(mask)]
        if strat == O.MERGE:
            convs = [{"w": ten[u["name"] + ".w"], "b": ten.get(u["name"] + ".b"), "pad": (u["ph"], u["pw"]),
                      "pre_relu": u.get("pre_relu", 0), "post_relu": u.get("post_relu", 0)} for u in us]
            parts = E.merged_conv(env[us[0]["in"][0]], convs, (us[0]["sh"], us[0]["sw"]))
            for u, part in zip(us, parts):
                env[u["name"]] = part
        else:
            for u in us:
                env[u["name"]] = E.eval_op(u, env, ten)
        settle()
    return [env[o] for o in spec["outputs"]]


def _schedules_with_strategies(blk, masks):
    """Every strategy assignment of one mask schedule: merge where allowed."""
    from oracle import schedule as O
    out = [[]]
    for m in masks:
        opts = [O.CONCURRENT] + ([O.MERGE] if O.mergeable(blk, m) else [])
        out = [q + [(m, t)] for q in out for t in opts]
    return out


def test_every_schedule_gives_identical_outputs_tiny():
    """Sec. 3: a schedule changes when operators run, never what they
    compute.  Every schedule of the tiny block (8 partitions, merge wherever
    it is allowed) gives outputs bit-identical to plain evaluation."""
    from oracle import schedule as O
    spec, ten = W.make("tiny", 2, 1)
    ref = E.outputs(spec, ten)
    blk = O.blocks_of(spec)[0]
    n = 0
    for masks in O.all_schedules(blk):
        for q in _schedules_with_strategies(blk, masks):
            out = evaluate_schedule(spec, ten, [blk], [(0, st) for st in q])
            for a, b in zip(out, ref):
                assert np.array_equal(a, b)
            n += 1
    assert n == 8 + 1     # {A, B1} can merge in the one partition that holds it as a stage


def test_sampled_schedules_give_identical_outputs_inception():
    """The same on the Inception block: 24 of its 34,516 schedules, drawn
    with a fixed seed, each with merge on every mergeable stage."""
    from oracle import schedule as O
    spec, ten = W.make("inception")
    ref = E.outputs(spec, ten)
    blk = O.blocks_of(spec)[0]
    all_q = list(O.all_schedules(blk))
    assert len(all_q) == 34516
    pick = np.random.default_rng(7).choice(len(all_q), 24, replace=False)
    merged = 0
    for i in pick:
        q = [(m, O.MERGE if O.mergeable(blk, m) else O.CONCURRENT) for m in all_q[i]]
        merged += sum(t == O.MERGE for _, t in q)
        out = evaluate_schedule(spec, ten, [blk], [(0, st) for st in q])
        for a, b in zip(out, ref):
            assert np.array_equal(a, b)
    assert merged > 0
