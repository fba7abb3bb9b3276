"""Host-side tests of the C-ABI library (no GPU): exported symbols, graph
building and its error paths, and the schedule search checked against the
oracle (Algorithm 1 and brute force) through an injected cost table."""
import os
import random
import re

import numpy as np
import pytest

import paper_2011_01302_amd as I
from oracle import schedule as O
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_symbols():
    txt = open(os.path.join(ROOT, "include", "ios.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(ios_[a-z_]+)\s*\(", txt)) - {"ios_cost_fn"})


def test_library_exports_every_declared_symbol():
    syms = header_symbols()
    assert len(syms) >= 20
    for s in syms:
        assert hasattr(I._lib, s), s
    assert sorted(I.EXPORTED) == syms


# ------------------------------------------------------------------ helpers

def table_cost(seed, hi=10_000, lo=1):
    """A seeded synthetic cost table keyed by (block, mask, strategy)."""
    memo = {}
    rnd = random.Random(seed)

    def cost(block, mask, strategy):
        k = (block, mask, strategy)
        if k not in memo:
            memo[k] = rnd.randint(lo, hi)
        return memo[k]
    return cost


def lib_schedule(g, cost, r=3, s=8, strategies=3, mode=I.IOS_SCHED_DP):
    o = I.ios_sched_opts_default()
    o.r, o.s, o.strategies, o.mode = r, s, strategies, mode
    q, c = I.ios_schedule(g.handle, o, lambda b, m, ids, t: cost(b, m, t))
    sched = I.ios_schedule_get(q)
    stats = I.ios_schedule_stats(q)
    I.ios_schedule_destroy(q)
    return c, sched, stats


def oracle_schedule(spec, cost, r=3, s=8, strategies=(0, 1)):
    total, out, states, trans = 0, [], 0, 0
    for b, blk in enumerate(O.blocks_of(spec)):
        res = O.ios_dp(blk, lambda m, t: cost(b, m, t), r, s, strategies)
        total += res.cost
        states += res.states
        trans += res.transitions
        for m, t in res.schedule:
            out.append((sorted(blk.units[i]["name"] for i in O.bits(m)), t))
    return total, out, states, trans


def names(g, sched):
    return [(sorted(g.names(ids)), t) for ids, t in sched]


# ------------------------------------------------------------------ schedule parity

@pytest.mark.parametrize("config,seed", [("tiny", 0), ("tiny", 1), ("inception", 0),
                                         ("inception", 1), ("squeeze", 0), ("randwire", 0),
                                         ("nasnet", 0), ("nasnet", 2)])
def test_dp_matches_oracle_dp_on_configs(config, seed):
    spec, ten = W.make(config, 1, seed)
    g = I.Graph(spec, ten)
    for table_seed, hi in [(100, 10_000), (101, 40)]:          # hi=40: many ties
        cost = table_cost(table_seed, hi=hi)
        c, sched, (states, trans, _) = lib_schedule(g, cost)
        oc, osched, ostates, otrans = oracle_schedule(spec, cost)
        assert c == oc
        assert names(g, sched) == osched
        assert (states, trans) == (ostates, otrans)
    g.close()


@pytest.mark.parametrize("strategies,ostrat", [(1, (0,)), (2, (1,)), (3, (0, 1))])
def test_strategy_variants_match_oracle(strategies, ostrat):
    for config in ["tiny", "inception", "squeeze"]:
        spec, ten = W.make(config)
        g = I.Graph(spec, ten)
        cost = table_cost(7)
        c, sched, _ = lib_schedule(g, cost, strategies=strategies)
        oc, osched, _, _ = oracle_schedule(spec, cost, strategies=ostrat)
        assert c == oc and names(g, sched) == osched
        if strategies == 1:
            assert all(t == I.IOS_CONCURRENT for _, t in sched)
        if strategies == 2:
            assert all(len(ids) == 1 or t == I.IOS_MERGE for ids, t in sched)
        g.close()


def add_dag_spec(n, edges):
    """A block of n ADD units wired by `edges` (sources read the input)."""
    preds = {v: [a for a, b in edges if b == v] for v in range(n)}
    ops = [{"name": f"u{v}", "kind": "add", "in": [f"u{p}" for p in preds[v]] or ["x"]}
           for v in range(n)]
    return {"name": "dag", "batch": 1, "inputs": [{"name": "x", "c": 2, "h": 3, "w": 3}],
            "ops": ops, "outputs": [f"u{v}" for v in range(n)
                                    if not any(a == v for a, _ in edges)]}


def test_dp_matches_brute_force_random_dags():
    rnd = random.Random(5)
    for trial in range(120):
        n = rnd.randint(1, 7)
        p = rnd.random() * 0.7
        edges = [(a, b) for a in range(n) for b in range(a + 1, n) if rnd.random() < p]
        spec = add_dag_spec(n, edges)
        g = I.Graph(spec, {})
        r, s = rnd.choice([0, 1, 2, 3]), rnd.choice([0, 1, 2, 3, 8])
        cost = table_cost(trial, hi=rnd.choice([3, 20, 1000]))
        c, sched, _ = lib_schedule(g, cost, r=r, s=s)
        blk = O.blocks_of(spec)[0]
        bc, bq, _ = O.brute_force(blk, lambda m, t: cost(0, m, t), r or None, s or None)
        assert c == bc
        assert names(g, sched) == [(sorted(f"u{i}" for i in O.bits(m)), t) for m, t in bq]
        g.close()


def test_fig5_state_space_through_the_library():
    g = I.Graph(add_dag_spec(3, [(0, 1)]), {})
    c, sched, (states, trans, measured) = lib_schedule(g, lambda b, m, t: 1, r=0, s=0)
    assert (states, trans) == (6, 12)
    assert c == 1                    # one stage: groups {a, b} and {c}
    g.close()


def test_baseline_schedules():
    spec, ten = W.make("inception")
    g = I.Graph(spec, ten)
    cost = table_cost(3)
    c_seq, seq, _ = lib_schedule(g, cost, mode=I.IOS_SCHED_SEQUENTIAL)
    assert [len(ids) for ids, _ in seq] == [1] * 8
    assert [g.names(ids)[0] for ids, _ in seq] == [u["name"] for u in W.unit_ops(spec)]
    c_gr, gr, _ = lib_schedule(g, cost, mode=I.IOS_SCHED_GREEDY)
    assert [sorted(g.names(ids)) for ids, _ in gr] == [
        ["b1", "b2a", "b3a", "pool"], ["b2b", "b3b", "b4"], ["b3c"]]
    c_dp, _, _ = lib_schedule(g, cost)
    assert c_dp <= c_seq and c_dp <= c_gr
    g.close()


def test_schedule_from_stages_validation():
    spec, ten = W.make("tiny")
    g = I.Graph(spec, ten)
    A, B1, B2 = (g.tid[n] for n in ("A", "B1", "B2"))
    q = I.ios_schedule_from_stages(g.handle, [[A, B1], [B2]], [I.IOS_MERGE, I.IOS_CONCURRENT])
    assert I.ios_schedule_get(q) == [([A, B1], 1), ([B2], 0)]
    I.ios_schedule_destroy(q)
    q = I.ios_schedule_from_stages(g.handle, [[B1, B2, A]], [I.IOS_CONCURRENT])
    I.ios_schedule_destroy(q)
    bad = [([[A], [B2], [B1]], [0, 0, 0], "IOS_E_BAD_STAGE"),      # consumer before producer
           ([[A, B1]], [0], "IOS_E_BAD_STAGE"),                    # B2 missing
           ([[A], [B1, B2]], [0, 1], "IOS_E_NOT_MERGEABLE"),       # chain cannot merge
           ([[A, A, B1], [B2]], [0, 0], "IOS_E_BAD_STAGE")]
    for stages, strat, err in bad:
        with pytest.raises(I.IosError) as e:
            I.ios_schedule_from_stages(g.handle, stages, strat)
        assert e.value.name == err
    assert I.ios_stage_mergeable(g.handle, [A, B1])
    assert not I.ios_stage_mergeable(g.handle, [A, B2])
    g.close()


def test_mergeable_agrees_with_oracle():
    for config in ["tiny", "inception", "squeeze"]:
        spec, ten = W.make(config)
        g = I.Graph(spec, ten)
        for b, blk in enumerate(O.blocks_of(spec)):
            ids = I.ios_block_units(g.handle, b)
            for m in range(1, 1 << blk.n):
                sel = [ids[i] for i in O.bits(m)]
                assert I.ios_stage_mergeable(g.handle, sel) == O.mergeable(blk, m), (config, m)
        g.close()


def test_blocks_match_oracle():
    for config in W.CONFIG_NAMES:
        spec, ten = W.make(config)
        g = I.Graph(spec, ten)
        lib = [g.names(b) for b in g.blocks()]
        orc = [[u["name"] for u in blk.units] for blk in O.blocks_of(spec)]
        assert lib == orc
        g.close()


# ------------------------------------------------------------------ error paths

def desc(kind, cout=0, k=1, s=1, p=0, pre=0, post=0, block=-1):
    d = I.ios_op_desc()
    d.kind, d.cout, d.kh, d.kw, d.stride_h, d.stride_w = kind, cout, k, k, s, s
    d.pad_h, d.pad_w, d.pre_relu, d.post_relu, d.block_id = p, p, pre, post, block
    return d


def expect(err, fn, *a):
    with pytest.raises(I.IosError) as e:
        fn(*a)
    assert e.value.name == err, e.value


def test_graph_error_paths():
    g = I.ios_graph_create(1)
    x = I.ios_add_input(g, 4, 5, 5)
    w = np.zeros((3, 4, 3, 3), np.float32)
    expect("IOS_E_ARG", I.ios_add_input, g, 0, 5, 5)
    expect("IOS_E_ARG", I.ios_add_op, g, desc(I.IOS_CONV, 3, 3), [99], w)
    expect("IOS_E_ARG", I.ios_add_op, g, desc(I.IOS_CONV, 3, 3), [x], None)   # no weights
    expect("IOS_E_SHAPE", I.ios_add_op, g, desc(I.IOS_CONV, 3, 7), [x], np.zeros(3 * 4 * 49, np.float32))
    expect("IOS_E_UNSUPPORTED", I.ios_add_op, g, desc(I.IOS_CONCAT), [x])     # concat of an input
    y = I.ios_add_input(g, 5, 5, 5)
    expect("IOS_E_SHAPE", I.ios_add_op, g, desc(I.IOS_ADD), [x, y])
    expect("IOS_E_STATE", I.ios_graph_blocks, g)
    expect("IOS_E_STATE", I.ios_schedule, g, None, lambda *a: 1)
    expect("IOS_E_STATE", I.ios_get_conv_tile, g, x)
    expect("IOS_E_STATE", I.ios_schedule_tune_tiles, g, None)
    expect("IOS_E_UNSUPPORTED", I.ios_mark_output, g, x)
    c = I.ios_add_op(g, desc(I.IOS_CONV, 3, 3, p=1), [x], w)
    cat = I.ios_add_op(g, desc(I.IOS_CONCAT), [c])
    expect("IOS_E_UNSUPPORTED", I.ios_add_op, g, desc(I.IOS_CONCAT), [c])    # already in a concat
    expect("IOS_E_UNSUPPORTED", I.ios_mark_output, g, c)                     # slice of a concat
    I.ios_mark_output(g, cat)
    I.ios_graph_finalize(g)
    expect("IOS_E_STATE", I.ios_graph_finalize, g)
    expect("IOS_E_STATE", I.ios_add_input, g, 1, 1, 1)
    expect("IOS_E_ARG", I.ios_profile_stage, g, [x])                          # not a unit
    expect("IOS_E_ARG", I.ios_block_units, g, 5)
    # conv tile shapes: argument errors come before any device work
    expect("IOS_E_ARG", I.ios_get_conv_tile, g, x)                            # not a unit
    expect("IOS_E_ARG", I.ios_set_conv_tile, g, c, I.IOS_CONV_TILE_SHAPES)
    expect("IOS_E_ARG", I.ios_set_conv_tile, g, c, -1)
    for pipelined in range(6, 12):                                            # 4 input channels, not 16k
        expect("IOS_E_ARG", I.ios_set_conv_tile, g, c, pipelined)
        expect("IOS_E_ARG", I.ios_set_unit_tiling, g, c, pipelined, -1)
    # per-stage tile choice: argument errors come before any device work
    q = I.ios_schedule_from_stages(g, [[c]], [I.IOS_CONCURRENT])
    o = I.ios_sched_opts_default()
    o.reps = 0
    expect("IOS_E_ARG", I.ios_schedule_tune_tiles, g, q, o)
    expect("IOS_E_ARG", I.ios_schedule_tune_tiles, g, None)
    g2 = I.ios_graph_create(1)
    y2 = I.ios_add_input(g2, 1, 2, 2)
    I.ios_mark_output(g2, I.ios_add_op(g2, desc(I.IOS_ADD), [y2]))
    I.ios_graph_finalize(g2)
    expect("IOS_E_ARG", I.ios_schedule_tune_tiles, g2, q)                    # another graph's schedule
    I.ios_graph_destroy(g2)
    I.ios_schedule_destroy(q)
    I.ios_graph_destroy(g)
    expect("IOS_E_ARG", I.ios_graph_create, 0)


def test_too_many_units_in_a_block():
    g = I.ios_graph_create(1)
    x = I.ios_add_input(g, 1, 2, 2)
    for i in range(65):
        I.ios_add_op(g, desc(I.IOS_ADD, block=0), [x])
    expect("IOS_E_TOO_MANY_OPS", I.ios_graph_finalize, g)
    I.ios_graph_destroy(g)
    # automatic blocks: 65 independent units cannot be cut
    g = I.ios_graph_create(1)
    x = I.ios_add_input(g, 1, 2, 2)
    for i in range(65):
        I.ios_add_op(g, desc(I.IOS_ADD), [x])
    expect("IOS_E_TOO_MANY_OPS", I.ios_graph_finalize, g)
    I.ios_graph_destroy(g)


def test_automatic_blocks_cut_long_chains():
    g = I.ios_graph_create(1)
    t = I.ios_add_input(g, 1, 2, 2)
    for i in range(70):
        t = I.ios_add_op(g, desc(I.IOS_ADD), [t])
    I.ios_graph_finalize(g)
    assert I.ios_graph_blocks(g) == 70          # every unit of a chain is a cut unit
    I.ios_graph_destroy(g)


def test_block_order_must_follow_edges():
    g = I.ios_graph_create(1)
    x = I.ios_add_input(g, 1, 2, 2)
    a = I.ios_add_op(g, desc(I.IOS_ADD, block=1), [x])
    I.ios_add_op(g, desc(I.IOS_ADD, block=0), [a])
    expect("IOS_E_BAD_STAGE", I.ios_graph_finalize, g)
    I.ios_graph_destroy(g)


def test_cost_callback_errors_propagate():
    spec, ten = W.make("tiny")
    g = I.Graph(spec, ten)

    def boom(b, m, ids, t):
        raise ValueError("no latency")

    with pytest.raises(I.IosError) as e:
        I.ios_schedule(g.handle, None, boom)
    assert e.value.name == "IOS_E_COST_FN"
    o = I.ios_sched_opts_default()
    o.strategies = 0
    with pytest.raises(I.IosError) as e:
        I.ios_schedule(g.handle, o, lambda *a: 1)
    assert e.value.name == "IOS_E_ARG"
    g.close()


def test_cost_table_dump(tmp_path):
    spec, ten = W.make("tiny")
    g = I.Graph(spec, ten)
    cost = table_cost(9)
    lib_schedule(g, cost)
    p = tmp_path / "costs.jsonl"
    I.ios_schedule_dump_costs(g.handle, str(p))
    import json
    rows = [json.loads(l) for l in open(p)]
    assert len(rows) == 7                           # distinct S' of the tiny block
    for r in rows:
        assert r["concurrent_ns"] == cost(r["block"], r["mask"], 0)
        blk = O.blocks_of(spec)[0]
        if O.mergeable(blk, r["mask"]):
            assert r["merge_ns"] == cost(r["block"], r["mask"], 1)
        else:
            assert r["merge_ns"] is None
    g.close()


def test_line_sep_tile_refused_where_it_does_not_apply():
    """The line SEPCONV tile choices (9: 32 output channels, 10: 64) take
    3x3 windows that keep the plane size, rows of a multiple of 4 floats up
    to 32 and at most 96 input channels; the two-block choice needs more than
    32 output channels.  Every other case is refused before any device work."""
    g = I.ios_graph_create(1)

    def sep(c, h, w, cout, k):
        x = I.ios_add_input(g, c, h, w)
        wts = np.zeros(c * k * k + cout * c, np.float32)
        return I.ios_add_op(g, desc(I.IOS_SEPCONV, cout, k, p=k // 2), [x], wts)
    cases = {
        "width 6": (sep(8, 6, 6, 40, 3), (9, 10)),
        "width 40": (sep(8, 40, 40, 40, 3), (9, 10)),
        "97 channels": (sep(97, 8, 8, 40, 3), (9, 10)),
        "5x5 window": (sep(8, 8, 8, 40, 5), (9, 10)),
        "32 outputs": (sep(8, 8, 8, 32, 3), (10,)),
    }
    for name, (u, tiles) in cases.items():
        I.ios_mark_output(g, u)
    I.ios_graph_finalize(g)
    for name, (u, tiles) in cases.items():
        for t in tiles:
            expect("IOS_E_ARG", I.ios_set_unit_tiling, g, u, t, -1)
        expect("IOS_E_ARG", I.ios_set_unit_tiling, g, u, 11, -1)             # past the last choice
    I.ios_graph_destroy(g)
