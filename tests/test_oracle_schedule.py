"""Pins for the schedule oracle: the paper's worked example (Fig. 5), the
closed forms of the complexity analysis (Sec. 4.2, App. A), Lemma 1 and 2,
known counts (compositions, ordered set partitions) and brute force."""
import itertools
import json
import math
import os
import random

import pytest

from oracle import schedule as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def random_dag(n, p, rnd):
    return O.block_from_edges(n, [(a, b) for a in range(n) for b in range(a + 1, n)
                                  if rnd.random() < p])


def test_fig5_states_transitions():
    g = json.load(open(os.path.join(GOLDEN, "fig5_worked_example.json")))
    blk = O.block_from_edges(len(g["units"]), [tuple(e) for e in g["edges"]])
    res = O.ios_dp(blk, lambda m, t: 1)
    assert res.states == g["states"]
    assert res.transitions == g["transitions"]
    assert sum(1 for _ in O.all_schedules(blk)) == 8


def test_fig5_memo_revisits_state_a():
    # the state {a} is reached more than once (the paper's step 7 finds it in
    # the memo after step 2): {a,b,c} - {b,c}, {a,b} - {b} and {a,c} - {c}.
    blk = O.block_from_edges(3, [(0, 1)])
    hits = 0
    for S in [0b111, 0b011, 0b101, 0b001, 0b100]:
        for Sp in O.endings(blk, S):
            if S & ~Sp == 0b001:
                hits += 1
    assert hits == 3


@pytest.mark.parametrize("c,d", [(1, 1), (2, 2), (3, 2), (2, 3), (3, 3), (4, 2), (1, 4)])
def test_independent_chains_closed_form(c, d):
    # App. A tight example: d independent chains of c operators.
    n = c * d
    edges = [(i * c + j, i * c + j + 1) for i in range(d) for j in range(c - 1)]
    blk = O.block_from_edges(n, edges)
    res = O.ios_dp(blk, lambda m, t: 1)
    assert res.states == (c + 1) ** d
    assert res.transitions == math.comb(c + 2, 2) ** d - (c + 1) ** d
    assert res.transitions <= O.transition_bound(n, d)


@pytest.mark.parametrize("n", range(1, 8))
def test_schedule_counts_chain_and_antichain(n):
    chain = O.block_from_edges(n, [(i, i + 1) for i in range(n - 1)])
    assert sum(1 for _ in O.all_schedules(chain)) == 2 ** (n - 1)   # compositions of n
    anti = O.block_from_edges(n, [])
    if n <= 6:
        assert sum(1 for _ in O.all_schedules(anti)) == O.fubini(n)  # ordered set partitions
    assert O.fubini(n) == [1, 1, 3, 13, 75, 541, 4683, 47293][n]


def test_endings_definitions_agree_random():
    rnd = random.Random(0)
    for _ in range(150):
        n = rnd.randint(1, 9)
        blk = random_dag(n, rnd.random() * 0.6, rnd)
        r = rnd.choice([None, 1, 2, 3])
        s = rnd.choice([None, 1, 2, 3, 8])
        S = rnd.randint(1, blk.full)
        # restrict to down-sets, the only states Scheduler sees (Lemma 2)
        down = S
        for u in range(n):
            if down >> u & 1 and blk.pred[u] & ~down:
                down &= ~(1 << u)
        for state in (blk.full, down):
            if state:
                assert O.endings(blk, state, r, s) == O.endings_plain(blk, state, r, s)


def test_lemma1_union_of_endings_is_ending():
    rnd = random.Random(1)
    for _ in range(100):
        n = rnd.randint(2, 8)
        blk = random_dag(n, 0.4, rnd)
        S = blk.full
        for S1 in O.endings_plain(blk, S):
            for S2 in O.endings_plain(blk, S & ~S1):
                assert O.is_ending(blk, S, S1 | S2)


def test_lemma2_states_are_complements_of_endings():
    rnd = random.Random(2)
    for _ in range(60):
        n = rnd.randint(1, 8)
        blk = random_dag(n, 0.4, rnd)
        seen = set()

        def walk(S):
            if S in seen:
                return
            seen.add(S)
            for Sp in O.endings(blk, S):
                walk(S & ~Sp)

        walk(blk.full)
        for S in seen:
            if S != blk.full:
                assert O.is_ending(blk, blk.full, blk.full & ~S)


def test_dp_equals_brute_force_random():
    rnd = random.Random(3)
    for trial in range(250):
        n = rnd.randint(1, 7)
        blk = random_dag(n, rnd.random() * 0.7, rnd)
        r = rnd.choice([None, 1, 2, 3])
        s = rnd.choice([None, 1, 2, 3, 8])
        hi = rnd.choice([2, 4, 50])
        table = {}

        def cost(m, t):
            key = (m, t)
            if key not in table:
                table[key] = rnd.randint(1, hi)
            return table[key]

        # the merge rule needs conv units; make the bare units mergeable at random
        merge_ok = {m: rnd.random() < 0.3 for m in range(1 << n)}
        orig = O.mergeable
        O.mergeable = lambda b, m: bin(m).count("1") >= 2 and merge_ok[m]
        try:
            dp = O.ios_dp(blk, cost, r, s)
            bf_cost, bf_q, count = O.brute_force(blk, cost, r, s)
        finally:
            O.mergeable = orig
        assert dp.cost == bf_cost
        assert dp.schedule == bf_q, (trial, dp.schedule, bf_q)


def test_dp_additive_costs_prefer_smallest_masks():
    # every schedule ties when a stage costs the sum of its units
    blk = O.block_from_edges(4, [(0, 1), (2, 3)])
    res = O.ios_dp(blk, lambda m, t: bin(m).count("1"))
    bf = O.brute_force(blk, lambda m, t: bin(m).count("1"))
    assert res.cost == 4 and res.schedule == bf[1]


def test_dp_constant_stage_cost_minimises_stage_count():
    # constant cost per stage: the optimum is the fewest stages allowed by P
    blk = O.block_from_edges(6, [(0, 1), (1, 2), (3, 4)])
    assert O.ios_dp(blk, lambda m, t: 10).cost == 10            # one stage, no pruning
    assert O.ios_dp(blk, lambda m, t: 10, r=2, s=8).cost == 20   # chain of 3 > r=2
    assert O.ios_dp(blk, lambda m, t: 10, r=1, s=8).cost == 30   # longest chain has 3 units
    assert O.ios_dp(blk, lambda m, t: 10, r=3, s=1).cost == 30   # 3 components, one per stage


def test_generate_stage_tie_prefers_merge():
    spec = W.make("tiny")[0]
    blk = O.blocks_of(spec)[0]
    assert O.mergeable(blk, 0b011)          # A and B1: 1x1 on x
    assert not O.mergeable(blk, 0b110)      # B1 -> B2 are not on the same input
    assert O.generate_stage(blk, 0b011, lambda m, t: 5) == (5, O.MERGE)
    assert O.generate_stage(blk, 0b011, lambda m, t: 5 - t) == (4, O.MERGE)
    assert O.generate_stage(blk, 0b011, lambda m, t: 5 + t) == (5, O.CONCURRENT)


def test_ios_merge_variant_runs_single_units_alone():
    """IOS-Merge (Sec. 6.1: operator merge only, no concurrent execution).
    A stage of one operator is that operator, so it still runs; a stage of
    several operators exists only if they merge.  (1) With no mergeable set
    the only schedules left are the n! / (orderings allowed by the edges)
    sequences of single units, each costing the sum of the singles.  (2) On
    the tiny block the two IOS-Merge schedules are, by hand,
    singles in some order, 3 + 4 + 6 = 13, and merge{A, B1} {B2} = 5 + 6 = 11;
    among the equal-cost orders of the singles the tie-break on the last
    stage's mask puts {A} (mask 1) last: {B1} {B2} {A}."""
    rnd = random.Random(11)
    for trial in range(30):
        n = rnd.randint(1, 6)
        blk = random_dag(n, 0.4, rnd)          # abstract units: nothing merges
        single = {1 << i: rnd.randint(1, 9) for i in range(n)}
        cost = lambda m, t: single.get(m, 1000)
        res = O.ios_dp(blk, cost, strategies=(O.MERGE,))
        assert res.cost == sum(single.values())
        assert all(m & (m - 1) == 0 for m, _ in res.schedule)
        assert sorted(m for m, _ in res.schedule) == sorted(single)
    blk = O.blocks_of(W.make("tiny")[0])[0]    # units A, B1, B2 (B1 -> B2)
    table = {(0b001, O.CONCURRENT): 3, (0b010, O.CONCURRENT): 4, (0b100, O.CONCURRENT): 6,
             (0b011, O.MERGE): 5}
    cost = lambda m, t: table.get((m, t), 100)
    res = O.ios_dp(blk, cost, strategies=(O.MERGE,))
    assert res.cost == 11 and res.schedule == [(0b011, O.MERGE), (0b100, O.CONCURRENT)]
    table[(0b011, O.MERGE)] = 8                 # now merging loses: 8 + 6 > 13
    res = O.ios_dp(blk, cost, strategies=(O.MERGE,))
    assert res.cost == 13 and [m for m, _ in res.schedule] == [0b010, 0b100, 0b001]


def test_merge_rules_on_configs():
    blk = O.blocks_of(W.make("inception")[0])[0]
    names = [u["name"] for u in blk.units]
    m = lambda *ns: sum(1 << names.index(x) for x in ns)
    assert O.mergeable(blk, m("b1", "b2a", "b3a"))
    assert not O.mergeable(blk, m("b1", "b4"))            # different inputs
    assert not O.mergeable(blk, m("b1", "pool"))          # different types
    assert not O.mergeable(blk, m("b2b", "b3b"))          # different inputs
    sq = O.blocks_of(W.make("squeeze")[0])
    assert O.mergeable(sq[0], 0b110)                       # e1 (1x1 p0) + e3 (3x3 p1)
    # 1x1 pad 1 with 3x3 pad 1 would give different output sizes
    blk2 = O.block_from_edges(2, [])
    blk2.units = [{"kind": "conv", "in": ["x"], "kh": 1, "kw": 1, "sh": 1, "sw": 1, "ph": 1, "pw": 1},
                  {"kind": "conv", "in": ["x"], "kh": 3, "kw": 3, "sh": 1, "sw": 1, "ph": 1, "pw": 1}]
    blk2.src = ["x", "x"]
    assert not O.mergeable(blk2, 0b11)
    blk2.units[0]["ph"] = blk2.units[0]["pw"] = 0
    assert O.mergeable(blk2, 0b11)
    blk2.units[1]["sh"] = 2
    assert not O.mergeable(blk2, 0b11)                     # different stride


def test_config_state_spaces():
    blk = O.blocks_of(W.make("tiny")[0])[0]
    res = O.ios_dp(blk, lambda m, t: 1)
    assert (res.states, res.transitions) == (6, 12)
    assert sum(1 for _ in O.all_schedules(blk)) == 8
    blk = O.blocks_of(W.make("inception")[0])[0]
    res = O.ios_dp(blk, lambda m, t: 1, 3, 8)
    assert (res.states, res.transitions) == (72, 1008)
    sq = O.blocks_of(W.make("squeeze")[0])
    assert [b.n for b in sq] == [3, 3, 3, 1, 3, 3, 3, 3, 1, 3]
    res = O.ios_dp(sq[0], lambda m, t: 1, 3, 8)
    assert (res.states, res.transitions) == (5, 9)
    assert sum(1 for _ in O.all_schedules(sq[0])) == 6


@pytest.mark.slow
def test_inception_schedule_count():
    blk = O.blocks_of(W.make("inception")[0])[0]
    assert sum(1 for _ in O.all_schedules(blk)) == 34516


def test_width_two_ways_and_bound():
    rnd = random.Random(4)
    for _ in range(80):
        n = rnd.randint(1, 9)
        blk = random_dag(n, rnd.random() * 0.6, rnd)
        d = O.width_bruteforce(blk)
        assert d == O.width_dilworth(blk)
        res = O.ios_dp(blk, lambda m, t: 1)
        assert res.transitions <= O.transition_bound(n, d) + 1e-9
    assert O.width_dilworth(O.blocks_of(W.make("inception")[0])[0]) == 4
    assert O.width_dilworth(O.blocks_of(W.make("tiny")[0])[0]) == 2


def test_table1_bound_column():
    g = json.load(open(os.path.join(GOLDEN, "table1_bound.json")))
    for row in g["rows"]:
        v = O.transition_bound(row["n"], row["d"])
        assert float(f"{v:.1e}") == row["bound"], (row, v)
