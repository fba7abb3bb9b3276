"""Whole-network workloads (Inception-V3, SqueezeNet, the RandWire and NASNet
stacks; scheduled block by block): the descriptions against the networks'
published layer tables or their construction, and the oracle's block split
and state spaces against closed forms.  No GPU."""
import math

import numpy as np

from oracle import evaluator as E
from oracle import schedule as O
import workloads as W


def spec():
    return W.SPECS["inception_v3"]()


def test_inception_v3_layer_table():
    """Grid sizes and depths at the module boundaries of the published
    Inception-V3 layer table: 299x299x3 in, 35x35 after the stem, 35x35x288
    after the three 35x35 modules, 17x17x768 after the reduction and after
    each 17x17 module, 8x8x1280 after the second reduction, 8x8x2048 after the
    8x8 modules, 1x1x2048 after pooling, 1000 logits."""
    s = spec()
    shp = W.infer_shapes(s)
    assert (s["inputs"][0]["c"], s["inputs"][0]["h"], s["inputs"][0]["w"]) == (3, 299, 299)
    assert shp["stem_1a"] == (32, 149, 149)
    assert shp["stem_2b"] == (64, 147, 147)
    assert shp["stem_p1"] == (64, 73, 73)
    assert shp["stem_p2"] == (192, 35, 35)
    assert shp["5b"] == (256, 35, 35)
    assert shp["5c"] == shp["5d"] == (288, 35, 35)
    for p in ("6a", "6b", "6c", "6d", "6e"):
        assert shp[p] == (768, 17, 17)
    assert shp["7a"] == (1280, 8, 8)
    assert shp["7b"] == shp["7c"] == (2048, 8, 8)
    assert shp["head_pool"] == (2048, 1, 1)
    assert shp["head_fc"] == (1000, 1, 1)
    # every conv keeps its grid except the stride-2 and unpadded ones
    for op in W.unit_ops(s):
        if op["kind"] == "conv" and op["sh"] == 1 and op["kh"] == 2 * op["ph"] + 1 \
                and op["kw"] == 2 * op["pw"] + 1:
            assert shp[op["name"]][1:] == shp[op["in"][0]][1:]


def test_inception_v3_blocks():
    """Eleven modules (the blocks the paper counts) plus the stem and the
    classifier head; every block within the 64-unit limit."""
    s = spec()
    blocks = O.blocks_of(s)
    assert len(blocks) == 13
    assert [b.n for b in blocks] == [7, 8, 8, 8, 5, 11, 11, 11, 11, 7, 10, 10, 2]
    assert [blocks[i].units[0]["name"].split("_")[0] for i in range(13)] == \
        ["stem"] + W.SPECS["inception_v3"]()["block_names"][1:-1] + ["head"]


def _down_sets(blk):
    """Number of down-sets of a block by brute force over every subset."""
    return sum(1 for S in range(1 << blk.n)
               if all(not (S >> v & 1) or (blk.pred[v] & ~S) == 0 for v in range(blk.n)))


def test_inception_v3_state_spaces():
    """The DP's states are the block's down-sets (Sec. 4.2).  A module whose
    branches share only the block input is a disjoint union of its branches,
    so its down-sets multiply: a chain of l units has l + 1, a unit feeding
    two leaves 5, a chain of two feeding two leaves 6.  With unit costs the
    DP visits exactly that many states under pruning r = 3, s = 8 (every
    single unit is a valid ending, so every down-set stays reachable)."""
    blocks = O.blocks_of(spec())
    chains = {0: [7], 1: [1, 2, 3, 2], 4: [1, 3, 1], 5: [1, 3, 5, 2], 9: [2, 4, 1], 12: [2]}
    expect = {b: math.prod(l + 1 for l in ls) for b, ls in chains.items()}
    expect[10] = 2 * 5 * 6 * 3                      # 1x1; 1x1 -> (1x3, 3x1); 1x1 -> 3x3 -> (1x3, 3x1); pool -> 1x1
    for b, n in expect.items():
        assert _down_sets(blocks[b]) == n
        res = O.ios_dp(blocks[b], lambda m, t: 1, 3, 8)
        assert res.states == n
    assert expect[1] == 72                          # the Inception block of the single-block runs
    assert _down_sets(blocks[2]) == _down_sets(blocks[1])
    assert all(_down_sets(blocks[b]) == 144 for b in (5, 6, 7, 8))


def test_inception_v3_merge_pairs():
    """Operator merge (Sec. 3, merge rule: same type, same input, same
    stride, smaller kernels zero-padded to the largest): the 1x3 / 3x1 pair
    of an 8x8 module merges into one 3x3 conv (pads (0,1) and (1,0) become
    (1,1)), the 1x1 convs reading a module's input merge, a stride-2 conv does
    not merge with a stride-1 one."""
    blocks = O.blocks_of(spec())
    for b in (10, 11):
        blk = blocks[b]
        names = [u["name"] for u in blk.units]
        m = lambda *ns: sum(1 << names.index(blk.units[0]["name"].split("_")[0] + "_" + x) for x in ns)
        assert O.mergeable(blk, m("3b1", "3b2"))
        assert O.mergeable(blk, m("d3c1", "d3c2"))
        assert O.mergeable(blk, m("1x1", "3a", "d3a"))
        assert not O.mergeable(blk, m("3b1", "d3c2"))          # different inputs
    blk = blocks[4]
    names = [u["name"] for u in blk.units]
    assert not O.mergeable(blk, (1 << names.index("6a_3x3")) | (1 << names.index("6a_dbla")))
    blk = blocks[5]
    names = [u["name"] for u in blk.units]
    assert O.mergeable(blk, sum(1 << names.index(n) for n in ("6b_1x1", "6b_7a", "6b_d7a")))


def test_inception_v3_dp_not_worse_than_baselines():
    """Under one additive cost table (a fixed launch cost plus a per-unit
    cost, merge cheaper than concurrent), the DP's total on every block is at
    most that of one unit per stage and of the widest single stage."""
    blocks = O.blocks_of(spec())
    for blk in blocks:
        cost = lambda m, t: 5 + 3 * bin(m).count("1") - (1 if t == O.MERGE else 0)
        res = O.ios_dp(blk, cost, 3, 8)
        seq = sum(min(cost(1 << v, O.CONCURRENT), cost(1 << v, O.MERGE) if O.mergeable(blk, 1 << v)
                      else 10 ** 9) for v in range(blk.n))
        assert res.cost <= seq
        assert res.cost <= 5 * blk.n + 3 * blk.n


def test_squeezenet_layer_table():
    """SqueezeNet v1.0's published layer table at 227x227: conv1 111x111x96,
    max-pool 55x55x96, fire2..4 at 55x55 (128, 128, 256), max-pool 27x27,
    fire5..8 at 27x27 (256, 384, 384, 512), max-pool 13x13, fire9 512,
    conv10 13x13x1000, global pool 1x1x1000; every fire module a 3-unit block
    whose two expand convs read the squeeze output and can merge."""
    s = W.SPECS["squeezenet"]()
    shp = W.infer_shapes(s)
    assert shp["conv1"] == (96, 111, 111) and shp["pool1"] == (96, 55, 55)
    assert [shp[f"f{m}"] for m in (2, 3, 4)] == [(128, 55, 55), (128, 55, 55), (256, 55, 55)]
    assert shp["pool4"] == (256, 27, 27)
    assert [shp[f"f{m}"][0] for m in (5, 6, 7, 8)] == [256, 384, 384, 512]
    assert shp["pool8"] == (512, 13, 13) and shp["f9"] == (512, 13, 13)
    assert shp["conv10"] == (1000, 13, 13) and shp["gpool"] == (1000, 1, 1)
    blocks = O.blocks_of(s)
    assert [b.n for b in blocks] == [2, 3, 3, 3, 1, 3, 3, 3, 3, 1, 3, 2]
    assert len(s["block_names"]) == len(blocks)
    for b in blocks:
        if b.n == 3:
            assert O.mergeable(b, 0b110)
            assert O.ios_dp(b, lambda m, t: 1, 3, 8).states == 5    # a squeeze unit feeding two


def test_randwire_net_layout():
    """Three WS(32, 4, 0.75) stages of SEPCONV nodes with 78, 156 and 312
    channels at 28x28, 14x14 and 7x7, each ending in the mean of its sinks,
    joined by 1x1 stride-2 convs; five blocks (stage, transition, ...), each
    stage's graph drawn from its own stream; the whole network evaluates in
    the oracle to the last stage's mean."""
    s, ten = W.make("randwire_net")
    shp = W.infer_shapes(s)
    assert [shp[f"s{k}out"] for k in (1, 2, 3)] == [(78, 28, 28), (156, 14, 14), (312, 7, 7)]
    assert shp["down1"] == (156, 14, 14) and shp["down2"] == (312, 7, 7)
    blocks = O.blocks_of(s)
    assert [b.n for b in blocks] == [33, 1, 33, 1, 33]
    assert len(s["block_names"]) == len(blocks)
    edges = [sorted((a, b) for a in range(32) for b in range(32) if blk.succ[a] >> b & 1)
             for blk in (blocks[0], blocks[2], blocks[4])]
    assert edges[0] != edges[1] != edges[2]
    for e in edges:
        assert len(e) >= 64                      # 2n = 64 WS edges among the nodes, plus edges to the mean
    out = E.outputs(s, ten)[0]
    assert out.shape == (1, 312, 7, 7) and np.isfinite(out).all()


def test_nasnet_net_layout():
    """Six normal cells (168 channels at 42x42, then 336 at 21x21) around a
    3x3 stride-2 conv; each cell's inputs pass through 1x1 convs to the cell
    width (the first cell reads the stack's inputs directly); concat widths
    5C; seven blocks; each cell drawn from its own stream."""
    s, ten = W.make("nasnet_net")
    shp = W.infer_shapes(s)
    assert [shp[f"k{k}out"] for k in range(1, 7)] == [(840, 42, 42)] * 3 + [(1680, 21, 21)] * 3
    assert shp["reduce"] == (336, 21, 21)
    assert "k1h" not in shp and shp["k2h"] == (168, 42, 42) and shp["k6hp"] == (336, 21, 21)
    blocks = O.blocks_of(s)
    assert len(blocks) == 7 and blocks[3].n == 1
    assert len(s["block_names"]) == len(blocks)
    kinds = [[u["kind"] for u in b.units] for b in blocks]
    assert len({tuple(k) for k in kinds}) > 2                   # cells differ
    out = E.outputs(W.with_batch(s, 1), ten)[0]
    assert out.shape == (1, 1680, 21, 21) and np.isfinite(out).all()
