"""Seeded synthetic workloads standing in for the paper's benchmark blocks.

The paper measures Inception-V3, RandWire, NASNet-A and SqueezeNet (Table 2,
Sec. 5).  No dataset or trained weight is needed for latency or parity, so
each network is replaced by a block of the same shapes built here:

  tiny       2-branch block 1x16x8x8 (used for brute-force schedule checks)
  inception  Inception-V3 mixed block, 192x35x35 -> 256x35x35
  randwire   32-node Watts-Strogatz WS(4, 0.75) DAG of sepconv nodes, 78x28x28
  nasnet     NASNet-A style normal cell, two 168x42x42 inputs -> 840x42x42
  squeeze    8 SqueezeNet fire modules, 96x55x55 input, two max-pools

and, for the block-wise whole-network runs (not one of the blocks above):

  inception_v3   the whole Inception-V3 network, 3x299x299 -> 1000 logits,
                 13 blocks (stem, eleven modules, head)
  squeezenet     the whole SqueezeNet v1.0 network, 3x227x227 -> 1000,
                 12 blocks (conv1 + pool, eight fire modules, two pools, head)
  randwire_net   three RandWire stages (78, 156, 312 channels at 28, 14, 7)
                 joined by strided 1x1 convs, 5 blocks
  nasnet_net     six NASNet-A style normal cells (168 then 336 channels at 42
                 then 21) around a strided conv, 7 blocks

A workload is a plain description (``spec``) plus a dict of float32 numpy
arrays (``tensors``).  The description lists the operators in insertion
order, which is a topological order; both the oracle and the library read it.
Inputs are U(-1, 1); weights are N(0, 2 / fan_in) with
fan_in = (Cin / groups) * kh * kw; biases are zero.

Operator kinds (one schedule unit each, except the two views):
  conv      dense 2-D cross-correlation + bias, optional ReLU before/after
  sepconv   sum of inputs -> ReLU -> depthwise kxk (pad k/2) -> pointwise 1x1
  maxpool / avgpool   kxk window, stride, pad (avg divides by k*k)
  add       elementwise sum of inputs
  mean      elementwise mean of inputs
  concat    channel concatenation (a view: producers write into slices)
  identity  a view of its input
"""
from __future__ import annotations

import copy
from typing import Dict, List, Tuple

import numpy as np

from . import rng

CONFIG_NAMES = ["tiny", "inception", "randwire", "nasnet", "squeeze"]


def _conv(name, inp, cout, k, pad, stride=1, post_relu=1, pre_relu=0, block=-1):
    kh, kw = (k, k) if isinstance(k, int) else k
    ph, pw = (pad, pad) if isinstance(pad, int) else pad
    return {"name": name, "kind": "conv", "in": [inp], "cout": cout,
            "kh": kh, "kw": kw, "sh": stride, "sw": stride, "ph": ph, "pw": pw,
            "pre_relu": pre_relu, "post_relu": post_relu, "block": block}


def _sep(name, inputs, cout, k, block=-1):
    return {"name": name, "kind": "sepconv", "in": list(inputs), "cout": cout,
            "kh": k, "kw": k, "sh": 1, "sw": 1, "ph": k // 2, "pw": k // 2,
            "pre_relu": 1, "post_relu": 0, "block": block}


def _pool(name, inp, kind, k, stride, pad, block=-1):
    return {"name": name, "kind": kind, "in": [inp], "kh": k, "kw": k,
            "sh": stride, "sw": stride, "ph": pad, "pw": pad, "block": block}


def _view(name, kind, inputs):
    return {"name": name, "kind": kind, "in": list(inputs)}


# ---------------------------------------------------------------- graphs

def spec_tiny(batch: int = 1, seed: int = 0) -> dict:
    ops = [
        _conv("A", "x", 16, 1, 0),
        _conv("B1", "x", 8, 1, 0),
        _conv("B2", "B1", 16, 3, 1),
        _view("out", "concat", ["A", "B2"]),
    ]
    return {"name": "tiny", "batch": batch, "seed": seed,
            "inputs": [{"name": "x", "c": 16, "h": 8, "w": 8}],
            "ops": ops, "outputs": ["out"]}


def spec_inception(batch: int = 1, seed: int = 0) -> dict:
    ops = [
        _conv("b1", "x", 64, 1, 0),
        _conv("b2a", "x", 48, 1, 0),
        _conv("b2b", "b2a", 64, 5, 2),
        _conv("b3a", "x", 64, 1, 0),
        _conv("b3b", "b3a", 96, 3, 1),
        _conv("b3c", "b3b", 96, 3, 1),
        _pool("pool", "x", "avgpool", 3, 1, 1),
        _conv("b4", "pool", 32, 1, 0),
        _view("out", "concat", ["b1", "b2b", "b3c", "b4"]),
    ]
    return {"name": "inception", "batch": batch, "seed": seed,
            "inputs": [{"name": "x", "c": 192, "h": 35, "w": 35}],
            "ops": ops, "outputs": ["out"]}


def ws_edges(n: int, k: int, p: float, stream: rng.Stream) -> List[Tuple[int, int]]:
    """Watts-Strogatz small-world graph, edges oriented low -> high index.

    Ring lattice: node i is joined to i+1 .. i+k/2 (mod n).  Then every
    lattice edge (i, i+j), j = 1 .. k/2, is rewired with probability p to
    (i, w), w drawn uniformly among nodes that are neither i nor already
    adjacent to i.
    """
    adj = [set() for _ in range(n)]
    lattice = []
    for j in range(1, k // 2 + 1):
        for i in range(n):
            a, b = i, (i + j) % n
            adj[a].add(b)
            adj[b].add(a)
            lattice.append((a, b))
    for a, b in lattice:
        if stream.u01() < p:
            cand = [w for w in range(n) if w != a and w not in adj[a]]
            if not cand:
                continue
            w = cand[stream.randint(len(cand))]
            adj[a].discard(b)
            adj[b].discard(a)
            adj[a].add(w)
            adj[w].add(a)
    edges = sorted({(min(a, b), max(a, b)) for a in range(n) for b in adj[a]})
    return edges


def _randwire_block(ops, prefix, inp, channels, graph_key, nodes=32, block=-1):
    """A WS(nodes, 4, 0.75) DAG of SEPCONV nodes reading `inp`; returns the
    name of its output (the mean of the sinks) and the graph's edges."""
    stream = rng.Stream(graph_key)
    edges = ws_edges(nodes, 4, 0.75, stream)
    preds = [[] for _ in range(nodes)]
    outdeg = [0] * nodes
    for a, b in edges:
        preds[b].append(a)
        outdeg[a] += 1
    for v in range(nodes):
        ins = [f"{prefix}n{u}" for u in sorted(preds[v])] or [inp]
        ops.append(_sep(f"{prefix}n{v}", ins, channels, 3, block=block))
    sinks = [f"{prefix}n{v}" for v in range(nodes) if outdeg[v] == 0]
    ops.append({"name": f"{prefix}out", "kind": "mean", "in": sinks, "block": block})
    return f"{prefix}out", edges


def spec_randwire(batch: int = 1, seed: int = 0, nodes: int = 32, channels: int = 78,
                  hw: int = 28) -> dict:
    ops = []
    _, edges = _randwire_block(ops, "", "x", channels, rng.key_of("randwire-graph", seed), nodes)
    return {"name": "randwire", "batch": batch, "seed": seed,
            "inputs": [{"name": "x", "c": channels, "h": hw, "w": hw}],
            "ops": ops, "outputs": ["out"], "ws_edges": edges}


RANDWIRE_NET_BLOCKS = ["stage1", "down1", "stage2", "down2", "stage3"]


def spec_randwire_net(batch: int = 1, seed: int = 0, channels: int = 78, hw: int = 28) -> dict:
    """The three random-graph stages of a RandWire network (small regime):
    WS(32, 4, 0.75) DAGs of SEPCONV nodes with C, 2C and 4C channels at 28x28,
    14x14 and 7x7, each drawn from its own seeded stream, joined by 1x1
    stride-2 convs (+ ReLU) that double the channels.  Blocks: each stage and
    each transition."""
    ops = []
    cur = "x"
    for k in range(3):
        c = channels << k
        if k:
            ops.append(_conv(f"down{k}", cur, c, 1, 0, stride=2, block=2 * k - 1))
            cur = f"down{k}"
        cur, _ = _randwire_block(ops, f"s{k + 1}", cur, c, rng.key_of("randwire-net-graph", seed, k),
                                 block=2 * k)
    return {"name": "randwire_net", "batch": batch, "seed": seed,
            "inputs": [{"name": "x", "c": channels, "h": hw, "w": hw}],
            "ops": ops, "outputs": [cur], "block_names": RANDWIRE_NET_BLOCKS}


NASNET_OPS = ["sep3", "sep5", "avgpool", "maxpool", "identity"]


def _nasnet_cell(ops, prefix, h, h_prev, channels, cell_key, block=-1):
    """Five combine blocks, each adding two ops applied to inputs drawn from
    {h, h_prev}, the ops drawn from NASNET_OPS (a separable conv is two
    chained SEPCONV units); the adds are concatenated.  Returns the concat's
    name and the draws."""
    stream = rng.Stream(cell_key)
    outs, choices = [], []
    for b in range(5):
        slot_out = []
        for s in range(2):
            side = stream.randint(2)
            inp = [h, h_prev][side]
            kind = NASNET_OPS[stream.randint(5)]
            choices.append((b, s, ["h", "h_prev"][side], kind))
            nm = f"{prefix}c{b}s{s}"
            if kind in ("sep3", "sep5"):
                k = 3 if kind == "sep3" else 5
                ops.append(_sep(nm + "u1", [inp], channels, k, block=block))
                ops.append(_sep(nm + "u2", [nm + "u1"], channels, k, block=block))
                slot_out.append(nm + "u2")
            elif kind in ("avgpool", "maxpool"):
                ops.append(_pool(nm, inp, kind, 3, 1, 1, block=block))
                slot_out.append(nm)
            else:
                ops.append(_view(nm, "identity", [inp]))
                slot_out.append(nm)
        ops.append({"name": f"{prefix}add{b}", "kind": "add", "in": slot_out, "block": block})
        outs.append(f"{prefix}add{b}")
    ops.append(_view(f"{prefix}out", "concat", outs))
    return f"{prefix}out", choices


def spec_nasnet(batch: int = 1, seed: int = 0, channels: int = 168, hw: int = 42) -> dict:
    ops = []
    _, choices = _nasnet_cell(ops, "", "h", "h_prev", channels, rng.key_of("nasnet-cell", seed))
    return {"name": "nasnet", "batch": batch, "seed": seed,
            "inputs": [{"name": "h", "c": channels, "h": hw, "w": hw},
                       {"name": "h_prev", "c": channels, "h": hw, "w": hw}],
            "ops": ops, "outputs": ["out"], "choices": choices}


NASNET_NET_BLOCKS = ["cell1", "cell2", "cell3", "reduce", "cell4", "cell5", "cell6"]


def spec_nasnet_net(batch: int = 1, seed: int = 0, channels: int = 168, hw: int = 42) -> dict:
    """A NASNet-A style stack: three normal cells with C channels at 42x42,
    a 3x3 stride-2 conv (+ ReLU) to 2C channels at 21x21 in place of the
    reduction cell, three normal cells with 2C channels.  A cell reads the
    two previous cells' outputs (5C or 10C channels) through 1x1 convs to C
    (its "reduce" inputs h and h_prev); the stack's inputs h, h_prev feed the
    first cell, the strided conv's output both inputs of the cell after it.
    Each cell's draws come from its own seeded stream.  Blocks: each cell
    with its two 1x1 convs, and the strided conv."""
    ops = []
    outs = {}
    block = 0

    def cell(k, h_src, hp_src, c):
        nonlocal block
        pre = f"k{k}"
        srcs = []
        for nm, src in (("h", h_src), ("hp", hp_src)):
            if src in ("h", "h_prev"):          # the stack's own inputs: already C channels
                srcs.append(src)
            else:
                ops.append(_conv(f"{pre}{nm}", src, c, 1, 0, block=block))
                srcs.append(f"{pre}{nm}")
        out, _ = _nasnet_cell(ops, pre, srcs[0], srcs[1], c, rng.key_of("nasnet-net-cell", seed, k), block=block)
        outs[k] = out
        block += 1
    cell(1, "h", "h_prev", channels)
    cell(2, outs[1], "h", channels)
    cell(3, outs[2], outs[1], channels)
    ops.append(_conv("reduce", outs[3], 2 * channels, 3, 1, stride=2, block=block))
    block += 1
    cell(4, "reduce", "reduce", 2 * channels)
    cell(5, outs[4], "reduce", 2 * channels)
    cell(6, outs[5], outs[4], 2 * channels)
    return {"name": "nasnet_net", "batch": batch, "seed": seed,
            "inputs": [{"name": "h", "c": channels, "h": hw, "w": hw},
                       {"name": "h_prev", "c": channels, "h": hw, "w": hw}],
            "ops": ops, "outputs": [outs[6]], "block_names": NASNET_NET_BLOCKS}


FIRE = [(16, 64), (16, 64), (32, 128), (32, 128), (48, 192), (48, 192), (64, 256), (64, 256)]


def spec_squeeze(batch: int = 1, seed: int = 0) -> dict:
    ops = []
    cur = "x"
    block = 0
    for m, (s, e) in enumerate(FIRE, start=1):
        ops.append(_conv(f"m{m}sq", cur, s, 1, 0, block=block))
        ops.append(_conv(f"m{m}e1", f"m{m}sq", e, 1, 0, block=block))
        ops.append(_conv(f"m{m}e3", f"m{m}sq", e, 3, 1, block=block))
        ops.append(_view(f"m{m}", "concat", [f"m{m}e1", f"m{m}e3"]))
        cur = f"m{m}"
        block += 1
        if m in (3, 7):
            ops.append(_pool(f"pool{m}", cur, "maxpool", 3, 2, 0, block=block))
            cur = f"pool{m}"
            block += 1
    return {"name": "squeeze", "batch": batch, "seed": seed,
            "inputs": [{"name": "x", "c": 96, "h": 55, "w": 55}],
            "ops": ops, "outputs": [cur]}


# ---------------------------------------------------------------- whole networks
#
# Inception-V3 (Szegedy et al., "Rethinking the Inception Architecture",
# 299x299 input, no auxiliary head, no batch-norm: each conv carries a bias
# and a ReLU) built from its published layer table: a stem of five convs and
# two max-pools, three 35x35 modules, a grid reduction to 17x17, four 17x17
# modules with factorised 7x7 convs, a reduction to 8x8, two 8x8 modules with
# split 1x3 / 3x1 outputs, global average pooling and the 1000-way classifier
# (a 1x1 conv on the 1x1 map, no ReLU).  The eleven modules are the blocks the
# paper schedules one at a time (Table 2, block-wise speed-up appendix); the
# stem and the head are blocks of their own.


def _inception_a(ops, p, inp, pool_features, block):
    ops += [_conv(f"{p}_1x1", inp, 64, 1, 0, block=block),
            _conv(f"{p}_5x5a", inp, 48, 1, 0, block=block),
            _conv(f"{p}_5x5b", f"{p}_5x5a", 64, 5, 2, block=block),
            _conv(f"{p}_3x3a", inp, 64, 1, 0, block=block),
            _conv(f"{p}_3x3b", f"{p}_3x3a", 96, 3, 1, block=block),
            _conv(f"{p}_3x3c", f"{p}_3x3b", 96, 3, 1, block=block),
            _pool(f"{p}_pool", inp, "avgpool", 3, 1, 1, block=block),
            _conv(f"{p}_pp", f"{p}_pool", pool_features, 1, 0, block=block),
            _view(p, "concat", [f"{p}_1x1", f"{p}_5x5b", f"{p}_3x3c", f"{p}_pp"])]


def _inception_b(ops, p, inp, block):
    # 35x35 -> 17x17 grid reduction
    ops += [_conv(f"{p}_3x3", inp, 384, 3, 0, stride=2, block=block),
            _conv(f"{p}_dbla", inp, 64, 1, 0, block=block),
            _conv(f"{p}_dblb", f"{p}_dbla", 96, 3, 1, block=block),
            _conv(f"{p}_dblc", f"{p}_dblb", 96, 3, 0, stride=2, block=block),
            _pool(f"{p}_pool", inp, "maxpool", 3, 2, 0, block=block),
            _view(p, "concat", [f"{p}_3x3", f"{p}_dblc", f"{p}_pool"])]


def _inception_c(ops, p, inp, c7, block):
    # 17x17 module, 7x7 convs factorised into 1x7 and 7x1
    r, c = ((1, 7), (0, 3)), ((7, 1), (3, 0))
    ops += [_conv(f"{p}_1x1", inp, 192, 1, 0, block=block),
            _conv(f"{p}_7a", inp, c7, 1, 0, block=block),
            _conv(f"{p}_7b", f"{p}_7a", c7, *r, block=block),
            _conv(f"{p}_7c", f"{p}_7b", 192, *c, block=block),
            _conv(f"{p}_d7a", inp, c7, 1, 0, block=block),
            _conv(f"{p}_d7b", f"{p}_d7a", c7, *c, block=block),
            _conv(f"{p}_d7c", f"{p}_d7b", c7, *r, block=block),
            _conv(f"{p}_d7d", f"{p}_d7c", c7, *c, block=block),
            _conv(f"{p}_d7e", f"{p}_d7d", 192, *r, block=block),
            _pool(f"{p}_pool", inp, "avgpool", 3, 1, 1, block=block),
            _conv(f"{p}_pp", f"{p}_pool", 192, 1, 0, block=block),
            _view(p, "concat", [f"{p}_1x1", f"{p}_7c", f"{p}_d7e", f"{p}_pp"])]


def _inception_d(ops, p, inp, block):
    # 17x17 -> 8x8 grid reduction
    ops += [_conv(f"{p}_3a", inp, 192, 1, 0, block=block),
            _conv(f"{p}_3b", f"{p}_3a", 320, 3, 0, stride=2, block=block),
            _conv(f"{p}_7a", inp, 192, 1, 0, block=block),
            _conv(f"{p}_7b", f"{p}_7a", 192, (1, 7), (0, 3), block=block),
            _conv(f"{p}_7c", f"{p}_7b", 192, (7, 1), (3, 0), block=block),
            _conv(f"{p}_7d", f"{p}_7c", 192, 3, 0, stride=2, block=block),
            _pool(f"{p}_pool", inp, "maxpool", 3, 2, 0, block=block),
            _view(p, "concat", [f"{p}_3b", f"{p}_7d", f"{p}_pool"])]


def _inception_e(ops, p, inp, block):
    # 8x8 module whose 3x3 branches end in parallel 1x3 and 3x1 convs
    r, c = ((1, 3), (0, 1)), ((3, 1), (1, 0))
    ops += [_conv(f"{p}_1x1", inp, 320, 1, 0, block=block),
            _conv(f"{p}_3a", inp, 384, 1, 0, block=block),
            _conv(f"{p}_3b1", f"{p}_3a", 384, *r, block=block),
            _conv(f"{p}_3b2", f"{p}_3a", 384, *c, block=block),
            _view(f"{p}_3", "concat", [f"{p}_3b1", f"{p}_3b2"]),
            _conv(f"{p}_d3a", inp, 448, 1, 0, block=block),
            _conv(f"{p}_d3b", f"{p}_d3a", 384, 3, 1, block=block),
            _conv(f"{p}_d3c1", f"{p}_d3b", 384, *r, block=block),
            _conv(f"{p}_d3c2", f"{p}_d3b", 384, *c, block=block),
            _view(f"{p}_d3", "concat", [f"{p}_d3c1", f"{p}_d3c2"]),
            _pool(f"{p}_pool", inp, "avgpool", 3, 1, 1, block=block),
            _conv(f"{p}_pp", f"{p}_pool", 192, 1, 0, block=block),
            _view(p, "concat", [f"{p}_1x1", f"{p}_3", f"{p}_d3", f"{p}_pp"])]


def spec_inception_7c(batch: int = 1, seed: int = 0) -> dict:
    """Inception-V3's last module (7c, an 8x8 module whose 3x3 branches end
    in parallel 1x3 and 3x1 convs) as a block of its own, 2048x8x8 ->
    2048x8x8: the block whose schedule the paper shows changing with the
    batch size (merging a 1x3 / 3x1 pair into one 3x3 conv pays at large
    batch)."""
    ops = []
    _inception_e(ops, "7c", "x", -1)
    return {"name": "inception_7c", "batch": batch, "seed": seed,
            "inputs": [{"name": "x", "c": 2048, "h": 8, "w": 8}], "ops": ops, "outputs": ["7c"]}


INCEPTION_V3_BLOCKS = ["stem", "5b", "5c", "5d", "6a", "6b", "6c", "6d", "6e", "7a", "7b", "7c", "head"]


def spec_inception_v3(batch: int = 1, seed: int = 0) -> dict:
    ops = [_conv("stem_1a", "x", 32, 3, 0, stride=2, block=0),
           _conv("stem_2a", "stem_1a", 32, 3, 0, block=0),
           _conv("stem_2b", "stem_2a", 64, 3, 1, block=0),
           _pool("stem_p1", "stem_2b", "maxpool", 3, 2, 0, block=0),
           _conv("stem_3b", "stem_p1", 80, 1, 0, block=0),
           _conv("stem_4a", "stem_3b", 192, 3, 0, block=0),
           _pool("stem_p2", "stem_4a", "maxpool", 3, 2, 0, block=0)]
    cur = "stem_p2"
    for b, (p, pf) in enumerate([("5b", 32), ("5c", 64), ("5d", 64)], start=1):
        _inception_a(ops, p, cur, pf, b)
        cur = p
    _inception_b(ops, "6a", cur, 4)
    cur = "6a"
    for b, (p, c7) in enumerate([("6b", 128), ("6c", 160), ("6d", 160), ("6e", 192)], start=5):
        _inception_c(ops, p, cur, c7, b)
        cur = p
    _inception_d(ops, "7a", cur, 9)
    cur = "7a"
    for b, p in enumerate(["7b", "7c"], start=10):
        _inception_e(ops, p, cur, b)
        cur = p
    ops += [_pool("head_pool", cur, "avgpool", 8, 1, 0, block=12),
            _conv("head_fc", "head_pool", 1000, 1, 0, post_relu=0, block=12)]
    return {"name": "inception_v3", "batch": batch, "seed": seed,
            "inputs": [{"name": "x", "c": 3, "h": 299, "w": 299}],
            "ops": ops, "outputs": ["head_fc"], "block_names": INCEPTION_V3_BLOCKS}


def spec_squeezenet(batch: int = 1, seed: int = 0) -> dict:
    """SqueezeNet v1.0 (Iandola et al.) from its published layer table, 227x227
    input: conv1 7x7/2 (96), max-pool 3x3/2, fire2..fire9 with max-pools
    3x3/2 after fire4 and fire8 (the fire modules of the stack above), conv10
    1x1 (1000) with ReLU, global 13x13 average pooling.  Blocks: conv1 and
    its pool, each fire module, each later pool, conv10 and the global pool."""
    ops = [_conv("conv1", "x", 96, 7, 0, stride=2, block=0),
           _pool("pool1", "conv1", "maxpool", 3, 2, 0, block=0)]
    cur, block = "pool1", 1
    for m, (s, e) in enumerate(FIRE, start=2):
        ops.append(_conv(f"f{m}sq", cur, s, 1, 0, block=block))
        ops.append(_conv(f"f{m}e1", f"f{m}sq", e, 1, 0, block=block))
        ops.append(_conv(f"f{m}e3", f"f{m}sq", e, 3, 1, block=block))
        ops.append(_view(f"f{m}", "concat", [f"f{m}e1", f"f{m}e3"]))
        cur = f"f{m}"
        block += 1
        if m in (4, 8):
            ops.append(_pool(f"pool{m}", cur, "maxpool", 3, 2, 0, block=block))
            cur = f"pool{m}"
            block += 1
    ops += [_conv("conv10", cur, 1000, 1, 0, block=block),
            _pool("gpool", "conv10", "avgpool", 13, 1, 0, block=block)]
    names = ["conv1", "fire2", "fire3", "fire4", "pool4", "fire5", "fire6", "fire7", "fire8", "pool8",
             "fire9", "head"]
    return {"name": "squeezenet", "batch": batch, "seed": seed,
            "inputs": [{"name": "x", "c": 3, "h": 227, "w": 227}],
            "ops": ops, "outputs": ["gpool"], "block_names": names}


NETWORK_NAMES = ["inception_v3", "squeezenet", "randwire_net", "nasnet_net"]

SPECS = {"tiny": spec_tiny, "inception": spec_inception, "randwire": spec_randwire,
         "nasnet": spec_nasnet, "squeeze": spec_squeeze, "inception_v3": spec_inception_v3,
         "squeezenet": spec_squeezenet, "randwire_net": spec_randwire_net, "nasnet_net": spec_nasnet_net,
         "inception_7c": spec_inception_7c}


# ---------------------------------------------------------------- shapes

def infer_shapes(spec: dict) -> Dict[str, Tuple[int, int, int]]:
    """(C, H, W) of every named tensor (batch excluded)."""
    shp = {t["name"]: (t["c"], t["h"], t["w"]) for t in spec["inputs"]}
    for op in spec["ops"]:
        ins = [shp[i] for i in op["in"]]
        k = op["kind"]
        c, h, w = ins[0]
        if k in ("conv", "sepconv", "maxpool", "avgpool"):
            ho = (h + 2 * op["ph"] - op["kh"]) // op["sh"] + 1
            wo = (w + 2 * op["pw"] - op["kw"]) // op["sw"] + 1
            co = op["cout"] if k in ("conv", "sepconv") else c
            shp[op["name"]] = (co, ho, wo)
        elif k == "concat":
            shp[op["name"]] = (sum(s[0] for s in ins), h, w)
        else:
            shp[op["name"]] = (c, h, w)
    return shp


def param_shapes(spec: dict) -> List[Tuple[str, tuple, int]]:
    """(tensor name, shape, fan_in) of every weight / bias, in a fixed order."""
    shp = infer_shapes(spec)
    out = []
    for op in spec["ops"]:
        cin = shp[op["in"][0]][0]
        if op["kind"] == "conv":
            out.append((op["name"] + ".w", (op["cout"], cin, op["kh"], op["kw"]),
                        cin * op["kh"] * op["kw"]))
            out.append((op["name"] + ".b", (op["cout"],), 0))
        elif op["kind"] == "sepconv":
            out.append((op["name"] + ".dw", (cin, 1, op["kh"], op["kw"]), op["kh"] * op["kw"]))
            out.append((op["name"] + ".pw", (op["cout"], cin, 1, 1), cin))
            out.append((op["name"] + ".b", (op["cout"],), 0))
    return out


def make_tensors(spec: dict, seed: int | None = None) -> Dict[str, np.ndarray]:
    """Seeded inputs U(-1,1), weights N(0, 2/fan_in), zero biases (float32)."""
    seed = spec.get("seed", 0) if seed is None else seed
    name = spec["name"]
    n = spec["batch"]
    tensors = {}
    idx = 0
    for t in spec["inputs"]:
        # inputs are keyed per image so that batch b's first image equals batch 1's
        imgs = [rng.uniform_pm1(rng.key_of(name, seed, "input", idx, i), (t["c"], t["h"], t["w"]))
                for i in range(n)]
        tensors[t["name"]] = np.stack(imgs, 0)
        idx += 1
    for pname, shape, fan_in in param_shapes(spec):
        if pname.endswith(".b"):
            tensors[pname] = np.zeros(shape, dtype=np.float32)
        else:
            tensors[pname] = rng.normal(rng.key_of(name, seed, "param", pname), shape,
                                        float(np.sqrt(2.0 / fan_in)))
    return tensors


def make(config: str, batch: int = 1, seed: int = 0):
    """(spec, tensors) for one of CONFIG_NAMES."""
    spec = SPECS[config](batch=batch, seed=seed)
    return spec, make_tensors(spec, seed)


def unit_ops(spec: dict) -> List[dict]:
    """Operators that are schedule units (views excluded), in insertion order."""
    return [op for op in spec["ops"] if op["kind"] not in ("concat", "identity")]


def with_batch(spec: dict, batch: int) -> dict:
    s = copy.deepcopy(spec)
    s["batch"] = batch
    return s
