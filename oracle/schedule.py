"""Oracle for the IOS schedule search (TEST INFRASTRUCTURE ONLY).

Follows the paper's Algorithm 1 (Sec. 4.1) in its own order and notation:

* an *ending* S' of S is a non-empty subset of S such that no edge leaves S'
  for S - S' (Sec. 4.1, Fig. 4);
* the pruning strategy P(S, S') holds iff S' has at most ``s`` groups and
  each group has at most ``r`` operators (Sec. 4.3), where the groups of a
  stage are the connected components of S' (operators joined by an edge share
  a group, Sec. 3 "Parallelization Strategy");
* GenerateStage takes the concurrent latency, the merge latency if the stage
  can be merged (else infinity) and keeps concurrent only if it is strictly
  faster;
* Scheduler(S) is the memoised recurrence
  cost[S] = min over endings S' of cost[S - S'] + stage_latency[S'],
  cost[{}] = 0, keeping the first minimum found;
* InterOperatorScheduler rebuilds Q from choice[] back to front.

Readings where the paper is silent (each also listed in the design notes):
* endings are visited in ascending bit-mask order, so a strict ``<`` keeps
  the smallest mask among equal-cost endings;
* bit i of a block mask is the i-th schedule unit of the block in insertion
  order;
* a stage is mergeable iff all its units are dense convs reading the same
  tensor, with equal stride and ReLU flags, at least two of them, and each
  kernel can be centred in the largest one with equal resulting padding.

``brute_force`` enumerates every ordered partition of a block into stages,
each an ending of what remains, and picks the minimum by plain comparison.
"""
from __future__ import annotations

import itertools
import math
from typing import Callable, Dict, List, Optional, Sequence, Tuple

INF = float("inf")
CONCURRENT, MERGE = 0, 1
VIEW_KINDS = ("concat", "identity")


# ------------------------------------------------------------ graph model

class Block:
    """One block of schedule units with edges restricted to the block."""

    def __init__(self, units: List[dict], succ: List[int], global_ids: List[int],
                 src: List[str]):
        self.units = units          # op dicts, local order
        self.n = len(units)
        self.succ = succ            # local successor bitmasks
        self.pred = [0] * self.n
        for u in range(self.n):
            for v in range(self.n):
                if succ[u] >> v & 1:
                    self.pred[v] |= 1 << u
        self.global_ids = global_ids
        self.src = src              # resolved input tensor name per unit (first input)

    @property
    def full(self) -> int:
        return (1 << self.n) - 1


def _resolve(name: str, views: Dict[str, dict]) -> str:
    while name in views and views[name]["kind"] == "identity":
        name = views[name]["in"][0]
    return name


def producers(name: str, views: Dict[str, dict], unit_index: Dict[str, int]) -> List[int]:
    if name in unit_index:
        return [unit_index[name]]
    if name in views:
        out = []
        for i in views[name]["in"]:
            out += producers(i, views, unit_index)
        return out
    return []   # a graph input


def blocks_of(spec: dict) -> List[Block]:
    """Split the schedule units into blocks (explicit ids, else one block)."""
    units = [op for op in spec["ops"] if op["kind"] not in VIEW_KINDS]
    views = {op["name"]: op for op in spec["ops"] if op["kind"] in VIEW_KINDS}
    uidx = {op["name"]: i for i, op in enumerate(units)}
    succ_g = [set() for _ in units]
    for v, op in enumerate(units):
        for nm in op["in"]:
            for u in producers(nm, views, uidx):
                succ_g[u].add(v)
    ids = [op.get("block", -1) for op in units]
    if all(b < 0 for b in ids):
        groups = [list(range(len(units)))]
    else:
        assert all(b >= 0 for b in ids), "either every unit names a block or none does"
        groups = [[i for i in range(len(units)) if ids[i] == b] for b in sorted(set(ids))]
    out = []
    for g in groups:
        loc = {gid: i for i, gid in enumerate(g)}
        succ = [0] * len(g)
        for i, gid in enumerate(g):
            for w in succ_g[gid]:
                if w in loc:
                    succ[i] |= 1 << loc[w]
        src = [_resolve(units[gid]["in"][0], views) for gid in g]
        out.append(Block([units[gid] for gid in g], succ, g, src))
    return out


def block_from_edges(n: int, edges: Sequence[Tuple[int, int]]) -> Block:
    """A bare block of n abstract units (all kind 'op') with the given edges."""
    succ = [0] * n
    for a, b in edges:
        assert a < b, "edges must go from lower to higher index"
        succ[a] |= 1 << b
    units = [{"name": f"u{i}", "kind": "op", "in": []} for i in range(n)]
    return Block(units, succ, list(range(n)), [f"u{i}" for i in range(n)])


# ------------------------------------------------------------ definitions

def bits(m: int) -> List[int]:
    return [i for i in range(m.bit_length()) if m >> i & 1]


def is_ending(blk: Block, S: int, Sp: int) -> bool:
    """S' (non-empty, inside S) is an ending of S iff no edge goes S' -> S-S'."""
    if Sp == 0 or Sp & ~S:
        return False
    rest = S & ~Sp
    return all(blk.succ[u] & rest == 0 for u in bits(Sp))


def groups(blk: Block, Sp: int) -> List[int]:
    """Connected components of S' (edges taken undirected), ordered by their
    lowest unit."""
    left = Sp
    comps = []
    while left:
        seed = left & -left
        comp, frontier = seed, seed
        while frontier:
            nxt = 0
            for u in bits(frontier):
                nxt |= (blk.succ[u] | blk.pred[u]) & Sp
            frontier = nxt & ~comp
            comp |= nxt
        comps.append(comp)
        left &= ~comp
    return comps


def prune_ok(blk: Block, Sp: int, r: Optional[int], s: Optional[int]) -> bool:
    """P(S, S'): at most s groups, each of at most r units (None = no limit)."""
    g = groups(blk, Sp)
    if s is not None and len(g) > s:
        return False
    if r is not None and any(bin(c).count("1") > r for c in g):
        return False
    return True


def endings_plain(blk: Block, S: int, r=None, s=None) -> List[int]:
    """Every ending of S satisfying P, by testing every non-empty subset."""
    out = []
    sub = S
    while sub:
        if is_ending(blk, S, sub) and prune_ok(blk, sub, r, s):
            out.append(sub)
        sub = (sub - 1) & S
    return sorted(out)


def endings(blk: Block, S: int, r=None, s=None) -> List[int]:
    """Same set as ``endings_plain``, built by deciding units from the last
    to the first: a unit may join S' only when all its successors inside S
    already have.  A group larger than r can only grow, so such branches
    stop early."""
    order = sorted(bits(S), reverse=True)
    out = []

    def comp_size(cur: int, u: int) -> int:
        comp, frontier = 1 << u, 1 << u
        while frontier:
            nxt = 0
            for x in bits(frontier):
                nxt |= (blk.succ[x] | blk.pred[x]) & cur
            frontier = nxt & ~comp
            comp |= nxt
        return bin(comp).count("1")

    def rec(i: int, cur: int):
        if i == len(order):
            if cur and (s is None or len(groups(blk, cur)) <= s):
                out.append(cur)
            return
        u = order[i]
        rec(i + 1, cur)
        if blk.succ[u] & S & ~cur == 0:
            nxt = cur | 1 << u
            if r is None or comp_size(nxt, u) <= r:
                rec(i + 1, nxt)

    rec(0, 0)
    return sorted(out)


def mergeable(blk: Block, Sp: int) -> bool:
    """Operator-merge eligibility (Sec. 3): same operator type (dense conv),
    same input, same stride, kernels that centre in the largest one with the
    same resulting padding; at least two units."""
    us = bits(Sp)
    if len(us) < 2:
        return False
    ops = [blk.units[u] for u in us]
    if any(op["kind"] != "conv" or len(op["in"]) != 1 for op in ops):
        return False
    if len({blk.src[u] for u in us}) != 1:
        return False
    if len({(op["sh"], op["sw"], op.get("pre_relu", 0), op.get("post_relu", 0)) for op in ops}) != 1:
        return False
    KH = max(op["kh"] for op in ops)
    KW = max(op["kw"] for op in ops)
    pads = set()
    for op in ops:
        if (KH - op["kh"]) % 2 or (KW - op["kw"]) % 2:
            return False
        pads.add((op["ph"] + (KH - op["kh"]) // 2, op["pw"] + (KW - op["kw"]) // 2))
    return len(pads) == 1


# ------------------------------------------------------------ Algorithm 1

CostFn = Callable[[int, int], Optional[float]]   # (S' mask, strategy) -> latency


def generate_stage(blk: Block, Sp: int, cost: CostFn, strategies=(CONCURRENT, MERGE)):
    """GenerateStage: (latency, strategy) of the better of the two.

    With concurrent execution switched off (the IOS-Merge variant of Sec. 6.1)
    a one-unit stage still runs, as the unit alone."""
    single = Sp & (Sp - 1) == 0
    l_conc = cost(Sp, CONCURRENT) if (CONCURRENT in strategies or single) else INF
    if MERGE in strategies and mergeable(blk, Sp):
        l_merge = cost(Sp, MERGE)
    else:
        l_merge = INF
    if l_conc < l_merge:
        return l_conc, CONCURRENT
    return l_merge, MERGE


class DPResult:
    def __init__(self, cost, schedule, states, transitions, stages_seen):
        self.cost = cost
        self.schedule = schedule          # [(S' mask, strategy)] first -> last
        self.states = states
        self.transitions = transitions
        self.stages_seen = stages_seen    # distinct S' passed to GenerateStage


def ios_dp(blk: Block, cost: CostFn, r=None, s=None, strategies=(CONCURRENT, MERGE),
           enum=endings) -> DPResult:
    """InterOperatorScheduler + Scheduler of Algorithm 1 on one block."""
    best: Dict[int, float] = {0: 0}
    choice: Dict[int, Tuple[int, int]] = {}
    stage_cache: Dict[int, Tuple[float, int]] = {}
    visited = {0}
    counter = [0]

    def stage(Sp):
        if Sp not in stage_cache:
            stage_cache[Sp] = generate_stage(blk, Sp, cost, strategies)
        return stage_cache[Sp]

    def scheduler(S: int) -> float:
        visited.add(S)
        if S in best:
            return best[S]
        c_best = INF
        for Sp in enum(blk, S, r, s):
            counter[0] += 1
            l_sp, t_sp = stage(Sp)
            l_s = scheduler(S & ~Sp) + l_sp
            if l_s < c_best:
                c_best = l_s
                choice[S] = (Sp, t_sp)
        best[S] = c_best
        return c_best

    import sys
    old = sys.getrecursionlimit()
    sys.setrecursionlimit(max(old, 10000))
    total = scheduler(blk.full)
    sys.setrecursionlimit(old)
    q = []
    S = blk.full
    while S:
        if S not in choice:
            return DPResult(INF, None, len(visited), counter[0], len(stage_cache))
        Sp, t = choice[S]
        q.insert(0, (Sp, t))
        S &= ~Sp
    return DPResult(total, q, len(visited), counter[0], len(stage_cache))


def all_schedules(blk: Block, r=None, s=None, S: Optional[int] = None):
    """Every schedule of S (default: the whole block) as a list of stage
    masks, first stage first: the last stage is an ending of S satisfying P
    and the rest is a schedule of what remains."""
    S = blk.full if S is None else S
    if S == 0:
        yield []
        return
    for Sp in endings_plain(blk, S, r, s):
        for rest in all_schedules(blk, r, s, S & ~Sp):
            yield rest + [Sp]


def brute_force(blk: Block, cost: CostFn, r=None, s=None, strategies=(CONCURRENT, MERGE)):
    """(min total latency, its schedule [(mask, strategy)], #schedules).

    Among schedules of equal total, the one whose stage masks read from the
    last stage backwards is lexicographically smallest wins."""
    best_key, best_q, count = None, None, 0
    for sched in all_schedules(blk, r, s):
        count += 1
        stages = [(Sp,) + tuple(reversed(generate_stage(blk, Sp, cost, strategies))) for Sp in sched]
        total = sum(l for _, _, l in stages)
        key = (total, [m for m, _, _ in reversed(stages)])
        if best_key is None or key < best_key:
            best_key, best_q = key, [(m, t) for m, t, _ in stages]
    return best_key[0], best_q, count


# ------------------------------------------------------------ width & bounds

def reach(blk: Block) -> List[int]:
    """Transitive closure: reach[u] = units reachable from u (excluding u)."""
    r = [0] * blk.n
    for u in reversed(range(blk.n)):
        m = blk.succ[u]
        for v in bits(blk.succ[u]):
            m |= r[v]
        r[u] = m
    return r


def width_bruteforce(blk: Block) -> int:
    """Largest set of units with no path between any two (Definition, Sec. 4.2)."""
    rc = reach(blk)
    best = 0
    for m in range(1, 1 << blk.n):
        us = bits(m)
        if len(us) <= best:
            continue
        if all(not (rc[a] >> b & 1) and not (rc[b] >> a & 1)
               for a, b in itertools.combinations(us, 2)):
            best = len(us)
    return best


def width_dilworth(blk: Block) -> int:
    """n minus a maximum matching of the comparability bipartite graph,
    i.e. the size of a smallest chain decomposition (Dilworth, App. A)."""
    rc = reach(blk)
    match_r = [-1] * blk.n

    def augment(u, seen):
        for v in bits(rc[u]):
            if v in seen:
                continue
            seen.add(v)
            if match_r[v] < 0 or augment(match_r[v], seen):
                match_r[v] = u
                return True
        return False

    m = sum(1 for u in range(blk.n) if augment(u, set()))
    return blk.n - m


def transition_bound(n: int, d: int) -> float:
    """C(n/d + 2, 2)^d with the binomial taken as x(x-1)/2 (Theorem, Sec. 4.2)."""
    x = n / d + 2
    return (x * (x - 1) / 2) ** d


def fubini(n: int) -> int:
    """Ordered set partitions of n items (all schedules of n independent units)."""
    a = [1]
    for m in range(1, n + 1):
        a.append(sum(math.comb(m, k) * a[m - k] for k in range(1, m + 1)))
    return a[n]
