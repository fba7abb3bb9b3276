// Host-side schedule search (Sec. 4, Algorithm 1) and the baseline
// schedules of Sec. 6.1 (sequential, greedy).
//
// For each block the dynamic program runs over states S (units still to be
// scheduled, as 64-bit block-local masks):
//   cost[S] = min over endings S' of S  of  cost[S - S'] + stage_latency[S']
// with cost[{}] = 0 (Sec. 4.1).  An ending S' of S is a non-empty subset with
// no edge from S' to S - S'; only endings satisfying the pruning strategy
// P(r, s) are tried: at most s groups (connected components of S'), each of
// at most r units (Sec. 4.3).  stage_latency comes from GenerateStage: the
// concurrent latency, and the merge latency when the units can merge; merge
// wins unless concurrent is strictly faster.  Among endings of equal total
// cost the smallest mask is kept, so the result does not depend on the
// enumeration order.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <functional>
#include <unordered_map>
#include <unordered_set>

#include "ios_internal.h"

namespace ios {

namespace {

inline int popcount(uint64_t x) { return __builtin_popcountll(x); }
inline int ctz(uint64_t x) { return __builtin_ctzll(x); }

// Connected component of `u` inside `set` (edges undirected).
uint64_t component(const Block &B, uint64_t set, int u) {
  uint64_t comp = 1ull << u, frontier = comp;
  while (frontier) {
    uint64_t nb = 0;
    for (uint64_t f = frontier; f; f &= f - 1) {
      int v = ctz(f);
      nb |= B.succ[v] | B.pred[v];
    }
    nb &= set;
    frontier = nb & ~comp;
    comp |= nb;
  }
  return comp;
}

int count_groups(const Block &B, uint64_t set) {
  int n = 0;
  while (set) {
    set &= ~component(B, set, ctz(set));
    ++n;
  }
  return n;
}

// Every ending of S satisfying P(r, s).  Units are decided from the highest
// local index down (reverse topological order): a unit may join S' only when
// all of its successors inside S already have.  A group can only grow as
// units join, so a branch whose group exceeds r is abandoned at once.
void enum_endings(const Block &B, uint64_t S, int r, int s, std::vector<uint64_t> &out) {
  int order[64], n = 0;
  for (int i = 63; i >= 0; --i)
    if (S >> i & 1) order[n++] = i;
  std::function<void(int, uint64_t)> rec = [&](int i, uint64_t cur) {
    if (i == n) {
      if (cur && (s <= 0 || count_groups(B, cur) <= s)) out.push_back(cur);
      return;
    }
    int u = order[i];
    rec(i + 1, cur);
    if ((B.succ[u] & S & ~cur) == 0) {
      uint64_t nxt = cur | (1ull << u);
      if (r <= 0 || popcount(component(B, nxt, u)) <= r) rec(i + 1, nxt);
    }
  };
  rec(0, 0);
}

std::vector<int> ops_of_mask(const Block &B, uint64_t m) {
  std::vector<int> v;
  for (; m; m &= m - 1) v.push_back(B.ops[ctz(m)]);
  return v;
}

inline int64_t sat_add(int64_t a, int64_t b) {
  if (a == kInf || b == kInf) return kInf;
  return a + b;
}

struct Provider {
  ios_graph *g;
  ios_cost_fn fn;
  void *ctx;
  ios_sched_opts o;
  int64_t measured = 0;

  // A stage of several SEPCONVs can be bound by their throughput together,
  // which the isolated tile choice of each (the row or the 32-channel line
  // tile, at batch 1) misjudges; such a stage is also measured with every
  // SEPCONV that admits it on the GEMM tile, and again on the 64-channel line
  // tile, and the fastest figure is the stage's latency (the per-stage tile
  // tuning of the chosen schedule makes the same choice).  IOS_SEP_TILE in
  // the environment keeps the choices fixed.
  int64_t measure(const std::vector<int> &ops, int strategy, int warmup, int reps, int repeats) {
    int64_t ns = profile_stage(g, ops, strategy, warmup, reps, repeats);
    if (strategy != IOS_CONCURRENT || std::getenv("IOS_SEP_TILE")) return ns;
    for (const int first : {kSepgFirst, kSepLineFirst + 1}) {
      const int second = first == kSepgFirst ? kSepgFirst + 1 : kSepLineFirst;
      std::vector<std::pair<int, int>> saved;
      for (int oi : ops) {
        Op &op = g->ops[oi];
        if (op.d.kind != IOS_SEPCONV) continue;
        const int v = sep_tile_ok(op, first) ? first : sep_tile_ok(op, second) ? second : -1;
        if (v < 0 || v == op.sep_tile) continue;
        saved.push_back({oi, op.sep_tile});
        op.sep_tile = v;
      }
      auto restore = [&] {
        for (const auto &p : saved) g->ops[p.first].sep_tile = p.second;
      };
      if (saved.size() < 2) {
        restore();
        continue;
      }
      int64_t ns2;
      try {
        ns2 = profile_stage(g, ops, strategy, warmup, reps, repeats);
      } catch (...) {
        restore();
        throw;
      }
      restore();
      ns = std::min(ns, ns2);
    }
    return ns;
  }

  int64_t latency(int block, uint64_t mask, int strategy, bool verify = false) {
    const Block &B = g->blocks[block];
    auto ops = ops_of_mask(B, mask);
    int64_t ns = kInf;
    if (verify) {
      ns = measure(ops, strategy, 3, o.verify_reps, 3);
    } else if (fn) {
      std::vector<int32_t> ids;
      for (int oi : ops) ids.push_back(g->ops[oi].out);
      int rc = fn(ctx, block, mask, ids.data(), (int32_t)ids.size(), strategy, &ns);
      if (rc != 0) fail(IOS_E_COST_FN, "cost callback returned " + std::to_string(rc));
      if (ns < 0) fail(IOS_E_COST_FN, "cost callback returned a negative latency");
    } else {
      ns = measure(ops, strategy, o.warmup, o.reps, o.repeats);
    }
    ++measured;
    CostRow &row = g->cost_table[block][mask];
    if (strategy == IOS_MERGE) {
      row.merge = ns;
      row.merge_measured = true;
    } else {
      row.conc = ns;
    }
    return ns;
  }

  // GenerateStage (Algorithm 1): the better strategy and its latency
  // (verify: measured with the verification protocol).
  std::pair<int64_t, int> generate_stage(int block, uint64_t mask, bool verify = false) {
    const Block &B = g->blocks[block];
    // with concurrent execution off (IOS-Merge) a one-unit stage still runs alone
    bool single = (mask & (mask - 1)) == 0;
    int64_t lc = ((o.strategies & 1) || single) ? latency(block, mask, IOS_CONCURRENT, verify) : kInf;
    int64_t lm = kInf;
    if ((o.strategies & 2) && stage_mergeable(g, ops_of_mask(B, mask)))
      lm = latency(block, mask, IOS_MERGE, verify);
    if (lc < lm) return {lc, IOS_CONCURRENT};
    return {lm, IOS_MERGE};
  }
};

struct Memo {
  int64_t cost;
  uint64_t choice;
  int strategy;
};

struct BlockDP {
  Provider &P;
  int block;
  const Block &B;
  int r, s;
  std::unordered_map<uint64_t, Memo> memo;
  std::unordered_map<uint64_t, std::pair<int64_t, int>> stages;
  int64_t transitions = 0;

  std::pair<int64_t, int> stage(uint64_t m) {
    auto it = stages.find(m);
    if (it != stages.end()) return it->second;
    auto v = P.generate_stage(block, m);
    stages.emplace(m, v);
    return v;
  }

  int64_t scheduler(uint64_t S) {
    auto it = memo.find(S);
    if (it != memo.end()) return it->second.cost;
    std::vector<uint64_t> ends;
    enum_endings(B, S, r, s, ends);
    Memo best{kInf, 0, IOS_CONCURRENT};
    for (uint64_t Sp : ends) {
      ++transitions;
      auto st = stage(Sp);
      int64_t c = sat_add(scheduler(S & ~Sp), st.first);
      if (c < best.cost || (c == best.cost && c != kInf && Sp < best.choice)) {
        best.cost = c;
        best.choice = Sp;
        best.strategy = st.second;
      }
    }
    memo[S] = best;
    return best.cost;
  }
};

void append_stage(ios_schedule_t *q, ios_graph *g, int block, uint64_t mask, int strategy) {
  const Block &B = g->blocks[block];
  for (uint64_t m = mask; m; m &= m - 1) q->unit_ids.push_back(g->ops[B.ops[ctz(m)]].out);
  q->offsets.push_back((int32_t)q->unit_ids.size());
  q->strategies.push_back(strategy);
  q->stage_block.push_back(block);
}

}  // namespace

ios_schedule_t *run_schedule(ios_graph *g, const ios_sched_opts &o, ios_cost_fn fn, void *ctx,
                             int64_t *cost_ns) {
  if (!(o.strategies & 1) && !(o.strategies & 2)) fail(IOS_E_ARG, "no strategy enabled");
  if (o.mode < IOS_SCHED_DP || o.mode > IOS_SCHED_GREEDY) fail(IOS_E_ARG, "unknown mode");
  g->cost_table.assign(g->blocks.size(), {});
  Provider P{g, fn, ctx, o};
  std::unique_ptr<ios_schedule_t> q(new ios_schedule_t);
  q->g = g;
  q->offsets.push_back(0);
  int64_t total = 0;
  for (int b = 0; b < (int)g->blocks.size(); ++b) {
    const Block &B = g->blocks[b];
    if (o.mode == IOS_SCHED_DP) {
      BlockDP dp{P, b, B, o.r, o.s, {}, {}, 0};
      dp.memo[0] = Memo{0, 0, IOS_CONCURRENT};
      int64_t c = dp.scheduler(B.full());
      if (c == kInf) fail(IOS_E_BAD_STAGE, "no schedule satisfies the pruning strategy");
      const int64_t states0 = (int64_t)dp.memo.size(), transitions0 = dp.transitions;   // the search itself
      auto chosen = [&]() {
        std::vector<std::pair<uint64_t, int>> rev;
        for (uint64_t S = B.full(); S;) {
          const Memo &m = dp.memo.at(S);
          rev.push_back({m.choice, m.strategy});
          S &= ~m.choice;
        }
        return rev;
      };
      std::vector<std::pair<uint64_t, int>> rev = chosen();
      if (o.verify_reps > 0 && !fn) {
        // verification rounds: measure the picked stages again, replace their
        // entries, search again on the updated table
        std::unordered_set<uint64_t> verified;
        for (int round = 0; round < 16; ++round) {
          bool fresh = false;
          for (const auto &st : rev)
            if (verified.insert(st.first).second) {
              dp.stages[st.first] = P.generate_stage(b, st.first, true);
              fresh = true;
            }
          if (!fresh) break;
          dp.memo.clear();
          dp.memo[0] = Memo{0, 0, IOS_CONCURRENT};
          c = dp.scheduler(B.full());
          rev = chosen();
        }
      }
      total = sat_add(total, c);
      for (auto it = rev.rbegin(); it != rev.rend(); ++it) append_stage(q.get(), g, b, it->first, it->second);
      q->states += states0;
      q->transitions += transitions0;
    } else if (o.mode == IOS_SCHED_SEQUENTIAL) {
      for (int i = 0; i < (int)B.ops.size(); ++i) {
        int64_t c = P.latency(b, 1ull << i, IOS_CONCURRENT);
        total = sat_add(total, c);
        append_stage(q.get(), g, b, 1ull << i, IOS_CONCURRENT);
      }
    } else {
      uint64_t rem = B.full();
      while (rem) {
        uint64_t ready = 0;
        for (uint64_t m = rem; m; m &= m - 1) {
          int u = ctz(m);
          if ((B.pred[u] & rem) == 0) ready |= 1ull << u;
        }
        int64_t c = P.latency(b, ready, IOS_CONCURRENT);
        total = sat_add(total, c);
        append_stage(q.get(), g, b, ready, IOS_CONCURRENT);
        rem &= ~ready;
      }
    }
  }
  q->measured = P.measured;
  *cost_ns = total;
  return q.release();
}

ios_schedule_t *schedule_from_stages(ios_graph *g, int n_stages, const int32_t *off,
                                     const int32_t *ids, const int32_t *strat) {
  if (n_stages < 1 || !off || !ids || !strat) fail(IOS_E_ARG, "bad stage list");
  if (off[0] != 0) fail(IOS_E_ARG, "stage_offsets[0] must be 0");
  std::vector<int> stage_of(g->ops.size(), -1);
  std::unique_ptr<ios_schedule_t> q(new ios_schedule_t);
  q->g = g;
  q->offsets.push_back(0);
  int last_block = -1;
  int total_units = 0;
  for (int k = 0; k < n_stages; ++k) {
    if (off[k + 1] <= off[k]) fail(IOS_E_BAD_STAGE, "empty stage");
    if (strat[k] != IOS_CONCURRENT && strat[k] != IOS_MERGE) fail(IOS_E_ARG, "bad strategy");
    std::vector<int> ops;
    for (int i = off[k]; i < off[k + 1]; ++i) ops.push_back(unit_op_of_tensor(g, ids[i]));
    std::sort(ops.begin(), ops.end());
    if (std::adjacent_find(ops.begin(), ops.end()) != ops.end())
      fail(IOS_E_BAD_STAGE, "unit repeated in a stage");
    int b = g->ops[ops[0]].block;
    for (int oi : ops) {
      if (g->ops[oi].block != b) fail(IOS_E_BAD_STAGE, "stage spans several blocks");
      if (stage_of[oi] >= 0) fail(IOS_E_BAD_STAGE, "unit scheduled twice");
    }
    if (b < last_block) fail(IOS_E_BAD_STAGE, "blocks out of order");
    last_block = b;
    for (int oi : ops) stage_of[oi] = k;
    for (int oi : ops)
      for (int t : g->ops[oi].in)
        for (int p : unit_producers(g, t)) {
          if (stage_of[p] < 0 || stage_of[p] > k)
            fail(IOS_E_BAD_STAGE, "a unit is scheduled before its producer");
          if (stage_of[p] == k && strat[k] == IOS_MERGE)
            fail(IOS_E_NOT_MERGEABLE, "merge stage contains a dependency");
        }
    if (strat[k] == IOS_MERGE && !stage_mergeable(g, ops))
      fail(IOS_E_NOT_MERGEABLE, "stage cannot be merged");
    for (int oi : ops) q->unit_ids.push_back(g->ops[oi].out);
    q->offsets.push_back((int32_t)q->unit_ids.size());
    q->strategies.push_back(strat[k]);
    q->stage_block.push_back(b);
    total_units += (int)ops.size();
  }
  if (total_units != (int)g->units.size()) fail(IOS_E_BAD_STAGE, "schedule misses some units");
  return q.release();
}

void dump_costs(const ios_graph *g, const char *path) {
  FILE *f = std::fopen(path, "w");
  if (!f) fail(IOS_E_ARG, std::string("cannot open ") + path);
  for (int b = 0; b < (int)g->cost_table.size(); ++b) {
    const Block &B = g->blocks[b];
    for (const auto &kv : g->cost_table[b]) {
      std::fprintf(f, "{\"block\": %d, \"mask\": %llu, \"units\": [", b, (unsigned long long)kv.first);
      bool first = true;
      for (uint64_t m = kv.first; m; m &= m - 1) {
        std::fprintf(f, first ? "%d" : ", %d", g->ops[B.ops[ctz(m)]].out);
        first = false;
      }
      std::fprintf(f, "], \"concurrent_ns\": ");
      if (kv.second.conc == kInf) std::fprintf(f, "null"); else std::fprintf(f, "%lld", (long long)kv.second.conc);
      std::fprintf(f, ", \"merge_ns\": ");
      if (!kv.second.merge_measured || kv.second.merge == kInf) std::fprintf(f, "null");
      else std::fprintf(f, "%lld", (long long)kv.second.merge);
      std::fprintf(f, "}\n");
    }
  }
  std::fclose(f);
}

}  // namespace ios
