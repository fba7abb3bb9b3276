// extern "C" entry points of libios (declared and documented in ios.h).
// Every call catches the library's internal errors and returns a code.
#include <cstdlib>
#include <algorithm>
#include <array>
#include <cstring>
#include <new>

#include "ios_internal.h"

namespace ios {
int add_input(ios_graph *g, int c, int h, int w);
int add_op(ios_graph *g, const ios_op_desc *d, const int32_t *in_ids, int n_in, const float *weights,
           const float *bias);
void mark_output(ios_graph *g, int tid);
ios_schedule_t *run_schedule(ios_graph *g, const ios_sched_opts &o, ios_cost_fn fn, void *ctx,
                             int64_t *cost_ns);
ios_schedule_t *schedule_from_stages(ios_graph *g, int n_stages, const int32_t *off,
                                     const int32_t *ids, const int32_t *strat);
void dump_costs(const ios_graph *g, const char *path);
}  // namespace ios

using namespace ios;

// The calling thread's last error message, in a fixed buffer so that setting
// it never allocates (ios_run_noalloc reports errors through it too).
static thread_local char g_last_error[512];

void ios::set_last_error_text(const char *msg) {
  std::strncpy(g_last_error, msg, sizeof(g_last_error) - 1);
  g_last_error[sizeof(g_last_error) - 1] = 0;
}

template <class F>
static int guarded(F &&f) {
  try {
    f();
    return IOS_OK;
  } catch (const Error &e) {
    set_last_error_text(e.msg.c_str());
    return e.code;
  } catch (const std::bad_alloc &) {
    set_last_error_text("host allocation failed");
    return IOS_E_OOM;
  } catch (const std::exception &e) {
    set_last_error_text(e.what());
    return IOS_E_ARG;
  }
}

static void need(bool c, const char *msg) {
  if (!c) fail(IOS_E_ARG, msg);
}
static void need_final(const ios_graph *g) {
  need(g != nullptr, "null graph");
  if (!g->finalized) fail(IOS_E_STATE, "graph not finalized");
}

static std::vector<int> ops_of_units(const ios_graph *g, const int32_t *ids, int n) {
  need(ids != nullptr && n >= 1, "empty unit list");
  std::vector<int> ops;
  for (int i = 0; i < n; ++i) ops.push_back(unit_op_of_tensor(g, ids[i]));
  std::sort(ops.begin(), ops.end());
  if (std::adjacent_find(ops.begin(), ops.end()) != ops.end()) fail(IOS_E_BAD_STAGE, "unit repeated");
  return ops;
}

extern "C" {

const char *ios_last_error(void) { return g_last_error; }

int ios_graph_create(int32_t batch, ios_graph **out) {
  return guarded([&] {
    need(out != nullptr, "null output pointer");
    need(batch >= 1, "batch must be >= 1");
    ios_graph *g = new ios_graph;
    g->batch = batch;
    *out = g;
  });
}

void ios_graph_destroy(ios_graph *g) {
  if (!g) return;
  if (g->device_ready) (void)hipSetDevice(g->device);
  for (auto &b : g->bufs)
    if (b.dev) (void)hipFree(b.dev);
  for (auto &op : g->ops) {
    if (op.d_wpk) (void)hipFree(op.d_wpk);
    if (op.d_bias) (void)hipFree(op.d_bias);
    if (op.d_dw) (void)hipFree(op.d_dw);
    if (op.d_dw_row) (void)hipFree(op.d_dw_row);
    if (op.d_pw_row) (void)hipFree(op.d_pw_row);
    if (op.d_wg) (void)hipFree(op.d_wg);
    if (op.d_pw_pipe) (void)hipFree(op.d_pw_pipe);
    if (op.d_pw_line) (void)hipFree(op.d_pw_line);
  }
  CompiledStage &s = g->prof_stage;
  if (s.d_table) (void)hipFree(s.d_table);
  if (s.d_ctr) (void)hipFree(s.d_ctr);
  if (s.d_mw) (void)hipFree(s.d_mw);
  if (s.d_mb) (void)hipFree(s.d_mb);
  if (g->d_err) (void)hipFree(g->d_err);
  if (g->ev0) (void)hipEventDestroy(g->ev0);
  if (g->ev1) (void)hipEventDestroy(g->ev1);
  if (g->stream) (void)hipStreamDestroy(g->stream);
  delete g;
}

int ios_add_input(ios_graph *g, int32_t c, int32_t h, int32_t w, int32_t *tensor_id) {
  return guarded([&] {
    need(g != nullptr && tensor_id != nullptr, "null argument");
    *tensor_id = add_input(g, c, h, w);
  });
}

int ios_add_op(ios_graph *g, const ios_op_desc *d, const int32_t *in_ids, int32_t n_in,
               const float *weights, const float *bias, int32_t *out_tensor_id) {
  return guarded([&] {
    need(g != nullptr && out_tensor_id != nullptr, "null argument");
    *out_tensor_id = add_op(g, d, in_ids, n_in, weights, bias);
  });
}

int ios_mark_output(ios_graph *g, int32_t tensor_id) {
  return guarded([&] {
    need(g != nullptr, "null graph");
    mark_output(g, tensor_id);
  });
}

int ios_graph_finalize(ios_graph *g) {
  return guarded([&] {
    need(g != nullptr, "null graph");
    finalize_graph(g);
  });
}

int ios_graph_blocks(const ios_graph *g, int32_t *n_blocks) {
  return guarded([&] {
    need_final(g);
    need(n_blocks != nullptr, "null argument");
    *n_blocks = (int32_t)g->blocks.size();
  });
}

int ios_block_units(const ios_graph *g, int32_t block, int32_t *n, int32_t *unit_ids) {
  return guarded([&] {
    need_final(g);
    need(n != nullptr && unit_ids != nullptr, "null argument");
    need(block >= 0 && block < (int)g->blocks.size(), "block out of range");
    const Block &B = g->blocks[block];
    for (size_t i = 0; i < B.ops.size(); ++i) unit_ids[i] = g->ops[B.ops[i]].out;
    *n = (int32_t)B.ops.size();
  });
}

int ios_stage_mergeable(ios_graph *g, const int32_t *unit_ids, int32_t n, int32_t *ok) {
  return guarded([&] {
    need_final(g);
    need(ok != nullptr, "null argument");
    *ok = stage_mergeable(g, ops_of_units(g, unit_ids, n)) ? 1 : 0;
  });
}

int ios_profile_stage(ios_graph *g, const int32_t *unit_ids, int32_t n, int32_t strategy,
                      int32_t warmup, int32_t reps, int32_t repeats, int64_t *latency_ns) {
  return guarded([&] {
    need_final(g);
    need(latency_ns != nullptr, "null argument");
    std::vector<int> ops = ops_of_units(g, unit_ids, n);
    if (strategy == IOS_MERGE && !stage_mergeable(g, ops)) fail(IOS_E_NOT_MERGEABLE, "stage cannot be merged");
    if (strategy != IOS_MERGE && strategy != IOS_CONCURRENT) fail(IOS_E_ARG, "unknown strategy");
    ensure_device(g);
    *latency_ns = profile_stage(g, ops, strategy, warmup, reps, repeats);
  });
}

int ios_get_conv_tile(ios_graph *g, int32_t unit_id, int32_t *shape) {
  return guarded([&] {
    need_final(g);
    need(shape != nullptr, "null argument");
    const int op = unit_op_of_tensor(g, unit_id);
    need(g->ops[op].d.kind == IOS_CONV, "not a conv unit");
    ensure_device(g);
    *shape = g->ops[op].tcfg;
  });
}

int ios_set_conv_tile(ios_graph *g, int32_t unit_id, int32_t shape) {
  return guarded([&] {
    need_final(g);
    const int op = unit_op_of_tensor(g, unit_id);
    need(g->ops[op].d.kind == IOS_CONV, "not a conv unit");
    need(shape >= 0 && shape < TC_COUNT, "tile shape out of range");
    need(conv_tile_ok(g->ops[op], shape), "pipelined tile shape not applicable to this conv");
    ensure_device(g);
    g->ops[op].tcfg = shape;
  });
}

int ios_get_unit_tiling(ios_graph *g, int32_t unit_id, int32_t *tile, int32_t *xcd_lg) {
  return guarded([&] {
    need_final(g);
    need(tile != nullptr && xcd_lg != nullptr, "null argument");
    const Op &op = g->ops[unit_op_of_tensor(g, unit_id)];
    ensure_device(g);
    *tile = op.d.kind == IOS_CONV ? op.tcfg : op.d.kind == IOS_SEPCONV ? op.sep_tile : 0;
    *xcd_lg = op.xcd_lg;
  });
}

int ios_set_unit_tiling(ios_graph *g, int32_t unit_id, int32_t tile, int32_t xcd_lg) {
  return guarded([&] {
    need_final(g);
    Op &op = g->ops[unit_op_of_tensor(g, unit_id)];
    need(xcd_lg == -1 || xcd_lg == 0 || xcd_lg == 2 || xcd_lg == 4, "xcd_lg must be -1, 0, 2 or 4");
    if (op.d.kind == IOS_CONV) {
      need(tile >= 0 && tile < TC_COUNT, "conv tile shape out of range");
      need(conv_tile_ok(op, tile), "pipelined tile shape not applicable to this conv");
    } else if (op.d.kind == IOS_SEPCONV) {
      need(sep_tile_ok(op, tile), "SEPCONV tile choice out of range or not applicable to this unit");
    } else {
      need(tile == 0, "this unit kind has no tile choice (tile must be 0)");
    }
    ensure_device(g);
    if (op.d.kind == IOS_CONV) op.tcfg = tile;
    else if (op.d.kind == IOS_SEPCONV) op.sep_tile = tile;
    op.xcd_lg = xcd_lg;
  });
}

void ios_sched_opts_default(ios_sched_opts *o) {
  if (!o) return;
  o->mode = IOS_SCHED_DP;
  o->r = 3;
  o->s = 8;
  o->strategies = 3;
  o->warmup = 3;
  o->reps = 20;
  o->repeats = 3;
  o->verify_reps = 0;
}

int ios_schedule(ios_graph *g, const ios_sched_opts *opts, ios_cost_fn fn, void *ctx,
                 ios_schedule_t **out, int64_t *cost_ns) {
  return guarded([&] {
    need_final(g);
    need(out != nullptr && cost_ns != nullptr, "null argument");
    ios_sched_opts o;
    ios_sched_opts_default(&o);
    if (opts) o = *opts;
    if (!fn) ensure_device(g);
    int64_t c = 0;
    ios_schedule_t *q = run_schedule(g, o, fn, ctx, &c);
    *out = q;
    *cost_ns = c;
  });
}

int ios_schedule_from_stages(ios_graph *g, int32_t n_stages, const int32_t *stage_offsets,
                             const int32_t *unit_ids, const int32_t *strategies,
                             ios_schedule_t **out) {
  return guarded([&] {
    need_final(g);
    need(out != nullptr, "null argument");
    *out = schedule_from_stages(g, n_stages, stage_offsets, unit_ids, strategies);
  });
}

// Conv tile shapes, SEPCONV output blocks per tile and the XCD tile order
// chosen per stage: each stage of q is measured with its tile order's run
// length set explicitly (else the stage kernel's L2-fill model picks it),
// with its convs' shapes varied one conv at a time (all of them together in
// a merge stage, whose merged conv takes one shape) and with each SEPCONV's
// tile choice varied, keeping a change only when the stage gets faster
// by more than kStageTileSlack.  A shape measured alone
// fills the GPU by itself; inside a stage other operators share the CUs, so
// larger tiles can pay off there.
static constexpr double kStageTileSlack = 0.02;

int ios_schedule_tune_tiles(ios_graph *g, ios_schedule_t *q, const ios_sched_opts *opts,
                            int64_t *cost_ns) {
  return guarded([&] {
    need_final(g);
    need(q != nullptr && q->g == g, "schedule does not belong to this graph");
    need(cost_ns != nullptr, "null argument");
    ios_sched_opts o;
    ios_sched_opts_default(&o);
    if (opts) o = *opts;
    need(o.warmup >= 0 && o.reps >= 1 && o.repeats >= 1, "bad profiling counts");
    ensure_device(g);
    const bool forced = std::getenv("IOS_CONV_TILE") != nullptr;
    const bool sep_forced = std::getenv("IOS_SEP_TILE") != nullptr;
    // on an error the units get their shapes and orders back
    std::vector<std::array<int, 4>> saved;
    for (int32_t u : q->unit_ids) {
      const int op = unit_op_of_tensor(g, u);
      saved.push_back({op, g->ops[op].tcfg, g->ops[op].xcd_lg, g->ops[op].sep_tile});
    }
    int64_t total = 0;
    try {
      for (size_t k = 0; k < q->strategies.size(); ++k) {
        std::vector<int> ops, convs;
        for (int i = q->offsets[k]; i < q->offsets[k + 1]; ++i) {
          const int op = unit_op_of_tensor(g, q->unit_ids[i]);
          ops.push_back(op);
          if (g->ops[op].d.kind == IOS_CONV) convs.push_back(op);
        }
        const int strat = q->strategies[k];
        auto measure = [&] { return profile_stage(g, ops, strat, o.warmup, o.reps, o.repeats); };
        for (int op : ops) g->ops[op].xcd_lg = -1;
        int64_t best = measure();
        // the XCD run length of the stage's tile order (see the stage kernel):
        // the modelled choice, or an explicit one measured faster
        auto tune_xcd_order = [&] {
          int keep = -1;
          for (int lg : {0, 2, 4}) {
            for (int op : ops) g->ops[op].xcd_lg = lg;
            const int64_t ns = measure();
            if ((double)ns < (double)best * (1.0 - kStageTileSlack)) {
              best = ns;
              keep = lg;
            }
          }
          for (int op : ops) g->ops[op].xcd_lg = keep;
          return keep >= 0;
        };
        // knobs: the convs that take one tile shape together (all of a merge
        // stage's), and each SEPCONV's tile choice; in a concurrent stage
        // also all its convs, and all its SEPCONVs, moved together first (a
        // wide stage can be bound by its operators' throughput together,
        // which no single operator's change shows)
        struct Knob {
          std::vector<int> ops;
          bool sep;
          int lo, hi;
        };
        std::vector<Knob> knobs;
        std::vector<int> seps;
        for (int op : ops)
          if (g->ops[op].d.kind == IOS_SEPCONV) seps.push_back(op);
        if (!forced && !convs.empty()) {
          if (strat == IOS_MERGE) {
            int largest = convs[0];
            for (int c : convs)
              if (g->ops[c].d.cout > g->ops[largest].d.cout) largest = c;
            for (int c : convs) g->ops[c].tcfg = g->ops[largest].tcfg;
            best = measure();
            knobs.push_back({convs, false, 0, TC_COUNT - 1});
          } else {
            if (convs.size() > 1) knobs.push_back({convs, false, 0, TC_COUNT - 1});
            for (int c : convs) knobs.push_back({{c}, false, 0, TC_COUNT - 1});
          }
        }
        if (!sep_forced) {
          if (seps.size() > 1) knobs.push_back({seps, true, 0, kSepTiles - 1});
          for (int op : seps) knobs.push_back({{op}, true, 0, kSepTiles - 1});
        }
        auto val = [&](int op, bool sep) -> int & { return sep ? g->ops[op].sep_tile : g->ops[op].tcfg; };
        auto ok = [&](int op, bool sep, int v) {
          return sep ? sep_tile_ok(g->ops[op], v) : conv_tile_ok(g->ops[op], v);
        };
        for (int pass = 0; pass < 2; ++pass) {
          bool improved = pass == 0 && tune_xcd_order();
          for (const auto &kn : knobs) {
            // a value applies to the knob's operators that admit it; the
            // others keep theirs
            std::vector<int> keep;
            for (int c : kn.ops) keep.push_back(val(c, kn.sep));
            for (int v = kn.lo; v <= kn.hi; ++v) {
              bool change = false;
              for (size_t i = 0; i < kn.ops.size(); ++i) change |= ok(kn.ops[i], kn.sep, v) && keep[i] != v;
              if (!change) continue;
              for (size_t i = 0; i < kn.ops.size(); ++i)
                val(kn.ops[i], kn.sep) = ok(kn.ops[i], kn.sep, v) ? v : keep[i];
              const int64_t ns = measure();
              if ((double)ns < (double)best * (1.0 - kStageTileSlack)) {
                best = ns;
                for (size_t i = 0; i < kn.ops.size(); ++i) keep[i] = val(kn.ops[i], kn.sep);
                improved = true;
              }
            }
            for (size_t i = 0; i < kn.ops.size(); ++i) val(kn.ops[i], kn.sep) = keep[i];
          }
          if (!improved) break;
        }
        total += best;
      }
    } catch (...) {
      for (const auto &v : saved) {
        g->ops[v[0]].tcfg = v[1];
        g->ops[v[0]].xcd_lg = v[2];
        g->ops[v[0]].sep_tile = v[3];
      }
      throw;
    }
    // stages compiled for q before this call used the old shapes
    for (auto &cs : q->compiled)
      if (cs) free_stage(cs.get());
    q->compiled.clear();
    *cost_ns = total;
  });
}

int ios_schedule_get(const ios_schedule_t *q, int32_t *n_stages, const int32_t **stage_offsets,
                     const int32_t **unit_ids, const int32_t **strategies) {
  return guarded([&] {
    need(q != nullptr && n_stages != nullptr, "null argument");
    *n_stages = (int32_t)q->strategies.size();
    if (stage_offsets) *stage_offsets = q->offsets.data();
    if (unit_ids) *unit_ids = q->unit_ids.data();
    if (strategies) *strategies = q->strategies.data();
  });
}

int ios_schedule_stats(const ios_schedule_t *q, int64_t *states, int64_t *transitions,
                       int64_t *stages_measured) {
  return guarded([&] {
    need(q != nullptr, "null schedule");
    if (states) *states = q->states;
    if (transitions) *transitions = q->transitions;
    if (stages_measured) *stages_measured = q->measured;
  });
}

void ios_schedule_destroy(ios_schedule_t *q) {
  if (!q) return;
  if (q->g && q->g->device_ready) (void)hipSetDevice(q->g->device);
  for (auto &cs : q->compiled)
    if (cs) free_stage(cs.get());
  for (auto e : q->events) (void)hipEventDestroy(e);
  delete q;
}

int ios_schedule_dump_costs(const ios_graph *g, const char *path) {
  return guarded([&] {
    need_final(g);
    need(path != nullptr, "null path");
    dump_costs(g, path);
  });
}

static std::vector<float *> run_buffers(ios_graph *g, const float *const *d_inputs,
                                        float *const *d_outputs) {
  need(g->inputs.empty() || d_inputs != nullptr, "null input list");
  need(g->outputs.empty() || d_outputs != nullptr, "null output list");
  std::vector<float *> p = default_buffers(g);
  for (size_t i = 0; i < g->bufs.size(); ++i) {
    const Buffer &b = g->bufs[i];
    if (b.input_index >= 0) {
      need(d_inputs[b.input_index] != nullptr, "null input pointer");
      p[i] = const_cast<float *>(d_inputs[b.input_index]);
    }
    if (b.output_index >= 0) {
      need(d_outputs[b.output_index] != nullptr, "null output pointer");
      p[i] = d_outputs[b.output_index];
    }
  }
  return p;
}

static void ensure_compiled(ios_graph *g, ios_schedule_t *q) {
  if (q->compiled.size() == q->strategies.size()) return;
  q->compiled.clear();
  for (size_t k = 0; k < q->strategies.size(); ++k) {
    std::vector<int> ops;
    for (int i = q->offsets[k]; i < q->offsets[k + 1]; ++i) ops.push_back(unit_op_of_tensor(g, q->unit_ids[i]));
    std::unique_ptr<CompiledStage> cs(new CompiledStage);
    compile_stage(g, ops, q->strategies[k], cs.get(), false);
    q->compiled.push_back(std::move(cs));
  }
}

int ios_run(ios_graph *g, ios_schedule_t *q, const float *const *d_inputs, float *const *d_outputs,
            void *hip_stream) {
  return guarded([&] {
    need_final(g);
    need(q != nullptr && q->g == g, "schedule does not belong to this graph");
    ensure_device(g);
    ensure_compiled(g, q);
    std::vector<float *> p = run_buffers(g, d_inputs, d_outputs);
    hipStream_t s = (hipStream_t)hip_stream;
    for (auto &cs : q->compiled) launch_compiled(g, *cs, p, s);
  });
}

int ios_run_timed(ios_graph *g, ios_schedule_t *q, const float *const *d_inputs,
                  float *const *d_outputs, void *hip_stream, int64_t *stage_ns) {
  return guarded([&] {
    need_final(g);
    need(q != nullptr && q->g == g, "schedule does not belong to this graph");
    need(stage_ns != nullptr, "null argument");
    ensure_device(g);
    ensure_compiled(g, q);
    std::vector<float *> p = run_buffers(g, d_inputs, d_outputs);
    hipStream_t s = (hipStream_t)hip_stream;
    size_t n = q->compiled.size();
    while (q->events.size() < n + 1) {
      hipEvent_t e;
      hip_check(hipEventCreate(&e), "hipEventCreate");
      q->events.push_back(e);
    }
    hip_check(hipEventRecord(q->events[0], s), "hipEventRecord");
    for (size_t k = 0; k < n; ++k) {
      launch_compiled(g, *q->compiled[k], p, s);
      hip_check(hipEventRecord(q->events[k + 1], s), "hipEventRecord");
    }
    hip_check(hipEventSynchronize(q->events[n]), "hipEventSynchronize");
    for (size_t k = 0; k < n; ++k) {
      float ms = 0.f;
      hip_check(hipEventElapsedTime(&ms, q->events[k], q->events[k + 1]), "hipEventElapsedTime");
      stage_ns[k] = (int64_t)((double)ms * 1e6 + 0.5);
    }
  });
}

int ios_device_status(ios_graph *g, void *hip_stream, int32_t *flags) {
  return guarded([&] {
    need_final(g);
    need(flags != nullptr, "null argument");
    ensure_device(g);
    hip_check(hipStreamSynchronize((hipStream_t)hip_stream), "hipStreamSynchronize");
    int32_t v = 0;
    hip_check(hipMemcpy(&v, g->d_err, sizeof(v), hipMemcpyDeviceToHost), "hipMemcpy(err)");
    if (v) hip_check(hipMemset(g->d_err, 0, sizeof(int32_t)), "hipMemset(err)");
    *flags = v;
  });
}

}  // extern "C"
