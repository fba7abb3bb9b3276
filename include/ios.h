/*
 * ios.h — C ABI of libios: inter-operator scheduling and stage execution of
 * multi-branch CNN blocks on one AMD Instinct MI355X (gfx950).
 *
 * The library implements the method of "IOS: Inter-Operator Scheduler for CNN
 * Acceleration" (Ding et al., MLSys 2021):
 *   - a computation graph G = (V, E) of schedule units (Sec. 3, "Computation
 *     Graph"; Table 2 "Conv-Relu" / "Relu-SepConv" units);
 *   - stages executed one after another, each with a parallelization strategy,
 *     "concurrent execution" or "operator merge" (Sec. 3, "Stage",
 *     "Parallelization Strategy", "Schedule");
 *   - the dynamic program over endings that picks the schedule minimising the
 *     summed stage latency (Sec. 4.1, Algorithm 1), with schedule pruning
 *     P(r, s) (Sec. 4.3) and block-wise optimisation (Sec. 4.2);
 *   - stage latencies measured on the device (Sec. 4.1, GenerateStage; Sec. 5).
 *
 * Conventions for every call:
 *   - Activations are float32, NCHW, contiguous; the batch N is fixed per graph.
 *   - Host arrays passed in are only read during the call and are copied where
 *     kept (the caller keeps ownership).  Device pointers are never freed by
 *     the library.
 *   - Every call returns IOS_OK (0) or a negative IOS_E_* code; on error
 *     ios_last_error() returns a message for the calling thread and no output
 *     argument is written.  No C++ exception crosses this ABI.
 *   - A graph handle (and every schedule made from it) must be used by one
 *     thread at a time.
 */
#ifndef IOS_H_
#define IOS_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ----------------------------------------------------------------- errors */
enum {
  IOS_OK = 0,
  IOS_E_ARG = -1,            /* null pointer, bad id, value out of range          */
  IOS_E_SHAPE = -2,          /* tensor shapes do not fit the operator             */
  IOS_E_STATE = -3,          /* call not allowed before/after ios_graph_finalize  */
  IOS_E_NOT_MERGEABLE = -4,  /* operator merge asked for a set that cannot merge  */
  IOS_E_BAD_STAGE = -5,      /* units do not form a valid stage / schedule        */
  IOS_E_TOO_MANY_OPS = -6,   /* more than 64 schedule units in one block          */
  IOS_E_OOM = -7,            /* host or device allocation failed                  */
  IOS_E_HIP = -8,            /* a HIP runtime call failed                         */
  IOS_E_COST_FN = -9,        /* the caller's cost callback returned non-zero      */
  IOS_E_UNSUPPORTED = -10,   /* valid request outside what the library supports   */
  IOS_E_DEVICE = -11         /* a stage kernel reported an error (see ios_device_status) */
};

/* --------------------------------------------------------------- operators */
/* Schedule-unit kinds.  CONCAT and IDENTITY are views: they create a tensor
 * but no schedule unit (producers of a concat write straight into its
 * channel slices, which plays the role of the paper's split/concat). */
enum {
  IOS_CONV = 0,      /* dense conv + bias ("Conv-Relu", Table 2)                 */
  IOS_SEPCONV = 1,   /* sum(inputs) -> ReLU -> depthwise kxk -> pointwise 1x1    */
  IOS_POOL_MAX = 2,  /* kxk max pool; taps outside the input are ignored         */
  IOS_POOL_AVG = 3,  /* kxk average pool; divides by kh*kw (padding counts 0)    */
  IOS_ADD = 4,       /* elementwise sum of n >= 1 inputs                          */
  IOS_MEAN = 5,      /* elementwise mean of n >= 1 inputs                         */
  IOS_CONCAT = 6,    /* channel concatenation, in input order (view)              */
  IOS_IDENTITY = 7   /* the input itself (view)                                   */
};

typedef struct {
  int32_t kind;                /* IOS_CONV .. IOS_IDENTITY                          */
  int32_t cout;                /* CONV / SEPCONV output channels; ignored otherwise */
  int32_t kh, kw;              /* CONV, pools: window; SEPCONV: depthwise window    */
  int32_t stride_h, stride_w;  /* CONV, pools (SEPCONV requires 1)                  */
  int32_t pad_h, pad_w;        /* zero padding (CONV, SEPCONV, POOL_AVG); max pool
                                  ignores out-of-bounds taps                        */
  int32_t pre_relu;            /* ReLU applied to the input (SEPCONV: to the sum)   */
  int32_t post_relu;           /* ReLU applied to the output (CONV only)            */
  int32_t block_id;            /* -1 = automatic; else >= 0, see ios_graph_finalize */
} ios_op_desc;

typedef struct ios_graph ios_graph;
typedef struct ios_schedule_t ios_schedule_t;

/* Create an empty graph for batch size `batch` (>= 1).  The paper tunes a
 * schedule per batch size (Sec. 7.2), so the batch is fixed per graph.
 * *out receives a handle owned by the caller; free it with ios_graph_destroy.
 * Errors: IOS_E_ARG (batch < 1, out NULL), IOS_E_OOM. */
int ios_graph_create(int32_t batch, ios_graph **out);

/* Free a graph and every device buffer it owns.  Schedules made from it must
 * be destroyed first.  NULL is ignored. */
void ios_graph_destroy(ios_graph *g);

/* Declare a graph input of shape [batch][c][h][w] (float32 NCHW): a tensor
 * of the computation graph G = (V, E) that no operator of G produces
 * (Sec. 3, "Computation Graph": edges carry tensors between operators; the
 * block's input feeds its first operators).  Inputs are numbered 0, 1, ...
 * in call order; ios_run takes them in that order.
 * *tensor_id receives the input's tensor id.
 * Errors: IOS_E_ARG (non-positive size, NULL), IOS_E_STATE (after finalize). */
int ios_add_input(ios_graph *g, int32_t c, int32_t h, int32_t w, int32_t *tensor_id);

/* Append one operator reading tensors in_ids[0 .. n_in-1] (already existing,
 * so insertion order is topological, Sec. 3).  Its output tensor id is
 * written to *out_tensor_id; for a schedule unit (every kind but CONCAT and
 * IDENTITY) that id also names the unit in schedules and cost callbacks.
 *   CONV     n_in = 1; weights [cout][cin][kh][kw]; bias [cout] or NULL (zero).
 *   SEPCONV  n_in >= 1 inputs of equal shape, summed; weights = depthwise
 *            [cin][1][kh][kw] followed by pointwise [cout][cin][1][1];
 *            bias [cout] or NULL; stride 1, pad (kh/2, kw/2) expected.
 *   POOL_*   n_in = 1; no weights.
 *   ADD/MEAN n_in >= 1 inputs of equal shape; no weights.
 *   CONCAT   n_in >= 1 inputs of equal batch/h/w; each must be a schedule
 *            unit's output (or a concat of them) not already in a concat.
 *   IDENTITY n_in = 1.
 * At most 16 inputs.  Weights are copied.
 * Errors: IOS_E_ARG, IOS_E_SHAPE, IOS_E_UNSUPPORTED, IOS_E_STATE. */
int ios_add_op(ios_graph *g, const ios_op_desc *d, const int32_t *in_ids, int32_t n_in,
               const float *weights, const float *bias, int32_t *out_tensor_id);

/* Mark a tensor as graph output number k (k = 0, 1, ... in call order).  It
 * must be a whole buffer: a unit output or a concat view that is not itself a
 * slice of a larger concat, and not a graph input.
 * Errors: IOS_E_ARG, IOS_E_UNSUPPORTED, IOS_E_STATE. */
int ios_mark_output(ios_graph *g, int32_t tensor_id);

/* Freeze the graph: assign blocks, plan concat slices, allocate device
 * intermediates, pack and upload weights.  Must be called once, before any
 * profile / schedule / run call.  Blocks (Sec. 4.2, optimising each block of a
 * stacked CNN separately): if every unit has block_id -1, all units form
 * block 0 when there are at most 64 of them, otherwise the units are cut
 * before every unit that is an ancestor or descendant of every other unit;
 * if any unit names a block, all must, a unit's block must not be lower than
 * its producers', and blocks run in ascending id.  A block holds at most 64
 * units.  Uses the current HIP device.
 * Errors: IOS_E_TOO_MANY_OPS, IOS_E_BAD_STAGE, IOS_E_OOM, IOS_E_HIP, IOS_E_STATE. */
int ios_graph_finalize(ios_graph *g);

/* Number of blocks, and the unit ids of block b in ascending order: bit i of a
 * block-local stage mask is unit_ids[i].  unit_ids must hold 64 entries.
 * Errors: IOS_E_ARG, IOS_E_STATE. */
int ios_graph_blocks(const ios_graph *g, int32_t *n_blocks);
int ios_block_units(const ios_graph *g, int32_t block, int32_t *n, int32_t *unit_ids);

/* Parallelization strategies of a stage (Sec. 3). */
enum { IOS_CONCURRENT = 0, IOS_MERGE = 1 };

/* Whether the units can form one operator-merge stage: at least two dense
 * convs reading the same tensor with equal stride and ReLU flags, each kernel
 * centring in the largest with the same resulting padding (Sec. 3).
 * *ok receives 1 or 0.  Errors: IOS_E_ARG, IOS_E_STATE. */
int ios_stage_mergeable(ios_graph *g, const int32_t *unit_ids, int32_t n, int32_t *ok);

/* Measure one stage on the device, as GenerateStage does (Sec. 4.1,
 * Algorithm 1): the stage's single grouped kernel is launched `warmup` times,
 * then `repeats` times `reps` back-to-back launches between two HIP events on
 * the library's stream; *latency_ns receives the median per-launch time,
 * rounded to ns.  Uses the graph's own buffers (inputs hold zeros), not the
 * caller's.  Units must lie in one block and be closed under the stage rule:
 * a unit's producers inside the block are either in the stage or scheduled
 * before it.  strategy IOS_MERGE requires ios_stage_mergeable.
 * Blocks the calling thread until the timing is done.
 * Errors: IOS_E_ARG, IOS_E_BAD_STAGE, IOS_E_NOT_MERGEABLE, IOS_E_HIP, IOS_E_STATE. */
int ios_profile_stage(ios_graph *g, const int32_t *unit_ids, int32_t n, int32_t strategy,
                      int32_t warmup, int32_t reps, int32_t repeats, int64_t *latency_ns);

/* Tile shape of a conv unit (unit_ids as in ios_block_units): after the
 * graph is finalized, the first call that touches the device measures every
 * conv alone with each shape and keeps one; these calls read that choice or
 * replace it, e.g. to replay the shapes of an earlier run.  Shapes are
 * 0 .. IOS_CONV_TILE_SHAPES - 1 (16x16, 16x32, 32x32, 32x64, 64x64 and
 * 128x64 output pixels x channels, operands loaded per wave; then 128x64,
 * 256x32 and 64x128 with both operands staged in LDS by a pipeline of
 * direct loads shared by the workgroup, and the same three shapes with a
 * private pipeline per wave, for large convolutions whose input channels are a multiple
 * of 16, with at most 32 taps and no input ReLU; a merge stage whose
 * merged window has more taps falls back to 16x32).  A new shape applies to stages compiled
 * afterwards (ios_profile_stage, ios_schedule, ios_schedule_from_stages),
 * not to schedules that already exist.  Both calls set up the device first
 * (hence the measurement) if no earlier call has.
 * Errors: IOS_E_ARG (not a conv unit, shape out of range or a pipelined
 * shape the conv does not admit, null pointer), IOS_E_STATE (not
 * finalized), IOS_E_HIP. */
enum { IOS_CONV_TILE_SHAPES = 12 };
int ios_get_conv_tile(ios_graph *g, int32_t unit_id, int32_t *shape);
int ios_set_conv_tile(ios_graph *g, int32_t unit_id, int32_t shape);

/* Every tuning choice of one unit, so that a tuned schedule can be replayed
 * exactly: `tile` is a CONV's tile shape (as above) or a SEPCONV's tile
 * choice (0, 1, 2: runs of 16, 32 or 64 consecutive output pixels with
 * every output channel, input rows staged in LDS; 3 .. 6: 16 pixels of one
 * output row with 1 .. 4 blocks of 16 output channels, for at most 256
 * input channels and windows up to 5 x 5; 7, 8: whole output rows in 128
 * or 64 MFMA columns x 64 or 128 output channels, for one input and a
 * 3 x 3 or 5 x 5 window that keeps the plane size; 9, 10: 32 / W whole
 * output rows x 32 or 64 output channels, with 16-byte loads, for a 3 x 3
 * window that keeps the plane size, rows of a multiple of 4 up to 32 floats
 * and at most 96 input channels), 0 for the other kinds;
 * `xcd_lg` is log2 of the run of consecutive tiles a stage holding the
 * unit sends to one XCD (0, 2 or 4), or -1 to let the library's L2-fill
 * model choose (ios_schedule_tune_tiles sets both per stage).  A stage whose
 * units disagree on xcd_lg uses the model.  These are implementation
 * choices of this library's stage kernel, not part of the paper's method;
 * like ios_set_conv_tile they apply to stages compiled afterwards, and both
 * calls set up the device first if no earlier call has.
 * Errors: IOS_E_ARG (bad unit, value out of range, null pointer),
 * IOS_E_STATE, IOS_E_HIP. */
int ios_get_unit_tiling(ios_graph *g, int32_t unit_id, int32_t *tile, int32_t *xcd_lg);
int ios_set_unit_tiling(ios_graph *g, int32_t unit_id, int32_t tile, int32_t xcd_lg);

/* Cost provider for the dynamic program: latency of stage `stage_mask`
 * (block-local bits, see ios_block_units; unit_ids lists the same units,
 * ascending) of block `block` under `strategy`.  Write a latency in ns, or
 * INT64_MAX for "impossible", to *latency_ns and return 0; any other return
 * aborts ios_schedule with IOS_E_COST_FN.  Never called with IOS_MERGE for a
 * set that cannot merge. */
typedef int (*ios_cost_fn)(void *ctx, int32_t block, uint64_t stage_mask,
                           const int32_t *unit_ids, int32_t n, int32_t strategy,
                           int64_t *latency_ns);

enum { IOS_SCHED_DP = 0, IOS_SCHED_SEQUENTIAL = 1, IOS_SCHED_GREEDY = 2 };

typedef struct {
  int32_t mode;        /* IOS_SCHED_DP (Algorithm 1), SEQUENTIAL (one unit per
                          stage, ascending id), GREEDY (every ready unit in the
                          next stage, concurrent) — Sec. 6.1 baselines        */
  int32_t r;           /* pruning: max units per group; <= 0 = unlimited     */
  int32_t s;           /* pruning: max groups per stage; <= 0 = unlimited    */
  int32_t strategies;  /* bit 0 concurrent, bit 1 merge: 3 = IOS-Both,
                          1 = IOS-Parallel, 2 = IOS-Merge (Sec. 6.1)         */
  int32_t warmup, reps, repeats;   /* profiler settings when fn is NULL     */
  int32_t verify_reps; /* DP with fn NULL, > 0: after a block's search the
                          stages of its schedule are measured again (3 warm-up
                          launches, 3 repeats of verify_reps launches), their
                          table entries replaced, and the search repeated on
                          the updated table until every stage it picks has been
                          measured that way (at most 16 rounds).  Guards a
                          search run with few launches per candidate against
                          stages whose short measurement came out low; the
                          result is optimal for the final table.  0 = off    */
} ios_sched_opts;

/* Fill opts with the paper's defaults: DP, r = 3, s = 8 (Sec. 5), both
 * strategies, warmup 3, reps 20, repeats 3, no verification rounds. */
void ios_sched_opts_default(ios_sched_opts *opts);

/* Find a schedule (Algorithm 1, block by block).  With fn == NULL each
 * candidate stage is measured with ios_profile_stage (a concurrent stage
 * holding two or more SEPCONVs that admit the GEMM SEPCONV tile is measured
 * also with them on it, likewise on the 64-channel line tile, and the fastest
 * figure counts, unless IOS_SEP_TILE fixes the tile choices); otherwise fn(ctx, ...) supplies latencies.  Ties: a stage keeps concurrent execution only if it is
 * strictly faster than merge; among equal-cost endings the smallest
 * block-local mask wins.  *out receives a schedule owned by the caller (free
 * with ios_schedule_destroy) and *cost_ns the minimised sum of stage
 * latencies (SEQUENTIAL / GREEDY: the sum under the same cost provider).
 * Errors: IOS_E_ARG, IOS_E_STATE, IOS_E_COST_FN, IOS_E_HIP, IOS_E_OOM. */
int ios_schedule(ios_graph *g, const ios_sched_opts *opts, ios_cost_fn fn, void *ctx,
                 ios_schedule_t **out, int64_t *cost_ns);

/* Build a schedule from an explicit stage list: stage k holds
 * unit_ids[stage_offsets[k] .. stage_offsets[k+1]-1] with strategy
 * strategies[k].  Every unit must appear once; each stage must lie in one
 * block, blocks must appear in ascending order, a unit's producers must be
 * in earlier stages or in the same stage (concurrent only), and merge stages
 * must be mergeable.  Errors: IOS_E_ARG, IOS_E_BAD_STAGE, IOS_E_NOT_MERGEABLE. */
int ios_schedule_from_stages(ios_graph *g, int32_t n_stages, const int32_t *stage_offsets,
                             const int32_t *unit_ids, const int32_t *strategies,
                             ios_schedule_t **out);

/* Read a schedule Q = [(S_1, T_1), ..., (S_k, T_k)] (Sec. 3, "Schedule"):
 * stages in execution order, unit ids ascending inside a stage.  The arrays
 * belong to the schedule and live until ios_schedule_destroy. */
int ios_schedule_get(const ios_schedule_t *q, int32_t *n_stages, const int32_t **stage_offsets,
                     const int32_t **unit_ids, const int32_t **strategies);

/* Search statistics of a DP schedule: distinct states S visited (the empty
 * set included), (S, S') transitions evaluated (Sec. 4.2) and distinct
 * stages S' whose latency was requested.  Zero for other schedules. */
int ios_schedule_stats(const ios_schedule_t *q, int64_t *states, int64_t *transitions,
                       int64_t *stages_measured);

/* Choose conv tile shapes and tile order per stage of q.  The stage profiler
 * of Sec. 4.1 measures a whole stage; this call uses the same measurement
 * (o's warmup / reps / repeats, or the defaults when o is NULL) to pick, for
 * every stage, (1) how its tiles are spread over the 8 XCDs (runs of 1, 4 or
 * 16 consecutive tiles per XCD, else the library's L2-fill model) and (2) the
 * tile shapes of its convs and the tile choices of its SEPCONVs in that
 * stage's company: in a concurrent stage first all its convs (all its
 * SEPCONVs) moved to one value together, then one operator at a time, each
 * value tried, a change kept when the stage gets more than 2% faster (two
 * passes); a merge stage's convs take one shape together.  The choices stay
 * set on the graph's units (ios_get_conv_tile reads the shapes), so call it
 * on the schedule that will run; q's stages are recompiled on its next run.
 * A unit belongs to one stage of a schedule, so the stages do not compete.
 * With IOS_CONV_TILE (IOS_SEP_TILE) set in the environment the conv shapes
 * (SEPCONV tile choices) stay fixed, the rest is still chosen; IOS_XCD_RUNS=0, 2 or 4 fixes the tile order's run
 * length (2^value) for every stage compiled while it is set, for tests.  *cost_ns = sum of the stages' final measured
 * latencies.
 * Errors: IOS_E_ARG (null pointer, bad counts, schedule of another graph),
 * IOS_E_STATE (not finalized), IOS_E_HIP. */
int ios_schedule_tune_tiles(ios_graph *g, ios_schedule_t *q, const ios_sched_opts *o,
                            int64_t *cost_ns);

void ios_schedule_destroy(ios_schedule_t *q);

/* Write the stage-latency table of the graph's last ios_schedule call as JSON
 * lines {"block", "mask", "units", "concurrent_ns", "merge_ns" (null if not
 * measured)} to `path`, so that the search can be replayed.  These are the
 * latencies GenerateStage measures for each candidate stage S' under both
 * strategies (Sec. 4.1, Algorithm 1), the only input of the recurrence
 * besides the graph.
 * Errors: IOS_E_ARG, IOS_E_STATE (no table). */
int ios_schedule_dump_costs(const ios_graph *g, const char *path);

/* Execute graph g under schedule q: the stages run one after another, in
 * schedule order, each with its own parallelization strategy (Sec. 3,
 * "Schedule": Q = [(S_1, T_1), ..., (S_k, T_k)], stage i+1 starts after
 * stage i ends), as one kernel launch per stage on `hip_stream` (a
 * hipStream_t; NULL = the default stream).
 * d_inputs[i] points to input i, d_outputs[k] to output k, each a device
 * buffer of the declared shape owned by the caller.  Asynchronous: returns
 * after the launches are queued, without synchronising.  Runs of one schedule
 * must not overlap in time (they share per-stage counters), so issue them on
 * one stream.  Errors: IOS_E_ARG, IOS_E_STATE, IOS_E_HIP. */
int ios_run(ios_graph *g, ios_schedule_t *q, const float *const *d_inputs,
            float *const *d_outputs, void *hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): ios_run
 * with no allocation of any kind.  The intermediate activations between
 * stages and the in-stage counters, which ios_run keeps in memory the graph
 * and the schedule allocated, live here in one fixed device array of 64 MiB
 * per device, which the library holds until the process ends; the caller
 * still passes the inputs and outputs, as for ios_run.  Preconditions: the
 * schedule has been run once with ios_run (which sets up the graph's device
 * side and compiles the stages), and the graph's intermediates fit the
 * array (8 KiB of counters, then each intermediate rounded up to 256 bytes).
 * Every call on one device shares that device's array and leaves its last
 * contents there: calls that overlap in time on one device race, so issue
 * them on one stream.  Asynchronous, like ios_run.
 * Errors: IOS_E_ARG (null pointers, schedule of another graph), IOS_E_STATE
 * (preconditions), IOS_E_UNSUPPORTED (intermediates larger than the array),
 * IOS_E_HIP. */
int ios_run_noalloc(ios_graph *g, const ios_schedule_t *q, const float *const *d_inputs,
                    float *const *d_outputs, void *hip_stream);

/* As ios_run, then records a HIP event before and after every stage launch,
 * waits for the stream, and writes each stage's GPU time in ns to
 * stage_ns[0 .. n_stages-1].  For per-stage measurement; blocks the caller. */
int ios_run_timed(ios_graph *g, ios_schedule_t *q, const float *const *d_inputs,
                  float *const *d_outputs, void *hip_stream, int64_t *stage_ns);

/* Wait for `hip_stream` and read the graph's device error word: *flags
 * receives 0 if every stage kernel since the last call finished normally,
 * else a bit set (1 = an intra-stage dependency wait gave up).  Clears it.
 * Errors: IOS_E_ARG, IOS_E_HIP. */
int ios_device_status(ios_graph *g, void *hip_stream, int32_t *flags);

/* Message describing the calling thread's most recent error. */
const char *ios_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* IOS_H_ */
