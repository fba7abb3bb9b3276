// Graph IR of libios: tensors, schedule units, views, blocks and the device
// copies of weights (Sec. 3 "Computation Graph"; Sec. 4.2 block-wise
// optimisation).
#include <algorithm>
#include <chrono>
#include <cstdlib>
#include <cstring>
#include <functional>

#include "ios_internal.h"

namespace ios {

void fail(int code, const std::string &msg) { throw Error{code, msg}; }

void hip_check(hipError_t e, const char *what) {
  if (e != hipSuccess)
    fail(e == hipErrorOutOfMemory ? IOS_E_OOM : IOS_E_HIP,
         std::string(what) + ": " + hipGetErrorString(e));
}

static bool is_unit_kind(int k) { return k >= IOS_CONV && k <= IOS_MEAN; }

int unit_op_of_tensor(const ios_graph *g, int tid) {
  if (tid < 0 || tid >= (int)g->tensors.size()) fail(IOS_E_ARG, "unit id out of range");
  const Tensor &t = g->tensors[tid];
  if (t.kind != T_UNIT) fail(IOS_E_ARG, "tensor " + std::to_string(tid) + " is not a unit output");
  return t.op;
}

// Schedule units whose outputs a tensor carries (views resolved).
std::vector<int> unit_producers(const ios_graph *g, int tid) {
  const Tensor &t = g->tensors[tid];
  if (t.kind == T_INPUT) return {};
  if (t.kind == T_UNIT) return {t.op};
  std::vector<int> out;
  for (int i : g->ops[t.op].in) {
    auto p = unit_producers(g, i);
    out.insert(out.end(), p.begin(), p.end());
  }
  return out;
}

int64_t op_flops(const ios_graph *g, const Op &op) {
  int64_t n = g->batch;
  switch (op.d.kind) {
    case IOS_CONV:
      return 2 * n * op.ho * op.wo * (int64_t)op.d.cout * op.cin * op.d.kh * op.d.kw;
    case IOS_SEPCONV:
      return 2 * n * op.ho * op.wo * (int64_t)op.cin * (op.d.kh * op.d.kw + op.d.cout);
    case IOS_POOL_MAX:
    case IOS_POOL_AVG:
      return n * op.ho * op.wo * (int64_t)op.cin * op.d.kh * op.d.kw;
    default:
      return n * op.ho * op.wo * (int64_t)op.cin * (int64_t)op.in.size();
  }
}

// ---------------------------------------------------------------- building

static int new_tensor(ios_graph *g, int c, int h, int w, int kind, int op) {
  Tensor t;
  t.c = c; t.h = h; t.w = w; t.kind = kind; t.op = op;
  g->tensors.push_back(t);
  return (int)g->tensors.size() - 1;
}

int add_input(ios_graph *g, int c, int h, int w) {
  if (g->finalized) fail(IOS_E_STATE, "graph already finalized");
  if (c <= 0 || h <= 0 || w <= 0) fail(IOS_E_ARG, "input sizes must be positive");
  int id = new_tensor(g, c, h, w, T_INPUT, -1);
  g->tensors[id].input_index = (int)g->inputs.size();
  g->inputs.push_back(id);
  return id;
}

static int out_size(int in, int k, int s, int p) { return (in + 2 * p - k) / s + 1; }

int add_op(ios_graph *g, const ios_op_desc *d, const int32_t *in_ids, int n_in,
           const float *weights, const float *bias) {
  if (g->finalized) fail(IOS_E_STATE, "graph already finalized");
  if (!d) fail(IOS_E_ARG, "null op descriptor");
  if (n_in < 1 || n_in > kMaxIn) fail(IOS_E_ARG, "an operator takes 1..16 inputs");
  if (!in_ids) fail(IOS_E_ARG, "null input list");
  for (int i = 0; i < n_in; ++i)
    if (in_ids[i] < 0 || in_ids[i] >= (int)g->tensors.size())
      fail(IOS_E_ARG, "input tensor id out of range");
  Op op;
  op.d = *d;
  op.in.assign(in_ids, in_ids + n_in);
  const Tensor &t0 = g->tensors[in_ids[0]];
  op.cin = t0.c; op.h = t0.h; op.wd = t0.w;
  int kind = d->kind;
  int oc = t0.c, oh = t0.h, ow = t0.w;
  auto same_shape = [&]() {
    for (int i = 1; i < n_in; ++i) {
      const Tensor &t = g->tensors[in_ids[i]];
      if (t.c != t0.c || t.h != t0.h || t.w != t0.w) fail(IOS_E_SHAPE, "inputs differ in shape");
    }
  };
  switch (kind) {
    case IOS_CONV:
    case IOS_SEPCONV:
    case IOS_POOL_MAX:
    case IOS_POOL_AVG: {
      if (kind != IOS_SEPCONV && n_in != 1) fail(IOS_E_ARG, "this operator takes one input");
      if (kind == IOS_SEPCONV) same_shape();
      if (d->kh < 1 || d->kw < 1 || d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 ||
          d->pad_w < 0)
        fail(IOS_E_ARG, "bad kernel / stride / padding");
      if (kind == IOS_SEPCONV && (d->stride_h != 1 || d->stride_w != 1))
        fail(IOS_E_UNSUPPORTED, "SEPCONV needs stride 1");
      if (kind == IOS_CONV && (d->kh > 16 || d->kw > 16))
        fail(IOS_E_UNSUPPORTED, "conv windows larger than 16x16");
      if (kind == IOS_POOL_MAX && (d->pad_h >= d->kh || d->pad_w >= d->kw))
        fail(IOS_E_ARG, "max-pool padding must be smaller than the window");
      oh = out_size(t0.h, d->kh, d->stride_h, d->pad_h);
      ow = out_size(t0.w, d->kw, d->stride_w, d->pad_w);
      if (oh < 1 || ow < 1) fail(IOS_E_SHAPE, "window larger than the padded input");
      if (kind == IOS_CONV || kind == IOS_SEPCONV) {
        if (d->cout < 1) fail(IOS_E_ARG, "cout must be positive");
        if (!weights) fail(IOS_E_ARG, "weights required");
        oc = d->cout;
        size_t nw = kind == IOS_CONV
                        ? (size_t)d->cout * t0.c * d->kh * d->kw
                        : (size_t)t0.c * d->kh * d->kw + (size_t)d->cout * t0.c;
        op.w.assign(weights, weights + nw);
        op.b.assign((size_t)d->cout, 0.f);
        if (bias) std::memcpy(op.b.data(), bias, sizeof(float) * d->cout);
        if (kind == IOS_SEPCONV && (d->kh > kSepMaxWindow || d->kw > kSepMaxWindow))
          fail(IOS_E_UNSUPPORTED, "SEPCONV depthwise window larger than 7x7");
        if (kind == IOS_SEPCONV && sep_geometry(0, t0.c, d->cout, t0.w, oh, ow, d->kh, d->kw).bm == 0)
          fail(IOS_E_UNSUPPORTED, "SEPCONV input rows too wide for the staged tile");
        // (the row tile is an alternative where it applies, never the only one)
      }
      break;
    }
    case IOS_ADD:
    case IOS_MEAN:
      same_shape();
      break;
    case IOS_CONCAT: {
      oc = 0;
      for (int i = 0; i < n_in; ++i) {
        const Tensor &t = g->tensors[in_ids[i]];
        if (t.h != t0.h || t.w != t0.w) fail(IOS_E_SHAPE, "concat inputs differ in size");
        if (t.kind != T_UNIT && t.kind != T_CONCAT)
          fail(IOS_E_UNSUPPORTED, "concat members must be unit outputs or concats");
        if (t.parent >= 0) fail(IOS_E_UNSUPPORTED, "tensor already placed in a concat");
        for (int j = 0; j < i; ++j)
          if (in_ids[j] == in_ids[i]) fail(IOS_E_UNSUPPORTED, "tensor repeated in a concat");
        oc += t.c;
      }
      break;
    }
    case IOS_IDENTITY:
      if (n_in != 1) fail(IOS_E_ARG, "identity takes one input");
      break;
    default:
      fail(IOS_E_ARG, "unknown operator kind");
  }
  op.ho = oh; op.wo = ow;
  int op_idx = (int)g->ops.size();
  int tkind = is_unit_kind(kind) ? T_UNIT : (kind == IOS_CONCAT ? T_CONCAT : T_IDENTITY);
  int tid = new_tensor(g, oc, oh, ow, tkind, op_idx);
  op.out = tid;
  if (is_unit_kind(kind)) {
    op.unit = (int)g->units.size();
    g->units.push_back(op_idx);
  }
  if (kind == IOS_CONCAT) {
    int off = 0;
    for (int i = 0; i < n_in; ++i) {
      Tensor &m = g->tensors[in_ids[i]];
      m.parent = tid;
      m.parent_off = off;
      off += m.c;
    }
  }
  g->ops.push_back(std::move(op));
  return tid;
}

void mark_output(ios_graph *g, int tid) {
  if (g->finalized) fail(IOS_E_STATE, "graph already finalized");
  if (tid < 0 || tid >= (int)g->tensors.size()) fail(IOS_E_ARG, "tensor id out of range");
  int t = tid;
  while (g->tensors[t].kind == T_IDENTITY) t = g->ops[g->tensors[t].op].in[0];
  const Tensor &r = g->tensors[t];
  if (r.kind == T_INPUT) fail(IOS_E_UNSUPPORTED, "a graph input cannot be an output");
  if (r.parent >= 0) fail(IOS_E_UNSUPPORTED, "an output must not be a slice of a concat");
  for (int o : g->outputs) {
    int u = o;
    while (g->tensors[u].kind == T_IDENTITY) u = g->ops[g->tensors[u].op].in[0];
    if (u == t) fail(IOS_E_UNSUPPORTED, "tensor already marked as an output");
  }
  g->outputs.push_back(tid);
}

// ---------------------------------------------------------------- blocks

static void assign_blocks(ios_graph *g) {
  int nu = (int)g->units.size();
  if (nu == 0) fail(IOS_E_BAD_STAGE, "graph has no schedule units");
  // unit-level adjacency (global)
  std::vector<std::vector<int>> succ(nu), pred(nu);
  for (int v = 0; v < nu; ++v) {
    const Op &op = g->ops[g->units[v]];
    for (int t : op.in)
      for (int p : unit_producers(g, t)) {
        int u = g->ops[p].unit;
        if (std::find(succ[u].begin(), succ[u].end(), v) == succ[u].end()) {
          succ[u].push_back(v);
          pred[v].push_back(u);
        }
      }
  }
  std::vector<int> bid(nu);
  int explicit_n = 0;
  for (int v = 0; v < nu; ++v) explicit_n += g->ops[g->units[v]].d.block_id >= 0;
  if (explicit_n != 0 && explicit_n != nu)
    fail(IOS_E_BAD_STAGE, "either every unit names a block or none does");
  if (explicit_n == nu) {
    std::vector<int> ids;
    for (int v = 0; v < nu; ++v) ids.push_back(g->ops[g->units[v]].d.block_id);
    std::vector<int> sorted = ids;
    std::sort(sorted.begin(), sorted.end());
    sorted.erase(std::unique(sorted.begin(), sorted.end()), sorted.end());
    for (int v = 0; v < nu; ++v)
      bid[v] = (int)(std::lower_bound(sorted.begin(), sorted.end(), ids[v]) - sorted.begin());
    for (int v = 0; v < nu; ++v)
      for (int u : pred[v])
        if (bid[u] > bid[v]) fail(IOS_E_BAD_STAGE, "a unit's block precedes its producer's");
  } else if (nu <= kMaxUnitsPerBlock) {
    std::fill(bid.begin(), bid.end(), 0);
  } else {
    // cut before every unit comparable with all others
    std::vector<std::vector<char>> anc(nu, std::vector<char>(nu, 0));
    for (int v = 0; v < nu; ++v)
      for (int u : pred[v]) {
        anc[v][u] = 1;
        for (int w = 0; w < nu; ++w) anc[v][w] |= anc[u][w];
      }
    int b = 0;
    for (int v = 0; v < nu; ++v) {
      bool cut = v > 0;
      for (int w = 0; w < nu && cut; ++w)
        if (w != v && !anc[v][w] && !anc[w][v]) cut = false;
      if (cut) ++b;
      bid[v] = b;
    }
  }
  int nb = *std::max_element(bid.begin(), bid.end()) + 1;
  g->blocks.assign(nb, Block{});
  for (int v = 0; v < nu; ++v) {
    Block &B = g->blocks[bid[v]];
    if ((int)B.ops.size() >= kMaxUnitsPerBlock)
      fail(IOS_E_TOO_MANY_OPS, "more than 64 schedule units in one block");
    Op &op = g->ops[g->units[v]];
    op.block = bid[v];
    op.local = (int)B.ops.size();
    B.ops.push_back(g->units[v]);
  }
  for (auto &B : g->blocks) {
    B.succ.assign(B.ops.size(), 0);
    B.pred.assign(B.ops.size(), 0);
  }
  for (int v = 0; v < nu; ++v)
    for (int u : succ[v]) {
      const Op &a = g->ops[g->units[v]], &c = g->ops[g->units[u]];
      if (a.block == c.block) {
        g->blocks[a.block].succ[a.local] |= 1ull << c.local;
        g->blocks[a.block].pred[c.local] |= 1ull << a.local;
      }
    }
}

// ---------------------------------------------------------------- merge rule

static int resolve_identity(const ios_graph *g, int t) {
  while (g->tensors[t].kind == T_IDENTITY) t = g->ops[g->tensors[t].op].in[0];
  return t;
}

bool stage_mergeable(const ios_graph *g, const std::vector<int> &ops) {
  if (ops.size() < 2) return false;
  const Op &o0 = g->ops[ops[0]];
  int KH = 0, KW = 0;
  for (int i : ops) {
    const Op &o = g->ops[i];
    if (o.d.kind != IOS_CONV) return false;
    if (resolve_identity(g, o.in[0]) != resolve_identity(g, o0.in[0])) return false;
    if (o.d.stride_h != o0.d.stride_h || o.d.stride_w != o0.d.stride_w ||
        o.d.pre_relu != o0.d.pre_relu || o.d.post_relu != o0.d.post_relu)
      return false;
    KH = std::max(KH, o.d.kh);
    KW = std::max(KW, o.d.kw);
  }
  int ph = -1, pw = -1;
  for (int i : ops) {
    const Op &o = g->ops[i];
    if ((KH - o.d.kh) % 2 || (KW - o.d.kw) % 2) return false;
    int a = o.d.pad_h + (KH - o.d.kh) / 2, b = o.d.pad_w + (KW - o.d.kw) / 2;
    if (ph < 0) { ph = a; pw = b; }
    if (a != ph || b != pw) return false;
  }
  return true;
}

// ---------------------------------------------------------------- finalize

static void resolve_buffers(ios_graph *g) {
  // every root tensor (unit output or concat with no parent) owns a buffer
  std::function<void(int)> place = [&](int t) {
    Tensor &T = g->tensors[t];
    if (T.buf >= 0) return;
    if (T.kind == T_INPUT) {
      Buffer b;
      b.ctot = T.c; b.h = T.h; b.w = T.w; b.input_index = T.input_index;
      g->bufs.push_back(b);
      T.buf = (int)g->bufs.size() - 1;
      T.coff = 0;
    } else if (T.kind == T_IDENTITY) {
      int s = g->ops[T.op].in[0];
      place(s);
      T.buf = g->tensors[s].buf;
      T.coff = g->tensors[s].coff;
    } else if (T.parent >= 0) {
      place(T.parent);
      T.buf = g->tensors[T.parent].buf;
      T.coff = g->tensors[T.parent].coff + T.parent_off;
    } else {
      Buffer b;
      b.ctot = T.c; b.h = T.h; b.w = T.w;
      g->bufs.push_back(b);
      T.buf = (int)g->bufs.size() - 1;
      T.coff = 0;
    }
  };
  for (int t = 0; t < (int)g->tensors.size(); ++t) place(t);
  for (int k = 0; k < (int)g->outputs.size(); ++k) {
    int t = resolve_identity(g, g->outputs[k]);
    g->bufs[g->tensors[t].buf].output_index = k;
  }
}

static int round_up(int a, int b) { return (a + b - 1) / b * b; }

template <class T>
static T *upload(const std::vector<T> &v) {
  T *p = nullptr;
  hip_check(hipMalloc(&p, sizeof(T) * std::max<size_t>(v.size(), 1)), "hipMalloc(weights)");
  hip_check(hipMemcpy(p, v.data(), sizeof(T) * v.size(), hipMemcpyHostToDevice), "hipMemcpy");
  return p;
}

bool conv_tile_ok(const Op &op, int cfg) {
  return cfg >= 0 && cfg < TC_COUNT &&
         (!tile_is_pipe(cfg) || pipe_conv_ok(op.cin, op.d.kh * op.d.kw, op.d.pre_relu));
}

bool sep_tile_ok(const Op &op, int tile) {
  if (tile < 0 || tile >= kSepTiles) return false;
  if (tile >= kSepLineFirst)
    return line_geometry(1 << (tile - kSepLineFirst), op.cin, op.d.cout, op.d.kh, op.d.kw, op.d.pad_h, op.d.pad_w,
                         op.d.stride_h, op.d.stride_w, op.h, op.wd, op.ho, op.wo).r != 0;
  if (tile >= kSepgFirst)
    return sepg_geometry(tile - kSepgFirst, (int)op.in.size(), op.d.kh, op.d.kw, op.d.pad_h, op.d.pad_w, op.h,
                         op.wd, op.ho, op.wo).bm != 0;
  if (tile < kSepStagedTiles)
    return sep_geometry(tile, op.cin, op.d.cout, op.wd, op.ho, op.wo, op.d.kh, op.d.kw).bm == (16 << tile);
  const int K = sep_row_window(op.d.kh, op.d.kw), nbt = tile - kSepStagedTiles + 1;
  return K != 0 && op.cin <= kSepRowMaxChannels && nbt <= round_up(op.d.cout, 16) / 16 &&
         sep_row_lds_bytes(round_up(op.cin, 4), K, nbt) <= kSepMaxLds;
}

// SEPCONV tile choice before measurement (IOS_SEP_TILE=<0..10> forces one;
// a choice the operator cannot use falls back to the staged tile of 16
// pixels).
static int choose_sep_tile(const Op &op) {
  int v = 1;
  if (const char *e = std::getenv("IOS_SEP_TILE")) v = std::atoi(e);
  v = std::max(0, std::min(v, kSepTiles - 1));
  return sep_tile_ok(op, v) ? v : 0;
}

// Conv tile shape for an M x N output before measurement.  IOS_CONV_TILE=<0..8>
// in the environment (read when a graph is finalized or a merged stage is
// built) forces one shape for every conv, for tuning and for tests; a
// pipelined shape is forced only on convs it applies to (pipe_ok).
// Tuning: warm-up time before the first measurement, and the fraction of the
// fastest time within which a conv tile shape with fewer workgroups is taken.
constexpr int kTuneWarmMs = 50;
constexpr double kTuneSlack = 0.03;

int choose_conv_tile(int64_t M, int N, bool pipe_ok) {
  if (const char *e = std::getenv("IOS_CONV_TILE")) {
    int v = std::atoi(e);
    if (v >= 0 && v < TC_COUNT && (pipe_ok || !tile_is_pipe(v))) return v;
  }
  int64_t t64 = ((M + 63) / 64) * ((N + 63) / 64);
  int64_t t32 = ((M + 31) / 32) * ((N + 31) / 32);
  if (t64 >= 2048) return TC_128x64;
  if (t64 >= 512) return TC_64x64_K2;
  if (t32 >= 256) return TC_32x32_K8;
  return TC_16x32_K8;
}

void finalize_graph(ios_graph *g) {
  if (g->finalized) fail(IOS_E_STATE, "graph already finalized");
  assign_blocks(g);
  resolve_buffers(g);
  for (const auto &b : g->bufs)
    if (b.elems(g->batch) * sizeof(float) >= (size_t)1 << 30)
      fail(IOS_E_UNSUPPORTED, "tensor of 1 GiB or more");
  for (int oi : g->units) {
    Op &op = g->ops[oi];
    if (op.d.kind == IOS_CONV) {
      op.CinP = round_up(op.cin, 4);
      op.Npad = round_up(op.d.cout, 16);
      op.tcfg = choose_conv_tile((int64_t)g->batch * op.ho * op.wo, op.d.cout,
                                 pipe_conv_ok(op.cin, op.d.kh * op.d.kw, op.d.pre_relu));
    } else if (op.d.kind == IOS_SEPCONV) {
      op.CinP = round_up(op.cin, 16);
      op.Npad = round_up(op.d.cout, 16);
      op.sep_tile = choose_sep_tile(op);
    }
  }
  g->cost_table.assign(g->blocks.size(), {});
  g->finalized = true;
}

// Device side of a finalized graph, set up on the first call that needs the
// GPU: activation buffers (zero-filled), packed weights, stream, events.
void ensure_device(ios_graph *g) {
  if (!g->finalized) fail(IOS_E_STATE, "graph not finalized");
  if (g->device_ready) {
    hip_check(hipSetDevice(g->device), "hipSetDevice");
    return;
  }
  hip_check(hipGetDevice(&g->device), "hipGetDevice");
  hip_check(hipStreamCreateWithFlags(&g->stream, hipStreamNonBlocking), "hipStreamCreate");
  hip_check(hipEventCreate(&g->ev0), "hipEventCreate");
  hip_check(hipEventCreate(&g->ev1), "hipEventCreate");
  hip_check(hipMalloc(&g->d_err, sizeof(int32_t)), "hipMalloc(err)");
  hip_check(hipMemset(g->d_err, 0, sizeof(int32_t)), "hipMemset");
  for (auto &b : g->bufs) {
    size_t n = b.elems(g->batch);
    hip_check(hipMalloc(&b.dev, sizeof(float) * n), "hipMalloc(activation)");
    hip_check(hipMemset(b.dev, 0, sizeof(float) * n), "hipMemset");
  }
  for (int oi : g->units) {
    Op &op = g->ops[oi];
    if (op.d.kind == IOS_CONV) {
      std::vector<float> wpk, bias(op.Npad, 0.f);
      int nb = 0;
      pack_conv_weights(op.w.data(), op.d.cout, op.cin, op.d.kh, op.d.kw, wpk, &op.NG, &nb);
      std::copy(op.b.begin(), op.b.end(), bias.begin());
      op.d_wpk = upload(wpk);
      op.d_bias = upload(bias);
      std::vector<float> wg;
      pack_conv_pipe(op.w.data(), op.d.cout, op.cin, op.d.kh, op.d.kw, wg, &op.pipe_nkb);
      op.d_wg = upload(wg);
    } else if (op.d.kind == IOS_SEPCONV) {
      // depthwise [CinP][kh * kw] (channels past cin zero); pointwise packed
      // like a 1x1 conv's weights (groups of 4 k-steps = 16 input channels)
      const int taps = op.d.kh * op.d.kw;
      std::vector<float> dw((size_t)op.CinP * taps, 0.f);
      std::copy(op.w.begin(), op.w.begin() + (size_t)op.cin * taps, dw.begin());
      std::vector<float> pwk, bias(op.Npad, 0.f);
      int nb = 0;
      pack_conv_weights(op.w.data() + (size_t)op.cin * taps, op.d.cout, op.cin, 1, 1, pwk, &op.NG, &nb);
      std::copy(op.b.begin(), op.b.end(), bias.begin());
      op.d_dw = upload(dw);
      op.d_wpk = upload(pwk);
      op.d_bias = upload(bias);
      // the GEMM tile's pointwise layout: [round16(cin)][round128(cout)]
      if (sep_tile_ok(op, kSepgFirst) || sep_tile_ok(op, kSepgFirst + 1)) {
        std::vector<float> pwp;
        int nkb = 0;
        pack_conv_pipe(op.w.data() + (size_t)op.cin * taps, op.d.cout, op.cin, 1, 1, pwp, &nkb);
        op.d_pw_pipe = upload(pwp);
      }
      // the row tile's layouts, where it applies: depthwise taps at the top
      // left of a K x K window, [CinP4][kkp(K)]; pointwise [CinP4][Npad]
      const int K = sep_row_window(op.d.kh, op.d.kw);
      if (K != 0 && op.cin <= kSepRowMaxChannels) {
        const int cp4 = round_up(op.cin, 4), kkp = sep_kkp(K);
        std::vector<float> dwr((size_t)cp4 * kkp, 0.f), pwr((size_t)cp4 * op.Npad, 0.f);
        for (int c = 0; c < op.cin; ++c)
          for (int u = 0; u < op.d.kh; ++u)
            for (int v = 0; v < op.d.kw; ++v)
              dwr[(size_t)c * kkp + u * K + v] = op.w[(size_t)c * taps + u * op.d.kw + v];
        const float *pw = op.w.data() + (size_t)op.cin * taps;
        for (int co = 0; co < op.d.cout; ++co)
          for (int ci = 0; ci < op.cin; ++ci) pwr[(size_t)ci * op.Npad + co] = pw[(size_t)co * op.cin + ci];
        op.d_dw_row = upload(dwr);
        op.d_pw_row = upload(pwr);
      }
      // the line tile's pointwise layout, where it applies: the A operands of
      // v_mfma_f32_32x32x2_f32, [block of 32 output channels][k-step of 2
      // input channels][lane = 32 k + channel in the block]
      if (sep_tile_ok(op, kSepLineFirst)) {
        const int nblk = (op.d.cout + 31) / 32, nks = (op.cin + 1) / 2;
        const float *pw = op.w.data() + (size_t)op.cin * taps;
        std::vector<float> pwl((size_t)nblk * nks * 64, 0.f);
        for (int b = 0; b < nblk; ++b)
          for (int ks = 0; ks < nks; ++ks)
            for (int l = 0; l < 64; ++l) {
              const int co = b * 32 + (l & 31), ci = 2 * ks + (l >> 5);
              if (co < op.d.cout && ci < op.cin)
                pwl[((size_t)b * nks + ks) * 64 + l] = pw[(size_t)co * op.cin + ci];
            }
        op.d_pw_line = upload(pwl);
      }
    }
  }
  hip_check(hipDeviceSynchronize(), "hipDeviceSynchronize");
  // layout of the intermediates in ios_run_noalloc's scratch array: after
  // the counter block, each buffer that is neither an input nor an output
  // at a 256-byte boundary
  noalloc_setup(g->device);
  g->noalloc_off.assign(g->bufs.size(), 0);
  size_t off = noalloc_counter_bytes();
  for (size_t i = 0; i < g->bufs.size(); ++i) {
    const Buffer &b = g->bufs[i];
    if (b.input_index >= 0 || b.output_index >= 0) continue;
    g->noalloc_off[i] = off;
    off += (b.elems(g->batch) * sizeof(float) + 255) & ~(size_t)255;
  }
  g->noalloc_bytes = off;
  g->device_ready = true;
  const bool tune_conv = !std::getenv("IOS_CONV_TILE"), tune_sep = !std::getenv("IOS_SEP_TILE");
  if ((tune_conv || tune_sep) && !g->units.empty()) {
    // keep the GPU busy for a while first, so that the measurements below
    // are taken at the clocks the stages will run at
    const auto t0 = std::chrono::steady_clock::now();
    while (std::chrono::steady_clock::now() - t0 < std::chrono::milliseconds(kTuneWarmMs))
      profile_stage(g, {g->units[0]}, IOS_CONCURRENT, 0, 100, 1);
  }
  // Tile shape of every conv, chosen by measuring the conv alone with each
  // shape (unless IOS_CONV_TILE forces one).  Among the shapes within
  // kTuneSlack of the fastest the one with the fewest workgroups wins: a
  // stage runs the conv beside others, and fewer workgroups leave more room
  // for them.
  if (tune_conv) {
    for (int oi : g->units) {
      Op &op = g->ops[oi];
      if (op.d.kind != IOS_CONV) continue;
      const int64_t M = (int64_t)g->batch * op.ho * op.wo;
      std::vector<std::pair<int64_t, int>> meas;   // (ns, cfg)
      for (int cfg = 0; cfg < TC_COUNT; ++cfg) {
        if (!conv_tile_ok(op, cfg)) continue;
        op.tcfg = cfg;
        meas.push_back({profile_stage(g, {oi}, IOS_CONCURRENT, 3, 20, 5), cfg});
      }
      int64_t fastest = INT64_MAX;
      for (auto &m : meas) fastest = std::min(fastest, m.first);
      auto tiles = [&](int cfg) {
        return ((M + tile_bm(cfg) - 1) / tile_bm(cfg)) * ((op.d.cout + tile_bn(cfg) - 1) / tile_bn(cfg));
      };
      int best = -1;
      for (auto &m : meas)
        if (m.first <= fastest + (int64_t)(fastest * kTuneSlack) &&
            (best < 0 || tiles(m.second) < tiles(best)))
          best = m.second;
      op.tcfg = best;
    }
  }
  // SEPCONV tile choice, likewise measured (unless IOS_SEP_TILE forces it).
  if (tune_sep) {
    for (int oi : g->units) {
      Op &op = g->ops[oi];
      if (op.d.kind != IOS_SEPCONV) continue;
      int best = op.sep_tile;
      int64_t best_ns = INT64_MAX;
      for (int t = 0; t < kSepTiles; ++t) {
        if (!sep_tile_ok(op, t)) continue;
        op.sep_tile = t;
        int64_t ns = profile_stage(g, {oi}, IOS_CONCURRENT, 2, 10, 3);
        if (ns < best_ns) { best_ns = ns; best = t; }
      }
      op.sep_tile = best;
    }
  }
}

}  // namespace ios
