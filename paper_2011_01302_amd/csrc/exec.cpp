// Stage lowering, launching and on-device latency measurement.
//
// A stage (S', T) of the schedule (Sec. 3) becomes ONE kernel launch whose
// workgroups each run one tile taken from a table that spans every operator
// of the stage:
//   - concurrent execution: every unit keeps its own tiles; units of one
//     group that depend on each other run in order because a consumer tile
//     waits until all tiles of its producers have finished (Sec. 3, groups
//     are executed sequentially, different groups concurrently);
//   - operator merge: the convs' kernels are zero-padded (centred) to the
//     largest kernel and stacked along output channels; the input is read
//     once and each output-channel range is written straight to its own
//     op's buffer, which stands in for the split operator (Sec. 3).
// GenerateStage measures a stage by launching it repeatedly between HIP
// events (Sec. 4.1).
#include <tuple>
#include <set>
#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <numeric>

#include "ios_internal.h"

namespace ios {

int choose_conv_tile(int64_t M, int N, bool pipe_ok);

static int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }
static int round_up(int a, int b) { return (a + b - 1) / b * b; }

std::vector<float *> default_buffers(const ios_graph *g) {
  std::vector<float *> p(g->bufs.size());
  for (size_t i = 0; i < g->bufs.size(); ++i) p[i] = g->bufs[i].dev;
  return p;
}

namespace {

struct SlotMap {
  std::vector<int> bufs;
  int get(int b) {
    for (size_t i = 0; i < bufs.size(); ++i)
      if (bufs[i] == b) return (int)i;
    if ((int)bufs.size() >= kMaxSlots) fail(IOS_E_BAD_STAGE, "stage touches more than 64 buffers");
    bufs.push_back(b);
    return (int)bufs.size() - 1;
  }
};

int resolved(const ios_graph *g, int t) {
  while (g->tensors[t].kind == T_IDENTITY) t = g->ops[g->tensors[t].op].in[0];
  return t;
}

void set_inputs(const ios_graph *g, const Op &op, DevOp &d, SlotMap &sm) {
  d.n_in = (int)op.in.size();
  for (int i = 0; i < d.n_in; ++i) {
    const Tensor &t = g->tensors[resolved(g, op.in[i])];
    d.in_slot[i] = sm.get(t.buf);
    d.in_coff[i] = t.coff;
    d.in_ctot[i] = g->bufs[t.buf].ctot;
    d.in_bytes[i] = (int32_t)(g->bufs[t.buf].elems(g->batch) * sizeof(float));
  }
}

void set_route(const ios_graph *g, DevOp &d, int r, int n0, int out_tensor, SlotMap &sm) {
  const Tensor &t = g->tensors[out_tensor];
  d.route_n0[r] = n0;
  d.route_slot[r] = sm.get(t.buf);
  d.route_coff[r] = t.coff;
  d.route_ctot[r] = g->bufs[t.buf].ctot;
}

void fill_common(const ios_graph *g, const Op &op, DevOp &d) {
  d.N = g->batch;
  d.Cin = op.cin; d.H = op.h; d.W = op.wd;
  d.Ho = op.ho; d.Wo = op.wo;
  d.kh = op.d.kh; d.kw = op.d.kw;
  d.sh = op.d.stride_h; d.sw = op.d.stride_w;
  d.ph = op.d.pad_h; d.pw = op.d.pad_w;
  d.pre_relu = op.d.pre_relu; d.post_relu = op.d.post_relu;
}

// The kernel's tile order across XCDs (workgroup b on XCD b % 8 runs tile
// xcd_tile(b, n, lg), per round of `grid` tiles).
constexpr int kXcdsHost = 8;   // XCDs of an MI355X: workgroup b runs on XCD b % 8

static int xcd_tile_host(int b, int n, int lg) {
  const int full = (n >> (3 + lg)) << (3 + lg);
  if (b >= full) return b;
  const int xcd = b & 7, local = b >> 3;
  return ((((local >> lg) << 3) + xcd) << lg) + (local & ((1 << lg) - 1));
}

// Run length 2^lg of the XCD tile order for a stage: the one whose modelled
// L2 fills are smallest, the shorter run on a tie.  Each XCD is taken to
// fetch, once, the input rows of every conv M-tile its workgroups touch
// (tile rows x input channels x kernel rows) and the weights of every conv
// N-tile (tile columns x padded reduction length).  Long runs keep the
// N-tiles of an M-tile (shared input rows) on one XCD; the plain order keeps
// an N-tile's weights on one XCD when an op has a multiple of 8 N-tiles.
static int choose_xcd_runs(const std::vector<DevOp> &ops, const std::vector<int32_t> &start, int grid) {
  const int n = start.back();
  double best = -1.0;
  int best_lg = 0;
  for (int lg : {0, 2, 4}) {
    std::set<std::tuple<int, int, int>> a_seen, b_seen;
    double bytes = 0.0;
    for (int b = 0; b < grid; ++b)
      for (int base = 0; base + b < n; base += grid) {
        const int t = base + xcd_tile_host(b, std::min(grid, n - base), lg);
        const int i = (int)(std::upper_bound(start.begin(), start.end(), t) - start.begin()) - 1;
        const DevOp &d = ops[i];
        if (d.kind != DK_CONV || t - start[i] >= d.n_tiles) continue;   // padding between op ranges
        const int ti = t - start[i], tm = ti / d.tiles_n, tn = ti % d.tiles_n;
        if (a_seen.insert({i, b & 7, tm}).second) bytes += 4.0 * tile_bm(d.tcfg) * d.CinP * d.kh;
        if (b_seen.insert({i, b & 7, tn}).second)
          bytes += 4.0 * tile_bn(d.tcfg) * (tile_is_pipe(d.tcfg) ? (double)kPipeKB : 16.0) * d.NG;
      }
    if (best < 0.0 || bytes < best) {
      best = bytes;
      best_lg = lg;
    }
  }
  return best_lg;
}

// Per-tile work estimate (MACs or elementwise ops), for ordering tiles.
double tile_work(const DevOp &d) {
  switch (d.kind) {
    case DK_CONV: {
      if (tile_is_pipe(d.tcfg)) return (double)tile_bm(d.tcfg) * tile_bn(d.tcfg) * kPipeKB * d.NG / kWaves;
      TileShape s = tile_shape(d.tcfg);
      return (double)tile_bm(d.tcfg) * tile_bn(d.tcfg) * 16.0 * d.NG / s.wk;
    }
    case DK_SEP:
      if (d.sep_row == 2)
        return (double)d.sepg_rout * d.Wo * d.CinP * (d.kh * d.kw + 32.0 * (kWaves / d.sep_nbt)) / kWaves;
      if (d.sep_row == 3) return 32.0 * d.CinP * (9.0 * d.n_in + 32.0 * d.sep_nbt) / kWaves;
      if (d.sep_row) return 16.0 * d.CinP * (d.row_k * d.row_k * d.n_in + 16.0 * d.sep_nbt) / kWaves;
      return (double)d.sep_bm * d.CinP * (d.kh * d.kw + 16.0 * d.sep_nbt) / kWaves;
    default:
      return (double)kEltPerTile * (d.kind <= DK_POOL_AVG ? d.kh * d.kw : d.n_in) / 4.0;
  }
}

template <class T>
void grow_upload(T **dptr, size_t *cap, const std::vector<T> &v, bool reuse) {
  size_t n = std::max<size_t>(v.size(), 1);
  if (!reuse || *cap < n) {
    if (reuse && *dptr) (void)hipFree(*dptr);
    hip_check(hipMalloc(dptr, sizeof(T) * n), "hipMalloc(stage)");
    if (reuse) *cap = n;
  }
  if (!v.empty())
    hip_check(hipMemcpy(*dptr, v.data(), sizeof(T) * v.size(), hipMemcpyHostToDevice),
              "hipMemcpy(stage)");
}

}  // namespace

void pack_conv_weights(const float *w, int cout, int cin, int kh, int kw, std::vector<float> &out,
                       int *ng, int *nb) {
  const int taps = kh * kw, spt = (cin + 3) / 4, ks_total = taps * spt;
  const int groups = (ks_total + 3) / 4, blocks = (cout + 15) / 16;
  out.assign((size_t)blocks * groups * 256, 0.f);
  for (int b = 0; b < blocks; ++b)
    for (int g = 0; g < groups; ++g)
      for (int kq = 0; kq < 4; ++kq)
        for (int j = 0; j < 16; ++j)
          for (int s = 0; s < 4; ++s) {
            const int ks = 4 * g + s, tap = ks / spt, c = (ks - tap * spt) * 4 + kq, n = 16 * b + j;
            if (ks >= ks_total || c >= cin || n >= cout) continue;
            out[(((size_t)b * groups + g) * 64 + kq * 16 + j) * 4 + s] = w[((size_t)n * cin + c) * taps + tap];
          }
  *ng = groups;
  *nb = blocks;
}

void pack_conv_pipe(const float *w, int cout, int cin, int kh, int kw, std::vector<float> &out, int *nkb) {
  const int taps = kh * kw, K = taps * cin, ldw = round_up(cout, 128), nb = cdiv(K, kPipeKB);
  out.assign((size_t)nb * kPipeKB * ldw, 0.f);
  for (int n = 0; n < cout; ++n)
    for (int c = 0; c < cin; ++c)
      for (int t = 0; t < taps; ++t) out[((size_t)t * cin + c) * ldw + n] = w[((size_t)n * cin + c) * taps + t];
  *nkb = nb;
}

SepGeom sep_geometry(int tile, int cin, int cout, int w, int ho, int wo, int kh, int kw) {
  SepGeom g;
  const int cinp = round_up(cin, 16), nb = round_up(cout, 16) / 16;
  for (int bm = 16 << std::max(0, std::min(tile, kSepStagedTiles - 1)); bm >= 16; bm >>= 1) {
    // rows of the image a run of bm consecutive output pixels can touch,
    // plus the window's halo
    const int span = std::min(ho, (wo - 1 + bm - 1) / wo + 1);
    const int rows = span + kh - 1;
    const int mb = bm / 16;
    // the largest chunk (a multiple of 16 channels) whose staging fits the
    // registers and LDS, then the same number of chunks made even; output
    // channels split into groups of at most nbt blocks so that a wave has at
    // most kSepPairs pairs and a chunk's pointwise weights fit the registers
    for (int ck = std::min(kSepMaxCk, cinp); ck >= 16; ck -= 16) {
      if (ck * rows * w > kSepStagePerThread * kThreads || ck * kh * kw > kSepDwPerThread * kThreads) continue;
      int nbt = std::min({nb, kSepPairs * kWaves / mb, kSepAPerThread * kThreads / 64 / (ck / 16)});
      if (nbt < 1) continue;
      nbt = cdiv(nb, cdiv(nb, nbt));                 // balance the channel groups
      if (sep_lds_floats(bm, ck, rows, w, kh * kw, nbt) * (int)sizeof(float) > kSepMaxLds) continue;
      const int nck = cdiv(cinp, ck);
      const int cke = round_up(cdiv(cinp, nck), 16);
      g.bm = bm; g.ck = cke; g.rows = rows; g.nck = nck; g.nbt = nbt;
      g.lds = sep_lds_floats(bm, cke, rows, w, kh * kw, nbt) * (int)sizeof(float);
      return g;
    }
  }
  return g;
}

void free_stage(CompiledStage *cs) {
  if (!cs->owns) return;
  if (cs->d_table) (void)hipFree(cs->d_table);
  if (cs->d_ctr) (void)hipFree(cs->d_ctr);
  if (cs->d_mw) (void)hipFree(cs->d_mw);
  if (cs->d_mb) (void)hipFree(cs->d_mb);
  cs->d_table = nullptr; cs->d_ctr = nullptr;
  cs->d_mw = nullptr; cs->d_mb = nullptr;
}

void compile_stage(ios_graph *g, const std::vector<int> &ops, int strategy, CompiledStage *cs,
                   bool reuse) {
  if (ops.empty()) fail(IOS_E_BAD_STAGE, "empty stage");
  int blk = g->ops[ops[0]].block;
  for (size_t i = 0; i < ops.size(); ++i) {
    if (g->ops[ops[i]].block != blk) fail(IOS_E_BAD_STAGE, "stage spans several blocks");
    if (i && ops[i] <= ops[i - 1]) fail(IOS_E_BAD_STAGE, "stage units must be distinct, ascending");
  }
  SlotMap sm;
  std::vector<DevOp> dops;
  std::vector<float> mw, mb;
  if (strategy == IOS_MERGE) {
    if (!stage_mergeable(g, ops)) fail(IOS_E_NOT_MERGEABLE, "stage cannot be merged");
    if ((int)ops.size() > kMaxRoutes) fail(IOS_E_UNSUPPORTED, "merge of more than 8 convs");
    const Op &o0 = g->ops[ops[0]];
    int KH = 0, KW = 0, total = 0;
    for (int i : ops) {
      KH = std::max(KH, g->ops[i].d.kh);
      KW = std::max(KW, g->ops[i].d.kw);
      total += g->ops[i].d.cout;
    }
    DevOp d{};
    d.kind = DK_CONV;
    fill_common(g, o0, d);
    d.kh = KH; d.kw = KW;
    d.ph = o0.d.pad_h + (KH - o0.d.kh) / 2;
    d.pw = o0.d.pad_w + (KW - o0.d.kw) / 2;
    d.Cout = total;
    d.CinP = round_up(o0.cin, 4);
    // merged kernel [total][cin][KH][KW]: each op's kernel centred, stacked
    // along output channels in ascending unit id (the concat order)
    std::vector<float> wm((size_t)total * o0.cin * KH * KW, 0.f);
    mb.assign(round_up(total, 16), 0.f);
    int n0 = 0;
    d.n_routes = (int)ops.size();
    for (size_t r = 0; r < ops.size(); ++r) {
      const Op &o = g->ops[ops[r]];
      int dh = (KH - o.d.kh) / 2, dwc = (KW - o.d.kw) / 2;
      for (int co = 0; co < o.d.cout; ++co) {
        mb[n0 + co] = o.b[co];
        for (int ci = 0; ci < o.cin; ++ci)
          for (int u = 0; u < o.d.kh; ++u)
            for (int v = 0; v < o.d.kw; ++v)
              wm[(((size_t)(n0 + co) * o0.cin + ci) * KH + u + dh) * KW + v + dwc] =
                  o.w[(((size_t)co * o.cin + ci) * o.d.kh + u) * o.d.kw + v];
      }
      set_route(g, d, (int)r, n0, o.out, sm);
      n0 += o.d.cout;
    }
    // tile shape: forced one, else the measured choice of the largest conv
    int largest = ops[0];
    for (int i : ops)
      if (op_flops(g, g->ops[i]) > op_flops(g, g->ops[largest])) largest = i;
    const bool pipe_ok = pipe_conv_ok(o0.cin, KH * KW, o0.d.pre_relu);
    d.tcfg = std::getenv("IOS_CONV_TILE") ? choose_conv_tile((int64_t)g->batch * o0.ho * o0.wo, total, pipe_ok)
                                           : g->ops[largest].tcfg;
    if (tile_is_pipe(d.tcfg) && !pipe_ok) d.tcfg = TC_16x32_K8;   // the merged window has more than 32 taps
    int nb = 0;
    if (tile_is_pipe(d.tcfg)) {
      pack_conv_pipe(wm.data(), total, o0.cin, KH, KW, mw, &d.NG);
      d.pipe_ldw = round_up(total, 128);
      d.Npad = round_up(total, 16);
    } else {
      pack_conv_weights(wm.data(), total, o0.cin, KH, KW, mw, &d.NG, &nb);
      d.Npad = nb * 16;
    }
    set_inputs(g, o0, d, sm);
    d.route_n0[d.n_routes] = total;
    d.w_bytes = (int32_t)(mw.size() * sizeof(float));
    dops.push_back(d);
  } else if (strategy == IOS_CONCURRENT) {
    // a pipelined conv tile's LDS rings beside the stage table must fit a
    // workgroup; in a stage of very many operators such a conv takes 16x32
    const int n_ops = (int)ops.size();
    const bool pipe_fits = (kSlotWords + ((4 + n_ops + 1 + 3) & ~3) + n_ops * kDevOpWords) * (int)sizeof(int32_t) +
                               pipe_lds_bytes(TC_W128x64) <= kMaxLdsBytes;
    for (size_t i = 0; i < ops.size(); ++i) {
      const Op &o = g->ops[ops[i]];
      DevOp d{};
      fill_common(g, o, d);
      set_inputs(g, o, d, sm);
      d.Cout = o.d.kind == IOS_CONV || o.d.kind == IOS_SEPCONV ? o.d.cout : o.cin;
      d.n_routes = 1;
      set_route(g, d, 0, 0, o.out, sm);
      d.route_n0[1] = d.Cout;
      switch (o.d.kind) {
        case IOS_CONV:
          d.kind = DK_CONV; d.tcfg = o.tcfg; d.CinP = o.CinP; d.Npad = o.Npad;
          d.bias = o.d_bias;
          if (tile_is_pipe(d.tcfg) && !pipe_fits) d.tcfg = TC_16x32_K8;
          if (tile_is_pipe(d.tcfg)) {
            d.NG = o.pipe_nkb;
            d.pipe_ldw = round_up(o.d.cout, 128);
            d.wpk = o.d_wg;
            d.w_bytes = (int32_t)((size_t)o.pipe_nkb * kPipeKB * d.pipe_ldw * sizeof(float));
          } else {
            d.NG = o.NG;
            d.wpk = o.d_wpk;
            d.w_bytes = (int32_t)((size_t)(o.Npad / 16) * o.NG * 256 * sizeof(float));
          }
          break;
        case IOS_SEPCONV: {
          if (o.sep_tile >= kSepLineFirst) {
            // line tile (see the stage kernel)
            const int nb = 1 << (o.sep_tile - kSepLineFirst);
            const LineGeom lg = line_geometry(nb, o.cin, o.d.cout, o.d.kh, o.d.kw, o.d.pad_h, o.d.pad_w,
                                              o.d.stride_h, o.d.stride_w, o.h, o.wd, o.ho, o.wo);
            if (lg.r == 0 || !o.d_pw_line || !o.d_dw_row) fail(IOS_E_UNSUPPORTED, "SEPCONV line tile does not apply");
            d.kind = DK_SEP; d.sep_row = 3;
            d.CinP = round_up(o.cin, 4); d.Npad = o.Npad;
            d.sep_nbt = nb;
            d.row_k = 3;
            d.line_r = lg.r; d.line_rows = lg.rows; d.line_q = lg.q; d.line_chp = lg.chp;
            d.line_nks = lg.nks; d.line_pitch = lg.pitch;
            d.wpk = o.d_pw_line; d.bias = o.d_bias; d.dw = o.d_dw_row;
            d.w_bytes = (int32_t)((size_t)cdiv(o.d.cout, 32) * lg.nks * 64 * sizeof(float));
            d.dw_bytes = (int32_t)((size_t)d.CinP * sep_kkp(3) * sizeof(float));
            break;
          }
          if (o.sep_tile >= kSepgFirst) {
            // GEMM tile (see the stage kernel)
            const SepgGeom sg = sepg_geometry(o.sep_tile - kSepgFirst, (int)o.in.size(), o.d.kh, o.d.kw,
                                              o.d.pad_h, o.d.pad_w, o.h, o.wd, o.ho, o.wo);
            if (sg.bm == 0 || !o.d_pw_pipe) fail(IOS_E_UNSUPPORTED, "SEPCONV GEMM tile does not apply");
            d.kind = DK_SEP; d.sep_row = 2;
            d.CinP = o.CinP; d.Npad = o.Npad;
            d.sep_nbt = sg.bm / 32;
            d.sep_nck = o.CinP / 16;
            d.sep_rows = sg.rows;
            d.sepg_rout = sg.rout; d.sepg_w2 = sg.w2; d.sepg_strips = sg.strips; d.sepg_ps = sg.ps;
            d.sepg_xs = sg.xs; d.sepg_ws = sg.ws;
            d.pipe_ldw = round_up(o.d.cout, 128);
            d.wpk = o.d_pw_pipe; d.bias = o.d_bias; d.dw = o.d_dw;
            d.w_bytes = (int32_t)((size_t)o.CinP * d.pipe_ldw * sizeof(float));
            d.dw_bytes = (int32_t)((size_t)o.CinP * o.d.kh * o.d.kw * sizeof(float));
            break;
          }
          if (o.sep_tile >= kSepStagedTiles) {
            // row tile (see the stage kernel)
            if (!sep_tile_ok(o, o.sep_tile)) fail(IOS_E_UNSUPPORTED, "SEPCONV row tile does not apply");
            d.kind = DK_SEP; d.sep_row = 1;
            d.CinP = round_up(o.cin, 4); d.Npad = o.Npad;
            d.wpk = o.d_pw_row; d.bias = o.d_bias; d.dw = o.d_dw_row;
            d.w_bytes = (int32_t)((size_t)d.CinP * o.Npad * sizeof(float));
            d.row_k = sep_row_window(o.d.kh, o.d.kw);
            d.sep_nbt = o.sep_tile - kSepStagedTiles + 1;
            d.dw_bytes = (int32_t)((size_t)d.CinP * sep_kkp(d.row_k) * sizeof(float));
            break;
          }
          d.kind = DK_SEP; d.CinP = o.CinP; d.Npad = o.Npad; d.NG = o.NG;
          d.wpk = o.d_wpk; d.bias = o.d_bias; d.dw = o.d_dw;
          d.w_bytes = (int32_t)((size_t)(o.Npad / 16) * o.NG * 256 * sizeof(float));
          d.dw_bytes = (int32_t)((size_t)o.CinP * o.d.kh * o.d.kw * sizeof(float));
          const SepGeom sg = sep_geometry(o.sep_tile, o.cin, o.d.cout, o.wd, o.ho, o.wo, o.d.kh, o.d.kw);
          if (sg.bm == 0) fail(IOS_E_UNSUPPORTED, "SEPCONV tile does not fit");
          d.sep_bm = sg.bm;
          d.sep_lbm = 31 - __builtin_clz((unsigned)sg.bm);
          d.sep_ck = sg.ck; d.sep_nck = sg.nck; d.sep_rows = sg.rows; d.sep_nbt = sg.nbt;
          break;
        }
        case IOS_POOL_MAX: d.kind = DK_POOL_MAX; break;
        case IOS_POOL_AVG: d.kind = DK_POOL_AVG; break;
        case IOS_ADD: d.kind = DK_ADD; break;
        case IOS_MEAN: d.kind = DK_MEAN; d.inv_n = 1.0f / (float)o.in.size(); break;
        default: fail(IOS_E_BAD_STAGE, "not a schedule unit");
      }
      // in-stage producers
      for (int t : o.in)
        for (int p : unit_producers(g, t)) {
          auto it = std::find(ops.begin(), ops.end(), p);
          if (it == ops.end()) continue;
          int j = (int)(it - ops.begin());
          bool dup = false;
          for (int k = 0; k < d.n_deps; ++k) dup |= d.dep[k] == j;
          if (dup) continue;
          if (d.n_deps >= kMaxDeps) fail(IOS_E_UNSUPPORTED, "too many in-stage producers");
          d.dep[d.n_deps++] = j;
        }
      dops.push_back(d);
    }
    for (auto &d : dops)
      for (int k = 0; k < d.n_deps; ++k) dops[d.dep[k]].signal = 1;
  } else {
    fail(IOS_E_ARG, "unknown strategy");
  }
  // tile counts
  for (auto &d : dops) {
    int64_t M = (int64_t)d.N * d.Ho * d.Wo;
    if (d.kind == DK_CONV) {
      d.tiles_m = cdiv(M, tile_bm(d.tcfg));
      d.tiles_n = cdiv(d.Cout, tile_bn(d.tcfg));
    } else if (d.kind == DK_SEP && d.sep_row == 2) {
      // GEMM tile: (image, block of sepg_rout output rows) x groups of 32 (8 / sep_nbt) channels
      d.tiles_per_plane = cdiv(d.Ho, d.sepg_rout);
      d.tiles_m = d.N * d.tiles_per_plane;
      d.tiles_n = cdiv(d.Cout, 32 * (kWaves / d.sep_nbt));
    } else if (d.kind == DK_SEP && d.sep_row == 3) {
      // line tile: (image, block of line_r output rows) x groups of 32 sep_nbt channels
      d.tiles_per_plane = cdiv(d.Ho, d.line_r);
      d.tiles_m = d.N * d.tiles_per_plane;
      d.tiles_n = cdiv(d.Cout, 32 * d.sep_nbt);
    } else if (d.kind == DK_SEP && d.sep_row) {
      // row tile: (image, output row, 16-pixel block of the row) x groups of
      // sep_nbt 16-channel output blocks
      d.row_bpr = cdiv(d.Wo, 16);
      d.tiles_m = d.N * d.Ho * d.row_bpr;
      d.tiles_n = cdiv(d.Npad / 16, d.sep_nbt);
    } else if (d.kind == DK_SEP) {
      // tiles: (image, run of sep_bm output pixels) x groups of sep_nbt
      // 16-channel output blocks
      d.tiles_per_plane = cdiv((int64_t)d.Ho * d.Wo, d.sep_bm);
      d.tiles_m = d.N * d.tiles_per_plane;
      d.tiles_n = cdiv(d.Npad / 16, d.sep_nbt);
    } else if (d.kind == DK_POOL_MAX || d.kind == DK_POOL_AVG) {
      // output rows per tile: as many as fit (with halo) in the LDS budget
      int rows = d.Ho;
      while (rows > 1 && ((rows - 1) * d.sh + d.kh) * d.W > kPoolLdsFloats) --rows;
      if (((rows - 1) * d.sh + d.kh) * d.W > kPoolLdsFloats)
        fail(IOS_E_UNSUPPORTED, "pooling input rows too wide for the LDS tile");
      // strided pools over few planes (the stems' down-sampling pools): bands
      // of rows until the pool has kPoolMinTiles tiles, each band at least one
      // output per thread.  Stride-1 pools keep whole planes: beside convs in
      // a stage, more and smaller pool tiles measured slower.
      const int n_planes = d.N * d.Cout;
      if (d.sh > 1 && n_planes * cdiv(d.Ho, rows) < kPoolMinTiles) {
        const int bands = cdiv(kPoolMinTiles, n_planes);
        rows = std::min(rows, std::max(cdiv(d.Ho, bands), cdiv(kThreads, d.Wo)));
      }
      d.rows_per_tile = rows;
      d.tiles_per_plane = cdiv(d.Ho, rows);
      d.tiles_m = d.N * d.Cout * d.tiles_per_plane;
      d.tiles_n = 1;
      d.planes_per_tile = 1;
      const int in_rows_all = std::min(d.H, (d.Ho - 1) * d.sh - d.ph + d.kh);
      if (rows == d.Ho && in_rows_all > 0) {
        // several whole planes per tile when the planes are small (so that
        // the threads of a tile have outputs to compute) or many (batches:
        // up to kPoolTileOutputs outputs per tile, so that fewer workgroups
        // pay the launch prologue), as long as the pool keeps kPoolMinTiles
        // tiles
        const int in_rows = in_rows_all;
        const int planes = d.N * d.Cout;
        const int p = std::min({std::max(kThreads, kPoolTileOutputs) / (d.Ho * d.Wo),
                                kPoolLdsFloats / (in_rows * d.W), planes / kPoolMinTiles});
        if (p > 1) {
          d.planes_per_tile = p;
          d.pool_in_rows = in_rows;
          d.tiles_m = cdiv(planes, p);
        }
      }
    } else {
      d.tiles_per_plane = cdiv((int64_t)d.Ho * d.Wo, kEltPerTile);
      d.tiles_m = d.N * d.Cout * d.tiles_per_plane;
      d.tiles_n = 1;
    }
    d.n_tiles = d.tiles_m * d.tiles_n;
    const auto fd = [](int v) { return make_fdiv((uint32_t)std::max(1, v)); };
    d.fd_tn = fd(d.tiles_n);
    d.fd_howo = fd(d.Ho * d.Wo);
    d.fd_wo = fd(d.Wo);
    d.fd_spt = fd(d.CinP / 4);
    d.fd_kw = fd(d.kw);
    d.fd_pimg = fd(d.kind == DK_SEP && d.sep_row == 1 ? d.Ho * d.row_bpr : d.tiles_per_plane);
    d.fd_ps = fd(d.sepg_ps);
    d.fd_w2 = fd(d.sepg_w2);
    d.fd_strips = fd(d.sepg_strips);
    d.fd_rbpr = fd(d.row_bpr);
    d.fd_cin = fd(d.Cin);
    d.fd_rw = fd(d.sep_rows * d.W);
    d.fd_w = fd(d.W);
    d.fd_tpp = fd(d.tiles_per_plane);
    d.fd_c = fd(d.Cout);
    d.fd_pin = fd(d.pool_in_rows * d.W);
    d.fd_lq = fd(d.line_q);
    d.fd_lw4 = fd(d.W / 4);
  }
  // tile order: producers before consumers (depth), longer tiles first; the
  // ops are stored in that order so that each owns a contiguous tile range
  int n = (int)dops.size();
  if (n > kMaxStageOps) fail(IOS_E_UNSUPPORTED, "more than 64 operators in one stage");
  std::vector<int> depth(n, 0);
  for (int i = 0; i < n; ++i)
    for (int k = 0; k < dops[i].n_deps; ++k) depth[i] = std::max(depth[i], depth[dops[i].dep[k]] + 1);
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
    if (depth[a] != depth[b]) return depth[a] < depth[b];
    return tile_work(dops[a]) > tile_work(dops[b]);
  });
  std::vector<int> pos(n);
  for (int i = 0; i < n; ++i) pos[order[i]] = i;
  std::vector<DevOp> sorted;
  std::vector<int32_t> start{0};
  bool persistent = false, big_conv = false, has_sep = false, has_row = false, has_pipe = false;
  for (const DevOp &d : dops) persistent |= d.n_deps > 0;
  int lds = 0;
  for (size_t k = 0; k < order.size(); ++k) {
    DevOp d = dops[order[k]];
    for (int j = 0; j < d.n_deps; ++j) d.dep[j] = pos[d.dep[j]];
    sorted.push_back(d);
    // Each op's range starts at a multiple of the XCD count (one tile per
    // workgroup launches): workgroup b runs on XCD b % 8, so tile i of every
    // op lands on the same XCD, and ops that read one tensor with the same
    // pixel tiling (the 1x1 convs of an Inception block) share its L2 lines
    // instead of fetching them once per op.  The padding workgroups exit at
    // once.
    int end = start.back() + d.n_tiles;
    if (!persistent && k + 1 < order.size()) end = round_up(end, kXcdsHost);
    start.push_back(end);
    big_conv |= d.kind == DK_CONV && !tile_is_light(d.tcfg) && !tile_is_pipe(d.tcfg);
    has_pipe |= d.kind == DK_CONV && tile_is_pipe(d.tcfg);
    has_sep |= d.kind == DK_SEP && (d.sep_row == 0 || d.sep_row == 2);
    has_row |= d.kind == DK_SEP && (d.sep_row == 1 || d.sep_row == 3);
    lds = std::max(lds, op_lds_bytes(d));
  }
  cs->ops = sorted;
  cs->op_start = start;
  cs->slot_buf = sm.bufs;
  // table: header, op_start, DevOps (the kernel copies it to LDS)
  const int devop_off = (4 + n + 1 + 3) & ~3;
  const int table_words = devop_off + n * kDevOpWords;
  cs->lds_bytes = (kSlotWords + table_words) * (int)sizeof(int32_t) + lds;
  if (cs->lds_bytes > kMaxLdsBytes) fail(IOS_E_UNSUPPORTED, "stage needs more LDS than a workgroup has");
  cs->persistent = persistent;
  const int kinds = (int)has_sep + (int)has_row + (int)has_pipe;
  cs->variant = big_conv || kinds > 1 ? KV_FULL
                : has_sep            ? KV_SEP
                : has_row            ? KV_SEPROW
                : has_pipe           ? KV_PIPE
                                     : KV_LIGHT;
  cs->grid = start.back();
  if (persistent) {
    int cap = stage_capacity(cs->variant, cs->lds_bytes);
    if (cap <= 0) fail(IOS_E_HIP, "cannot size the persistent launch of a stage with dependencies");
    cs->grid = std::min(cs->grid, cap);
  }
  cs->owns = !reuse;
  // device copies
  if (!mw.empty()) {
    size_t *wc = reuse ? &g->prof_w_cap : nullptr, *bc = reuse ? &g->prof_b_cap : nullptr;
    size_t dummy_w = 0, dummy_b = 0;
    grow_upload(&cs->d_mw, wc ? wc : &dummy_w, mw, reuse);
    grow_upload(&cs->d_mb, bc ? bc : &dummy_b, mb, reuse);
    cs->ops[0].wpk = cs->d_mw;
    cs->ops[0].bias = cs->d_mb;
  }
  cs->table.assign(table_words, 0);
  cs->table[0] = n;
  cs->table[1] = start.back();
  cs->table[2] = devop_off;
  // XCD run length: forced by IOS_XCD_RUNS=<0|2|4> (log2 of the run), else
  // the one ios_schedule_tune_tiles set on all of the stage's units, else
  // the L2-fill model's choice
  int lg = g->ops[ops[0]].xcd_lg;
  for (int i : ops)
    if (g->ops[i].xcd_lg != lg) lg = -1;
  if (const char *e = std::getenv("IOS_XCD_RUNS")) {
    const int v = std::atoi(e);
    if (v != 0 && v != 2 && v != 4) fail(IOS_E_ARG, "IOS_XCD_RUNS must be 0, 2 or 4");
    lg = v;
  }
  cs->table[3] = lg >= 0 ? lg : choose_xcd_runs(sorted, start, cs->grid);
  for (int i = 0; i <= n; ++i) cs->table[4 + i] = start[i];
  std::memcpy(&cs->table[devop_off], cs->ops.data(), sizeof(DevOp) * n);
  size_t d0 = 0, d2 = 0;
  grow_upload(&cs->d_table, reuse ? &g->prof_ops_cap : &d0, cs->table, reuse);
  std::vector<int32_t> ctr(2 + kCtrStride * kCtrCopies, 0);
  grow_upload(&cs->d_ctr, reuse ? &g->prof_ctr_cap : &d2, ctr, reuse);
}

void launch_compiled(ios_graph *g, const CompiledStage &cs, const std::vector<float *> &buf_ptr,
                     hipStream_t stream) {
  StageArgs a{};
  a.n_slots = (int)cs.slot_buf.size();
  for (int i = 0; i < a.n_slots; ++i) a.slot[i] = buf_ptr[cs.slot_buf[i]];
  a.ctr = cs.d_ctr;
  a.err = g->d_err;
  a.spin_limit = 1 << 24;
  hip_check(launch_stage(cs.d_table, (int)cs.table.size(), a, cs.persistent, cs.grid, cs.lds_bytes,
                         cs.variant, stream),
            "stage launch");
}

int64_t profile_stage(ios_graph *g, const std::vector<int> &ops, int strategy, int warmup,
                      int reps, int repeats) {
  if (reps < 1 || repeats < 1 || warmup < 0) fail(IOS_E_ARG, "bad profiling counts");
  CompiledStage &cs = g->prof_stage;
  compile_stage(g, ops, strategy, &cs, true);
  std::vector<float *> bufs = default_buffers(g);
  for (int i = 0; i < warmup; ++i) launch_compiled(g, cs, bufs, g->stream);
  std::vector<double> per;
  for (int r = 0; r < repeats; ++r) {
    hip_check(hipEventRecord(g->ev0, g->stream), "hipEventRecord");
    for (int i = 0; i < reps; ++i) launch_compiled(g, cs, bufs, g->stream);
    hip_check(hipEventRecord(g->ev1, g->stream), "hipEventRecord");
    hip_check(hipEventSynchronize(g->ev1), "hipEventSynchronize");
    float ms = 0.f;
    hip_check(hipEventElapsedTime(&ms, g->ev0, g->ev1), "hipEventElapsedTime");
    per.push_back((double)ms * 1e6 / reps);
  }
  // a bounded intra-stage wait that gave up during the measurement makes the
  // latency meaningless: fail here (and clear the flag) rather than let a
  // later ios_device_status report it against ios_run
  int32_t err = 0;
  hip_check(hipMemcpy(&err, g->d_err, sizeof(err), hipMemcpyDeviceToHost), "hipMemcpy(err)");
  if (err) {
    hip_check(hipMemset(g->d_err, 0, sizeof(int32_t)), "hipMemset(err)");
    fail(IOS_E_DEVICE, "a stage kernel reported an error while the stage was being measured");
  }
  std::sort(per.begin(), per.end());
  return (int64_t)(per[per.size() / 2] + 0.5);
}

}  // namespace ios
