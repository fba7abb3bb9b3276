// Internal data structures of libios shared by the host sources and the
// stage kernel.  Nothing here is part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <memory>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/ios.h"

namespace ios {

constexpr int kMaxIn = 16;        // inputs of one operator
constexpr int kMaxRoutes = 8;     // destinations of one (merged) conv: s <= 8 ops
constexpr int kMaxDeps = 16;      // in-stage producers one operator waits for
constexpr int kMaxSlots = 64;     // distinct buffers touched by one stage
constexpr int kThreads = 512;     // threads per workgroup (8 wave64)
constexpr int kWaves = kThreads / 64;
constexpr int kMaxStageOps = 64;  // operators of one stage (a block holds at most 64 units)
// Each op's completion counter is kept in kCtrCopies copies kCtrStride ints
// apart (different memory channels); a waiting workgroup polls one copy.
constexpr int kCtrCopies = 32;
constexpr int kCtrStride = 64;    // >= kMaxStageOps
constexpr int kMaxUnitsPerBlock = 64;
constexpr int64_t kInf = INT64_MAX;
// Device array that ios_run_noalloc uses for the intermediates and the
// in-stage counters (one per device, held until the process ends).
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;

// Kinds of work a stage kernel tile can do.
enum DevKind : int32_t {
  DK_CONV = 0,      // implicit-GEMM conv on fp32 MFMA (also merged convs)
  DK_SEP = 1,       // fused sum -> ReLU -> depthwise -> pointwise (MFMA)
  DK_POOL_MAX = 2,
  DK_POOL_AVG = 3,
  DK_ADD = 4,
  DK_MEAN = 5,
};

// Conv tile shapes.  A workgroup has 8 waves arranged WM x WN x WK; each
// wave owns FM x FN blocks of 16x16 outputs and 1/WK of the reduction.
enum TileCfg : int32_t {
  TC_16x16_K8 = 0,   // FM1 FN1 WM1 WN1 WK8
  TC_16x32_K8 = 1,   // FM1 FN2 WM1 WN1 WK8
  TC_32x32_K8 = 2,   // FM2 FN2 WM1 WN1 WK8
  TC_32x64_K4 = 3,   // FM2 FN2 WM1 WN2 WK4
  TC_64x64_K2 = 4,   // FM2 FN2 WM2 WN2 WK2
  TC_128x64 = 5,     // FM2 FN2 WM4 WN2 WK1
  // pipelined tiles (see the stage kernel): 8 waves of 32x32 outputs on
  // v_mfma_f32_32x32x2_f32, operands staged in LDS by direct loads; first
  // through one ring shared by the workgroup (a barrier per block) ...
  TC_P128x64 = 6,    // 4 (pixels) x 2 (channels) waves
  TC_P256x32 = 7,    // 8 x 1
  TC_P64x128 = 8,    // 2 x 4
  // ... then through a private ring per wave (no barrier)
  TC_W128x64 = 9,
  TC_W256x32 = 10,
  TC_W64x128 = 11,
  TC_COUNT = 12,
};
static_assert(TC_COUNT == IOS_CONV_TILE_SHAPES, "tile shapes of the public API");

struct TileShape { int fm, fn, wm, wn, wk; };
inline TileShape tile_shape(int cfg) {
  switch (cfg) {
    case TC_16x16_K8: return {1, 1, 1, 1, 8};
    case TC_16x32_K8: return {1, 2, 1, 1, 8};
    case TC_32x32_K8: return {2, 2, 1, 1, 8};
    case TC_32x64_K4: return {2, 2, 1, 2, 4};
    case TC_64x64_K2: return {2, 2, 2, 2, 2};
    default: return {2, 2, 4, 2, 1};
  }
}
// Tile shapes the light kernel variant contains (one 16-pixel block per wave).
inline bool tile_is_light(int cfg) { return cfg == TC_16x16_K8 || cfg == TC_16x32_K8; }
inline bool tile_is_pipe(int cfg) { return cfg >= TC_P128x64 && cfg < TC_COUNT; }
inline bool tile_is_wave_ring(int cfg) { return cfg >= TC_W128x64 && cfg < TC_COUNT; }
// pipelined tiles: waves along pixels (and kWaves / that along channels)
inline int pipe_wm(int cfg) {
  const int k = tile_is_wave_ring(cfg) ? cfg - TC_W128x64 : cfg - TC_P128x64;
  return k == 0 ? 4 : k == 1 ? 8 : 2;
}
inline int tile_bm(int cfg) {
  if (tile_is_pipe(cfg)) return 32 * pipe_wm(cfg);
  TileShape s = tile_shape(cfg);
  return 16 * s.fm * s.wm;
}
inline int tile_bn(int cfg) {
  if (tile_is_pipe(cfg)) return 32 * (kWaves / pipe_wm(cfg));
  TileShape s = tile_shape(cfg);
  return 16 * s.fn * s.wn;
}
// Pipelined tiles: reduction blocks of kPipeKB channels of one tap, a ring of
// kPipeStages blocks of both operands in LDS (per workgroup or per wave);
// weights packed [k][round128(Cout)]
// with k = (u kw + v) Cin + c, zero past Cout.  They apply to convs whose Cin
// is a multiple of kPipeKB (a block never spans two taps), with at most 32
// taps (one bit per tap in a lane's mask) and no input ReLU (the operands
// reach LDS through no register).
constexpr int kPipeKB = 16;
constexpr int kPipeStages = 4;
// Per-wave rings: blocks of kWaveKB channels, kWaveStages slots (64 KB per
// workgroup, so that two workgroups fit on a CU).
constexpr int kWaveKB = 8;
constexpr int kWaveStages = 4;
inline int pipe_lds_bytes(int cfg) {
  if (tile_is_wave_ring(cfg))                        // a ring per wave: A and B of each slot
    return kWaves * kWaveStages * 2 * kWaveKB * 32 * (int)sizeof(float);
  return kPipeStages * kPipeKB * (tile_bm(cfg) + tile_bn(cfg)) * (int)sizeof(float);
}
inline bool pipe_conv_ok(int cin, int taps, int pre_relu) {
  return cin > 0 && cin % kPipeKB == 0 && taps <= 32 && !pre_relu;
}

// SEPCONV tile: BM = 16 << tile consecutive output pixels of one image x
// sep_nbt blocks of 16 output channels; the input channels are reduced in
// chunks of sep_ck (32 or 16), whose input rows (with the window's halo) are
// staged in LDS.  The shape follows from the tile choice and the operator's
// sizes (sep_geometry), within these limits.
// Tile choices: 0 .. kSepStagedTiles - 1 the staged tile (BM = 16 << choice),
// then kSepRowMaxNB choices of the row tile (16 output pixels of one output
// row x 1 .. kSepRowMaxNB channel blocks; Cin <= 256, windows up to 5 x 5),
// then kSepgTiles choices of the GEMM tile (whole output rows in 128 or 64
// MFMA columns x 64 or 128 output channels; one input, 3 x 3 or 5 x 5
// windows that keep the size), then kSepLineTiles choices of the line tile
// (32 / Wo whole output rows x 32 or 64 output channels; 3 x 3 windows that
// keep the size, rows of a multiple of 4 floats up to 32, Cin <= 96).
constexpr int kSepStagedTiles = 3;       // BM = 16, 32, 64
constexpr int kSepRowMaxNB = 4;
constexpr int kSepgTiles = 2;
constexpr int kSepgFirst = kSepStagedTiles + kSepRowMaxNB;
constexpr int kSepLineTiles = 2;
constexpr int kSepLineFirst = kSepgFirst + kSepgTiles;
constexpr int kSepTiles = kSepLineFirst + kSepLineTiles;
constexpr int kSepgStages = 3;           // GEMM tile: ring slots of 16 input channels (two chunks in flight)
constexpr int kSepgMaxRows = 4;          // GEMM tile: output rows per tile at most
constexpr int kSepgMaxCopies = 12;       // GEMM tile: 64-float input copies per wave and chunk at most
constexpr int kSepgMaxLds = 128 * 1024;  // GEMM tile: LDS bytes at most (the stage table comes on top)
// GEMM tile geometry (bm = 0: the choice does not apply): rout output rows
// per tile (2 .. kSepgMaxRows), staged input rows (rows), the staged plane's
// row pitch (w2 = W + 2 pw, a zero halo on both sides) and pitch (ps, odd),
// the floats per ring slot of the input planes (xs) and of the depthwise
// weights (ws), and the depthwise strips of 2 output columns per row.
struct SepgGeom {
  int bm = 0, bn = 0, rout = 0, rows = 0, w2 = 0, ps = 0, xs = 0, ws = 0, strips = 0, lds = 0;
};
// LDS bytes of a GEMM tile: the ring (input planes, pointwise and depthwise
// weights per slot) and two B operand buffers [16][bm + 1].
inline int sepg_lds_bytes(int xs, int ws, int bm, int bn) {
  return (kSepgStages * (xs + 16 * bn + ws) + 2 * 16 * (bm + 1)) * 4;
}
inline SepgGeom sepg_geometry(int choice, int n_in, int kh, int kw, int ph, int pw, int H, int W, int Ho, int Wo) {
  SepgGeom g;
  const int wmw = choice == 0 ? 4 : 2, bm = 32 * wmw, bn = 32 * (8 / wmw);
  if (n_in != 1 || kh != kw || (kh != 3 && kh != 5) || ph != kh / 2 || pw != kw / 2 || Ho != H || Wo != W ||
      Wo < 1)
    return g;
  const int rout = std::min(std::min(bm / Wo, Ho), kSepgMaxRows);
  if (rout < 2 && Ho >= 2) return g;
  if (rout < 1) return g;
  const int rows = rout + kh - 1, w2 = W + 2 * pw, ps = (rows * w2) | 1;
  const int xs = (16 * ps + 63) / 64 * 64, ws = (16 * kh * kw + 63) / 64 * 64;
  if (xs > kSepgMaxCopies * 8 * 64) return g;
  if (sepg_lds_bytes(xs, ws, bm, bn) > kSepgMaxLds) return g;
  g.bm = bm; g.bn = bn; g.rout = std::max(rout, 2); g.rows = g.rout + kh - 1; g.w2 = w2;
  g.ps = (g.rows * w2) | 1; g.xs = (16 * g.ps + 63) / 64 * 64; g.ws = ws; g.strips = (Wo + 1) / 2;
  g.lds = sepg_lds_bytes(g.xs, ws, bm, bn);
  if (g.xs > kSepgMaxCopies * 8 * 64 || g.lds > kSepgMaxLds) return SepgGeom{};
  return g;
}

// Line tile geometry (r = 0: the choice does not apply): r output rows per
// tile (r Wo <= 32 MFMA columns), rows = r + 2 input rows staged per channel,
// q = rows W / 4 16-byte pieces per channel, chp = 512 / q channels loaded at
// once (a thread loads kLineMaxLoads channels of one piece at most), nks =
// k-steps of 2 channels, pitch = W + 8 floats per staged row (the data at
// column 4, zeros around it).  LDS (floats): the staged rows [2 nks][rows]
// [pitch] (later the partial sums [8 waves][16][64]), the depthwise outputs
// [nks][64] (at dwb), the depthwise weights [2 nks][kkp] (dww), the pointwise
// weights [nb][nks][64] (al), the biases [32 nb] (bl).
constexpr int kLineInFlight = 4;         // inputs whose loads are in flight at once
constexpr int kLineMaxLoads = 4;         // 16-byte loads per thread and input
constexpr int kLineMaxCin = 96;
constexpr int kLineMaxLds = 128 * 1024;  // bytes (the stage table comes on top)
struct LineGeom {
  int r = 0, rows = 0, q = 0, chp = 0, nks = 0, pitch = 0;
  int dwb = 0, dww = 0, al = 0, bl = 0, floats = 0;
};
__host__ __device__ inline void line_offsets(LineGeom &g, int nb) {
  const int slab = 2 * g.nks * g.rows * g.pitch, red = 8 * 1024;
  g.dwb = slab > red ? slab : red;
  g.dww = g.dwb + g.nks * 64;
  g.al = g.dww + 2 * g.nks * 12;
  g.bl = g.al + nb * g.nks * 64;
  g.floats = g.bl + ((32 * nb + 63) & ~63);
}
inline LineGeom line_geometry(int nb, int cin, int cout, int kh, int kw, int ph, int pw, int sh, int sw, int H,
                              int W, int Ho, int Wo) {
  LineGeom g;
  if (kh != 3 || kw != 3 || ph != 1 || pw != 1 || sh != 1 || sw != 1 || Ho != H || Wo != W || W % 4 != 0 ||
      W > 32 || cin < 1 || cin > kLineMaxCin || cout < 1 || (nb > 1 && cout <= 16 * nb))
    return g;
  g.r = std::min(32 / W, Ho);
  g.rows = g.r + 2;
  g.q = g.rows * (W / 4);
  g.chp = 512 / g.q;
  g.nks = (cin + 1) / 2;
  g.pitch = W + 8;
  if (g.chp < 1 || (2 * g.nks + g.chp - 1) / g.chp > kLineMaxLoads) return LineGeom{};
  line_offsets(g, nb);
  if (g.floats * 4 > kLineMaxLds) return LineGeom{};
  return g;
}

constexpr int kSepRowMaxChannels = 256;
constexpr int kSepPairs = 4;             // (pixel block, channel block) pairs per wave at most
constexpr int kSepStagePerThread = 8;   // staged input floats per thread and chunk at most
constexpr int kSepMaxLds = 64 * 1024;    // bytes of LDS one SEPCONV tile may use
constexpr int kSepMaxWindow = 7;         // depthwise windows up to 7 x 7
constexpr int kSepMaxCk = 64;            // input channels per chunk at most
constexpr int kSepDwPerThread = 4;       // depthwise weights per thread and chunk at most
constexpr int kSepAPerThread = 2;        // 16-byte pointwise weight loads per thread and chunk at most
struct SepGeom {
  int bm = 0, ck = 0, rows = 0, nck = 0, nbt = 0, lds = 0;
};
// Tile geometry of a SEPCONV for tile choice `tile` (BM = 16 << tile, lowered
// until the staging fits); bm = 0 if nothing fits.
SepGeom sep_geometry(int tile, int cin, int cout, int w, int ho, int wo, int kh, int kw);
// Whether SEPCONV tile choice `tile` can run `op` (graph.cpp).
struct Op;
bool sep_tile_ok(const Op &op, int tile);
bool conv_tile_ok(const Op &op, int cfg);
__host__ __device__ inline int sep_pitch(int bm) { return (bm & 31) == 16 ? bm : bm + 16; }
// Row tile: the depthwise window padded to K x K, K = 3 or 5 (0 = too
// large); its weights packed [CinP][sep_kkp(K)].
inline int sep_row_window(int kh, int kw) {
  int k = kh > kw ? kh : kw;
  return k <= 3 ? 3 : k <= 5 ? 5 : 0;
}
__host__ __device__ inline int sep_kkp(int K) { return (K * K + 3) & ~3; }
// LDS of one wave of a row tile (floats, a multiple of 64): depthwise and
// pointwise weights of its k-steps, plus 64 floats so that no 64-lane copy
// can reach the next wave's region; the tile's LDS also holds the
// [wave][16 nbt columns][17] partial sums afterwards.
__host__ __device__ inline int sep_row_wave_floats(int CinP, int K, int nbt) {
  const int ksw = (CinP / 4 + 7) / 8;
  return ((ksw * 4 * (sep_kkp(K) + 16 * nbt) + 63) & ~63) + 64;
}
// The tile's biases (16 nbt floats, 64 reserved) follow both regions.
__host__ __device__ inline int sep_row_bias_offset(int CinP, int K, int nbt) {
  const int w = 8 * sep_row_wave_floats(CinP, K, nbt), r = 8 * kSepRowMaxNB * 16 * 17;
  return w > r ? w : r;
}
__host__ __device__ inline int sep_row_lds_bytes(int CinP, int K, int nbt) {
  return (sep_row_bias_offset(CinP, K, nbt) + 64) * 4;
}
// LDS of a SEPCONV tile in floats: the staged input and depthwise weights of
// one chunk, two pointwise weight buffers, the depthwise outputs and the
// tile's biases (whole copies of 64 floats).
__host__ __device__ inline int sep_lds_floats(int bm, int ck, int rows, int w, int kk, int nbt) {
  return ck * rows * w + ck * kk + 2 * nbt * (ck / 16) * 256 + ck * sep_pitch(bm) + (nbt * 16 + 63) / 64 * 64;
}
// Elementwise tiles: add / mean handle up to kEltPerTile contiguous outputs of
// one channel plane; a pool tile handles a band of output rows of one plane
// whose input rows (with halo) fit in kPoolLdsFloats of LDS.
constexpr int kEltPerTile = 4 * kThreads;
constexpr int kPoolLdsFloats = 8192;
// Pools whose whole plane fits one tile take several planes per tile, up to
// max(threads, kPoolTileOutputs) outputs, as long as the launch keeps at
// least kPoolMinTiles pool tiles.
constexpr int kPoolMinTiles = 256;
constexpr int kPoolTileOutputs = 4096;

// Division by a run-time constant d >= 1 as a multiply-high and a shift:
// n / d == (umulhi(n, mul) + n) >> shr for 0 <= n < 2^31 (Granlund and
// Montgomery, PLDI 1994), so that the kernel never expands an integer divide.
struct FDiv { uint32_t mul, shr; };
inline FDiv make_fdiv(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  return {(uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1), l};
}

// One operator of a compiled stage, as the kernel sees it.
struct alignas(16) DevOp {
  int32_t kind, tcfg;
  int32_t n_in;
  int32_t in_slot[kMaxIn], in_coff[kMaxIn], in_ctot[kMaxIn];
  int32_t in_bytes[kMaxIn];    // size of each input's buffer (buffer-load range)
  int32_t N, Cin, H, W;        // input (batch, channels, height, width)
  int32_t Cout, Ho, Wo;        // output
  int32_t kh, kw, sh, sw, ph, pw;
  int32_t pre_relu, post_relu;
  int32_t CinP;                // CONV: Cin rounded up to 4 (reduction per tap); SEP: up to 16
  int32_t Npad;                // Cout rounded up to 16
  int32_t NG;                  // groups of 4 k-steps of the packed weights (CONV: K = taps x CinP; SEP: pointwise)
  int32_t tiles_m, tiles_n, n_tiles;
  int32_t n_routes;            // output column ranges -> destination buffers
  int32_t route_n0[kMaxRoutes + 1];
  int32_t route_slot[kMaxRoutes], route_coff[kMaxRoutes], route_ctot[kMaxRoutes];
  int32_t n_deps;
  int32_t dep[kMaxDeps];       // stage-local indices of ops this op waits for
  int32_t signal;              // 1 if another op of the stage waits for this one
  float inv_n;                 // MEAN: 1 / n_in
  int32_t rows_per_tile;       // POOL: output rows per tile
  int32_t tiles_per_plane;     // POOL / ADD / MEAN: tiles per (image, channel) plane
  int32_t planes_per_tile;     // POOL: whole planes per tile when a plane is small (else 1)
  int32_t pool_in_rows;        // POOL with planes_per_tile > 1: input rows staged per plane
  int32_t sep_bm, sep_lbm;     // SEP: output pixels per tile, log2
  int32_t sep_ck, sep_nck;     // SEP: input channels per chunk, chunks
  int32_t sep_rows;            // SEP: input rows staged per chunk
  int32_t sep_nbt;             // SEP: 16-channel output blocks per tile
  int32_t sep_row;             // SEP: 0 = staged tile, 1 = row tile, 2 = GEMM tile (sep_nbt = its waves along
                               // pixels), 3 = line tile (sep_nbt = its 32-channel output blocks)
  int32_t sepg_rout, sepg_w2;  // SEP GEMM tile: output rows per tile, staged row pitch (W + 2 pw)
  int32_t sepg_strips, sepg_ps;// SEP GEMM tile: depthwise strips of 2 columns per row, staged plane pitch
  int32_t sepg_xs, sepg_ws;    // SEP GEMM tile: floats per ring slot of the input planes and depthwise weights
  int32_t row_k, row_bpr;      // SEP row tile: padded window K, 16-pixel blocks per output row
  int32_t line_r, line_rows;   // SEP line tile: output rows per tile, staged input rows (see LineGeom)
  int32_t line_q, line_chp;    // SEP line tile: 16-byte pieces per staged channel, channels loaded at once
  int32_t line_nks, line_pitch;// SEP line tile: k-steps of 2 channels, staged row pitch
  int32_t pipe_ldw;            // CONV pipelined tile: row length of the packed weights (NG = k-blocks)
  int32_t w_bytes;             // size of wpk in bytes
  int32_t dw_bytes;            // SEP: size of dw in bytes
  // divisors of the tile and pixel decompositions (see FDiv)
  FDiv fd_tn;                  // tiles_n
  FDiv fd_howo, fd_wo;         // Ho * Wo, Wo
  FDiv fd_spt, fd_kw;          // CONV: k-steps per tap, kw
  FDiv fd_pimg, fd_rw, fd_w;   // SEP: pixel tiles (row tile: 16-pixel blocks) per image, staged floats per channel, W
  FDiv fd_rbpr;                // SEP row tile: 16-pixel blocks per row
  FDiv fd_cin;                 // CONV pipelined tile: Cin
  FDiv fd_ps, fd_w2, fd_strips;// SEP GEMM tile: sepg_ps, sepg_w2, sepg_strips
  FDiv fd_tpp, fd_c;           // POOL / ADD / MEAN: tiles_per_plane, Cout
  FDiv fd_pin;                 // POOL with planes_per_tile > 1: floats staged per plane
  FDiv fd_lq, fd_lw4;          // SEP line tile: line_q, W / 4
  const float *wpk;            // CONV: see pack_conv_weights; SEP: the pointwise weights packed the same way
  const float *bias;           // [Npad]
  const float *dw;             // SEP: depthwise [round16(Cin)][kh * kw], channels past Cin zero
};

// A compiled stage's table in device memory (int32 words): a header
// {n_ops, n_tiles, devop_off, 0}, op_start[n_ops + 1] (op i owns tiles
// [op_start[i], op_start[i+1]) in tile order), zero padding to a multiple of
// 4 words, then DevOp[n_ops] from word devop_off.  Every workgroup copies the
// table and the launch's buffer pointers to LDS when it starts (one memory
// round trip for all of its metadata).
constexpr int kDevOpWords = (int)(sizeof(DevOp) / 4);
constexpr int kSlotWords = 2 * kMaxSlots;   // LDS words holding the buffer pointers
constexpr int kMaxLdsBytes = 160 * 1024;    // LDS of one workgroup (gfx950)

// Kernel arguments besides the table: per-launch buffer pointers and the
// intra-stage signalling state.
struct StageArgs {
  int32_t *ctr;        // [1] workgroups finished, [2 + i + kCtrStride * r] tiles done of op i (copy r)
  int32_t *err;        // device error word
  int32_t spin_limit;  // polls before a dependency wait gives up
  int32_t n_slots;
  float *slot[kMaxSlots];
};

// Launch one stage (defined in the HIP translation unit).
// Kernel variant of a stage (see the stage kernel): the smallest one that
// contains every tile kind the stage uses.
enum KernelVariant { KV_LIGHT = 0, KV_SEP = 1, KV_FULL = 2, KV_SEPROW = 3, KV_PIPE = 4, KV_COUNT = 5 };
// table / table_words: the compiled stage's table (a multiple of 4 words);
// lds_bytes: the dynamic LDS, slots and table included.
hipError_t launch_stage(const int32_t *table, int table_words, const StageArgs &args, bool persistent,
                        int grid, int lds_bytes, int variant, hipStream_t stream);
// Workgroups of `variant` with `lds_bytes` of LDS that fit on the device at once (0 if unknown).
int stage_capacity(int variant, int lds_bytes);
// Dynamic LDS a tile of `op` needs (besides the slots and the table).
int op_lds_bytes(const DevOp &op);

// ------------------------------------------------------------------ host IR

enum TensorKind { T_INPUT = 0, T_UNIT = 1, T_CONCAT = 2, T_IDENTITY = 3 };

struct Tensor {
  int c = 0, h = 0, w = 0;
  int kind = T_INPUT;
  int op = -1;              // producing op (unit or view)
  int parent = -1;          // concat tensor containing this one
  int parent_off = 0;       // channel offset inside the parent
  int input_index = -1;
  // resolved at finalize
  int buf = -1, coff = 0;
};

struct Buffer {
  int ctot = 0, h = 0, w = 0;
  int input_index = -1, output_index = -1;
  float *dev = nullptr;     // graph-owned storage (dummy for inputs/outputs)
  size_t elems(int batch) const { return (size_t)batch * ctot * h * w; }
};

struct Op {
  ios_op_desc d{};
  int out = -1;                  // output tensor id
  std::vector<int> in;           // input tensor ids
  std::vector<float> w, b;       // host copies of weights / bias
  int unit = -1;                 // index among schedule units, -1 for views
  int block = -1, local = -1;    // block and bit inside the block
  int cin = 0, h = 0, wd = 0, ho = 0, wo = 0;
  // device copies (units only)
  int CinP = 0, Npad = 0, NG = 0, tcfg = TC_16x32_K8;
  int sep_tile = 1;              // SEPCONV: tile choice (16 << sep_tile output pixels per tile)
  int xcd_lg = -1;               // XCD run length 2^xcd_lg of the stage holding it; -1: modelled
  float *d_wpk = nullptr, *d_bias = nullptr, *d_dw = nullptr;
  float *d_pw_pipe = nullptr;    // SEPCONV GEMM tile: pointwise weights packed like a pipelined 1x1 conv's
  float *d_dw_row = nullptr, *d_pw_row = nullptr;   // SEPCONV row tile: [CinP4][kkp(K)], [CinP4][Npad]
  float *d_pw_line = nullptr;    // SEPCONV line tile: pointwise [ceil(Cout/32)][ceil(Cin/2)][64] (A operands)
  float *d_wg = nullptr;         // CONV, pipelined tiles: [nkb * kPipeKB][round128(Cout)]
  int pipe_nkb = 0;
};

struct Block {
  std::vector<int> ops;          // op indices (units), ascending
  std::vector<uint64_t> succ, pred;
  uint64_t full() const { return ops.size() == 64 ? ~0ull : ((1ull << ops.size()) - 1); }
};

struct CompiledStage {
  std::vector<DevOp> ops;        // in tile order (producers before consumers)
  std::vector<int32_t> op_start; // tile ranges, size ops + 1
  std::vector<int> slot_buf;     // slot -> buffer index
  int lds_bytes = 0;
  bool persistent = false;       // some op waits for another: persistent launch
  int grid = 0;                  // workgroups launched
  int variant = 0;               // KernelVariant
  std::vector<int32_t> table;    // header, op_start, DevOps (see kDevOpWords)
  // device copies (owned unless reused by the profiler)
  int32_t *d_table = nullptr;
  int32_t *d_ctr = nullptr;
  float *d_mw = nullptr, *d_mb = nullptr;   // merged weights / bias
  bool owns = true;
};

struct CostRow { int64_t conc = kInf, merge = kInf; bool merge_measured = false; };

}  // namespace ios

struct ios_graph {
  int batch = 1;
  bool finalized = false;
  bool device_ready = false;      // buffers / weights / stream allocated
  std::vector<ios::Tensor> tensors;
  std::vector<ios::Buffer> bufs;
  std::vector<ios::Op> ops;
  std::vector<int> inputs;       // tensor ids
  std::vector<int> outputs;      // tensor ids
  std::vector<int> units;        // op indices that are schedule units
  std::vector<ios::Block> blocks;
  hipStream_t stream = nullptr;  // library stream for profiling
  int device = 0;
  int32_t *d_err = nullptr;
  // the stage profiler's compiled stage (reused by every candidate stage)
  ios::CompiledStage prof_stage;
  size_t prof_ops_cap = 0, prof_ctr_cap = 0, prof_w_cap = 0, prof_b_cap = 0;
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  // ios_run_noalloc: byte offset of each intermediate buffer in the scratch
  // array (counters first), and the bytes the graph needs there
  std::vector<size_t> noalloc_off;
  size_t noalloc_bytes = 0;
  // last search's cost table, per block: mask -> latencies
  std::vector<std::map<uint64_t, ios::CostRow>> cost_table;
};

struct ios_schedule_t {
  ios_graph *g = nullptr;
  std::vector<int32_t> offsets, unit_ids, strategies;
  std::vector<int> stage_block;
  int64_t states = 0, transitions = 0, measured = 0;
  std::vector<std::unique_ptr<ios::CompiledStage>> compiled;
  std::vector<hipEvent_t> events;
};

namespace ios {

// Errors: thrown inside the library, turned into codes at the ABI.
struct Error {
  int code;
  std::string msg;
};
[[noreturn]] void fail(int code, const std::string &msg);
void hip_check(hipError_t e, const char *what);
// api.cpp: set the calling thread's ios_last_error() text (no allocation)
void set_last_error_text(const char *msg);
// noalloc.hip: per-device set-up of the scratch array (device address, zero
// counters); the counter block's size, which the intermediates follow
void noalloc_setup(int device);
size_t noalloc_counter_bytes();

// graph.cpp
int unit_op_of_tensor(const ios_graph *g, int tensor_id);   // op index or throws
std::vector<int> unit_producers(const ios_graph *g, int tensor_id);
void finalize_graph(ios_graph *g);
void ensure_device(ios_graph *g);
bool stage_mergeable(const ios_graph *g, const std::vector<int> &ops);
int64_t op_flops(const ios_graph *g, const Op &op);

// exec.cpp
// Conv weights w[cout][cin][kh][kw] in the layout the conv tile loads: for
// each block of 16 output channels nb and group g of 4 k-steps (k-step ks =
// tap * CinP/4 + channel/4, tap-major), 64 lanes x 4 floats, lane kq*16 + j
// holding rows 4*(4g+s) + kq (s = 0..3) of column 16 nb + j, i.e. the B
// operands of four consecutive 16x16x4 MFMAs.  Zero-padded to CinP and to 16
// channels.  Sets *ng = groups, *nb = blocks.
void pack_conv_weights(const float *w, int cout, int cin, int kh, int kw, std::vector<float> &out,
                       int *ng, int *nb);
// Conv weights for the pipelined tiles: [nkb * kPipeKB][round128(cout)], row
// k = (u kw + v) cin + c, zero past the kernel and past cout.
void pack_conv_pipe(const float *w, int cout, int cin, int kh, int kw, std::vector<float> &out, int *nkb);
void compile_stage(ios_graph *g, const std::vector<int> &ops, int strategy, CompiledStage *cs,
                   bool reuse);
void free_stage(CompiledStage *cs);
void launch_compiled(ios_graph *g, const CompiledStage &cs, const std::vector<float *> &buf_ptr,
                     hipStream_t stream);
int64_t profile_stage(ios_graph *g, const std::vector<int> &ops, int strategy, int warmup,
                      int reps, int repeats);
std::vector<float *> default_buffers(const ios_graph *g);

}  // namespace ios
