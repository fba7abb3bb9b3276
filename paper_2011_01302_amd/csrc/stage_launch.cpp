// Host side of the stage kernel: LDS sizes, occupancy and launches.  Each
// (kernel variant, launch kind) is compiled in a translation unit of its own
// (stage_kernel_<variant>[_persist].hip) so that they build in parallel; each
// exports a kernel pointer getter and a launcher.
#include "ios_internal.h"

namespace ios {

void *stage_kernel_fn_light();
hipError_t stage_launch_light(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_light_persist();
hipError_t stage_launch_light_persist(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_sep();
hipError_t stage_launch_sep(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_sep_persist();
hipError_t stage_launch_sep_persist(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_seprow();
hipError_t stage_launch_seprow(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_seprow_persist();
hipError_t stage_launch_seprow_persist(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_pipe();
hipError_t stage_launch_pipe(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_pipe_persist();
hipError_t stage_launch_pipe_persist(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_full();
hipError_t stage_launch_full(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);
void *stage_kernel_fn_full_persist();
hipError_t stage_launch_full_persist(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s);

int op_lds_bytes(const DevOp &op) {
  if (op.kind == DK_CONV && tile_is_pipe(op.tcfg)) return pipe_lds_bytes(op.tcfg);
  if (op.kind == DK_CONV) {
    TileShape s = tile_shape(op.tcfg);
    return s.wk * tile_bn(op.tcfg) * (tile_bm(op.tcfg) + 1) * (int)sizeof(float);
  }
  if (op.kind == DK_SEP && op.sep_row == 2)
    return sepg_lds_bytes(op.sepg_xs, op.sepg_ws, 32 * op.sep_nbt, 32 * (kWaves / op.sep_nbt));
  if (op.kind == DK_SEP && op.sep_row == 3) {
    LineGeom g;
    g.r = op.line_r; g.rows = op.line_rows; g.q = op.line_q; g.chp = op.line_chp; g.nks = op.line_nks;
    g.pitch = op.line_pitch;
    line_offsets(g, op.sep_nbt);
    return g.floats * (int)sizeof(float);
  }
  if (op.kind == DK_SEP && op.sep_row) return sep_row_lds_bytes(op.CinP, op.row_k, op.sep_nbt);
  if (op.kind == DK_SEP)
    return sep_lds_floats(op.sep_bm, op.sep_ck, op.sep_rows, op.W, op.kh * op.kw, op.sep_nbt) * (int)sizeof(float);
  if ((op.kind == DK_POOL_MAX || op.kind == DK_POOL_AVG) && op.planes_per_tile > 1)
    return op.planes_per_tile * op.pool_in_rows * op.W * (int)sizeof(float);
  if (op.kind == DK_POOL_MAX || op.kind == DK_POOL_AVG)
    return ((op.rows_per_tile - 1) * op.sh + op.kh) * op.W * (int)sizeof(float);
  return 0;
}

static void *kernel_of(int variant, bool persist) {
  switch (variant) {
    case KV_LIGHT: return persist ? stage_kernel_fn_light_persist() : stage_kernel_fn_light();
    case KV_SEP: return persist ? stage_kernel_fn_sep_persist() : stage_kernel_fn_sep();
    case KV_SEPROW: return persist ? stage_kernel_fn_seprow_persist() : stage_kernel_fn_seprow();
    case KV_PIPE: return persist ? stage_kernel_fn_pipe_persist() : stage_kernel_fn_pipe();
    default: return persist ? stage_kernel_fn_full_persist() : stage_kernel_fn_full();
  }
}

int stage_capacity(int variant, int lds_bytes) {
  int dev = 0, per_cu = 0;
  hipDeviceProp_t prop;
  if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void *)kernel_of(variant, true),
                                                   kThreads, lds_bytes) != hipSuccess)
    return 0;
  return per_cu * prop.multiProcessorCount;
}

hipError_t launch_stage(const int32_t *table, int table_words, const StageArgs &args, bool persistent,
                        int grid, int lds_bytes, int variant, hipStream_t stream) {
  // dynamic LDS above the default limit must be allowed per kernel, once
  static int allowed[2][KV_COUNT] = {};
  int &al = allowed[persistent ? 1 : 0][variant];
  if (lds_bytes > 64 * 1024 && lds_bytes > al) {
    hipError_t e = hipFuncSetAttribute(kernel_of(variant, persistent),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
    if (e != hipSuccess) return e;
    al = kMaxLdsBytes;
  }
  const int4 *t = (const int4 *)table;
  const int w = table_words;
  switch (variant) {
    case KV_LIGHT:
      return persistent ? stage_launch_light_persist(t, w, args, grid, lds_bytes, stream)
                        : stage_launch_light(t, w, args, grid, lds_bytes, stream);
    case KV_SEP:
      return persistent ? stage_launch_sep_persist(t, w, args, grid, lds_bytes, stream)
                        : stage_launch_sep(t, w, args, grid, lds_bytes, stream);
    case KV_SEPROW:
      return persistent ? stage_launch_seprow_persist(t, w, args, grid, lds_bytes, stream)
                        : stage_launch_seprow(t, w, args, grid, lds_bytes, stream);
    case KV_PIPE:
      return persistent ? stage_launch_pipe_persist(t, w, args, grid, lds_bytes, stream)
                        : stage_launch_pipe(t, w, args, grid, lds_bytes, stream);
    default:
      return persistent ? stage_launch_full_persist(t, w, args, grid, lds_bytes, stream)
                        : stage_launch_full(t, w, args, grid, lds_bytes, stream);
  }
}

}  // namespace ios
