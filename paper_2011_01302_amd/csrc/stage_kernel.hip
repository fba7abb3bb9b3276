// The stage kernel: one launch executes every operator of one schedule stage
// (Sec. 3, "Stage" and "Parallelization Strategy").  Each workgroup (256
// threads = 4 wave64) runs one tile from the stage's tile table:
//   DK_CONV   implicit-GEMM convolution, M = output pixels, N = output
//             channels, K = taps x input channels (tap-major), on
//             v_mfma_f32_16x16x4_f32; the 4 waves split M, N and/or K and
//             reduce their partial sums through LDS; bias + ReLU are applied
//             in the epilogue, which writes each output channel to its
//             destination (a merged conv has several destinations).
//   DK_SEP    "Relu-SepConv" unit (Table 2): the sum of the inputs, ReLU and
//             the depthwise kxk filter are computed into LDS for 32 pixels x
//             all channels, then the pointwise 1x1 runs on MFMA from LDS.
//   DK_POOL_* / DK_ADD / DK_MEAN   elementwise tiles on the vector ALUs.
// Operators of one group run in order (Sec. 3: a group is executed
// sequentially): when a stage has such chains, workgroups take tiles through
// an atomic ticket in topological order and a consumer tile waits until every
// tile of its producers has finished.  A workgroup only waits for tickets
// smaller than its own, all held by workgroups already running, so the waits
// always end.
#include "ios_internal.h"

namespace ios {

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ floatx4 mfma16x16x4(float a, float b, floatx4 c) {
  // D[16x16] += A[16x4] * B[4x16]; lane l supplies A[l%16][l/16] and
  // B[l/16][l%16]; lane l, element j holds D[4*(l/16)+j][l%16].
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float *route_ptr(const StageArgs &a, const DevOp &op, int n, int img,
                                            int pix, int howo) {
  int r = 0;
  while (r + 1 < op.n_routes && n >= op.route_n0[r + 1]) ++r;
  return a.slot[op.route_slot[r]] +
         ((size_t)img * op.route_ctot[r] + op.route_coff[r] + (n - op.route_n0[r])) * howo + pix;
}

// ------------------------------------------------------------------ conv

template <int FM, int FN, int WM, int WN, int WK>
__device__ void conv_tile(const StageArgs &a, const DevOp &op, int t, float *lds) {
  constexpr int BM = 16 * FM * WM, BN = 16 * FN * WN, LDM = BM + 1;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wk = wave % WK, wmn = wave / WK, wm = wmn % WM, wn = wmn / WM;
  const int tm = t / op.tiles_n, tn = t - tm * op.tiles_n;
  const int Wo = op.Wo, howo = op.Ho * Wo, M = op.N * howo;
  const int H = op.H, W = op.W, HW = H * W;
  const int row16 = lane & 15, kq = lane >> 4;
  const float *__restrict__ xin = a.slot[op.in_slot[0]];

  int base[FM], ih0[FM], iw0[FM];
  bool mv[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    int m = tm * BM + wm * 16 * FM + fm * 16 + row16;
    mv[fm] = m < M;
    int mm = mv[fm] ? m : 0;
    int img = mm / howo, r = mm - img * howo, oh = r / Wo, ow = r - oh * Wo;
    ih0[fm] = oh * op.sh - op.ph;
    iw0[fm] = ow * op.sw - op.pw;
    base[fm] = (img * op.in_ctot[0] + op.in_coff[0]) * HW;
  }

  floatx4 acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int CinP = op.CinP, Cin = op.Cin, Npad = op.Npad, kw = op.kw;
  const int spt = CinP >> 2;                       // k-steps of 4 per tap
  const int total = op.kh * kw * spt;
  const int s0 = total * wk / WK, s1 = total * (wk + 1) / WK;
  int tap = s0 / spt, ci = (s0 - tap * spt) * 4;
  const float *__restrict__ wp =
      op.wpk + (size_t)(tap * CinP + ci + kq) * Npad + tn * BN + wn * 16 * FN + row16;
  const bool relu_in = op.pre_relu != 0;

  int aoff[FM];
  bool aval[FM];
  auto setup = [&](int tp) {
    int u = tp / kw, v = tp - u * kw;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      int ih = ih0[fm] + u, iw = iw0[fm] + v;
      aval[fm] = mv[fm] && ih >= 0 && ih < H && iw >= 0 && iw < W;
      aoff[fm] = aval[fm] ? base[fm] + ih * W + iw : 0;
    }
  };
  setup(tap);

  for (int s = s0; s < s1; ++s) {
    const int c = ci + kq;
    const bool cv = c < Cin;
    float av[FM], bv[FN];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      float x = (aval[fm] && cv) ? xin[aoff[fm] + c * HW] : 0.f;
      av[fm] = relu_in ? fmaxf(x, 0.f) : x;
    }
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) bv[fn] = wp[fn * 16];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma16x16x4(av[fm], bv[fn], acc[fm][fn]);
    wp += 4 * Npad;
    ci += 4;
    if (ci == CinP) {
      ci = 0;
      ++tap;
      if (s + 1 < s1) setup(tap);
    }
  }

  // partial sums -> LDS as [wk][col][row]
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int row = wm * 16 * FM + fm * 16 + 4 * kq + j;
        int col = wn * 16 * FN + fn * 16 + row16;
        lds[(wk * BN + col) * LDM + row] = acc[fm][fn][j];
      }
  __syncthreads();
  for (int idx = tid; idx < BM * BN; idx += kThreads) {
    int col = idx / BM, row = idx - col * BM;
    int m = tm * BM + row, n = tn * BN + col;
    if (m >= M || n >= op.Cout) continue;
    float v = op.bias[n];
#pragma unroll
    for (int w = 0; w < WK; ++w) v += lds[(w * BN + col) * LDM + row];
    if (op.post_relu) v = fmaxf(v, 0.f);
    int img = m / howo, pix = m - img * howo;
    *route_ptr(a, op, n, img, pix, howo) = v;
  }
}

// ------------------------------------------------------------------ sepconv

__device__ void sep_tile(const StageArgs &a, const DevOp &op, int t, float *lds) {
  constexpr int BM = kSepBM, LDM = BM + 1, MAXJ = kMaxChannels / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Wo = op.Wo, howo = op.Ho * Wo, M = op.N * howo;
  const int H = op.H, W = op.W, HW = H * W;
  const int CinP = op.CinP, Cin = op.Cin, kh = op.kh, kw = op.kw, taps = kh * kw;
  const int n_in = op.n_in;

  // phase 1: t[c][m] = sum_taps dw[c][tap] * ReLU(sum_i x_i[c][pixel + tap])
  for (int idx = tid; idx < CinP * BM; idx += kThreads) {
    int c = idx / BM, mm = idx - c * BM, m = t * BM + mm;
    float v = 0.f;
    if (c < Cin && m < M) {
      int img = m / howo, r = m - img * howo, oh = r / Wo, ow = r - oh * Wo;
      const float *wdw = op.dw + c * taps;
      for (int u = 0; u < kh; ++u) {
        int ih = oh + u - op.ph;
        if (ih < 0 || ih >= H) continue;
        for (int q = 0; q < kw; ++q) {
          int iw = ow + q - op.pw;
          if (iw < 0 || iw >= W) continue;
          float s = 0.f;
          for (int i = 0; i < n_in; ++i)
            s += a.slot[op.in_slot[i]][(img * op.in_ctot[i] + op.in_coff[i] + c) * HW + ih * W + iw];
          if (op.pre_relu) s = fmaxf(s, 0.f);
          v = fmaf(wdw[u * kw + q], s, v);
        }
      }
    }
    lds[c * LDM + mm] = v;
  }
  __syncthreads();

  // phase 2: pointwise 1x1 on MFMA; wave w owns 16-column blocks w, w+4, ...
  const int NB = op.Npad >> 4;
  const int row16 = lane & 15, kq = lane >> 4;
  floatx4 acc[kSepFM][MAXJ];
#pragma unroll
  for (int fm = 0; fm < kSepFM; ++fm)
#pragma unroll
    for (int j = 0; j < MAXJ; ++j) acc[fm][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < CinP; c0 += 4) {
    float av[kSepFM];
#pragma unroll
    for (int fm = 0; fm < kSepFM; ++fm) av[fm] = lds[(c0 + kq) * LDM + fm * 16 + row16];
    const float *wrow = op.wpk + (size_t)(c0 + kq) * op.Npad + row16;
#pragma unroll
    for (int j = 0; j < MAXJ; ++j) {
      int nb = wave + 4 * j;
      if (nb < NB) {
        float b = wrow[nb * 16];
#pragma unroll
        for (int fm = 0; fm < kSepFM; ++fm) acc[fm][j] = mfma16x16x4(av[fm], b, acc[fm][j]);
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    int nb = wave + 4 * j;
    if (nb < NB) {
#pragma unroll
      for (int fm = 0; fm < kSepFM; ++fm)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          lds[(nb * 16 + row16) * LDM + fm * 16 + 4 * kq + e] = acc[fm][j][e];
    }
  }
  __syncthreads();
  for (int idx = tid; idx < op.Cout * BM; idx += kThreads) {
    int n = idx / BM, mm = idx - n * BM, m = t * BM + mm;
    if (m >= M) continue;
    float v = lds[n * LDM + mm] + op.bias[n];
    if (op.post_relu) v = fmaxf(v, 0.f);
    int img = m / howo, pix = m - img * howo;
    *route_ptr(a, op, n, img, pix, howo) = v;
  }
}

// ------------------------------------------------------------------ elementwise

__device__ void pool_tile(const StageArgs &a, const DevOp &op, int t, bool is_max) {
  const int howo = op.Ho * op.Wo, C = op.Cout, chw = C * howo;
  const int total = op.N * chw, HW = op.H * op.W;
  const float *__restrict__ xin = a.slot[op.in_slot[0]];
  float *__restrict__ out = a.slot[op.route_slot[0]];
  const float inv = 1.0f / (float)(op.kh * op.kw);
  for (int e = 0; e < kEltPerTile / kThreads; ++e) {
    int idx = t * kEltPerTile + e * kThreads + threadIdx.x;
    if (idx >= total) break;
    int img = idx / chw, r = idx - img * chw, c = r / howo, pix = r - c * howo;
    int oh = pix / op.Wo, ow = pix - oh * op.Wo;
    const float *x = xin + (size_t)(img * op.in_ctot[0] + op.in_coff[0] + c) * HW;
    float acc = is_max ? -INFINITY : 0.f;
    for (int u = 0; u < op.kh; ++u) {
      int ih = oh * op.sh + u - op.ph;
      if (ih < 0 || ih >= op.H) continue;
      for (int q = 0; q < op.kw; ++q) {
        int iw = ow * op.sw + q - op.pw;
        if (iw < 0 || iw >= op.W) continue;
        float v = x[ih * op.W + iw];
        acc = is_max ? fmaxf(acc, v) : acc + v;
      }
    }
    if (!is_max) acc *= inv;
    out[(size_t)(img * op.route_ctot[0] + op.route_coff[0] + c) * howo + pix] = acc;
  }
}

__device__ void sum_tile(const StageArgs &a, const DevOp &op, int t, bool mean) {
  const int hw = op.Ho * op.Wo, C = op.Cout, chw = C * hw;
  const int total = op.N * chw;
  float *__restrict__ out = a.slot[op.route_slot[0]];
  for (int e = 0; e < kEltPerTile / kThreads; ++e) {
    int idx = t * kEltPerTile + e * kThreads + threadIdx.x;
    if (idx >= total) break;
    int img = idx / chw, r = idx - img * chw, c = r / hw, pix = r - c * hw;
    float s = 0.f;
    for (int i = 0; i < op.n_in; ++i)
      s += a.slot[op.in_slot[i]][(size_t)(img * op.in_ctot[i] + op.in_coff[i] + c) * hw + pix];
    if (mean) s *= op.inv_n;
    out[(size_t)(img * op.route_ctot[0] + op.route_coff[0] + c) * hw + pix] = s;
  }
}

// ------------------------------------------------------------------ kernel

__global__ __launch_bounds__(kThreads) void ios_stage_kernel(StageArgs a) {
  extern __shared__ float lds[];
  __shared__ int s_ticket;
  const int tid = threadIdx.x;
  int t;
  if (a.use_ticket) {
    if (tid == 0)
      s_ticket = __hip_atomic_fetch_add(&a.ctr[0], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    t = __builtin_amdgcn_readfirstlane(s_ticket);
  } else {
    t = blockIdx.x;
  }
  if (t >= a.n_tiles) {   // only if the counters were not left at zero
    if (tid == 0) __hip_atomic_fetch_or(a.err, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  const Tile tile = a.tiles[t];
  const int opi = __builtin_amdgcn_readfirstlane(tile.op);
  const int ti = __builtin_amdgcn_readfirstlane(tile.idx);
  const DevOp &op = a.ops[opi];

  if (op.n_deps) {
    if (tid == 0) {
      for (int k = 0; k < op.n_deps; ++k) {
        const int d = op.dep[k];
        const int need = a.ops[d].n_tiles;
        int spins = 0;
        while (__hip_atomic_load(&a.ctr[2 + d], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < need) {
          __builtin_amdgcn_s_sleep(2);
          if (++spins > a.spin_limit) {
            __hip_atomic_fetch_or(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
        }
      }
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }

  switch (op.kind) {
    case DK_CONV:
      switch (op.tcfg) {
        case TC_16x16_K4: conv_tile<1, 1, 1, 1, 4>(a, op, ti, lds); break;
        case TC_32x32_K4: conv_tile<2, 2, 1, 1, 4>(a, op, ti, lds); break;
        case TC_64x64: conv_tile<2, 2, 2, 2, 1>(a, op, ti, lds); break;
        default: conv_tile<2, 2, 1, 2, 2>(a, op, ti, lds); break;
      }
      break;
    case DK_SEP: sep_tile(a, op, ti, lds); break;
    case DK_POOL_MAX: pool_tile(a, op, ti, true); break;
    case DK_POOL_AVG: pool_tile(a, op, ti, false); break;
    case DK_ADD: sum_tile(a, op, ti, false); break;
    default: sum_tile(a, op, ti, true); break;
  }

  if (op.signal) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (tid == 0)
      __hip_atomic_fetch_add(&a.ctr[2 + opi], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (a.use_ticket && tid == 0) {
    int f = __hip_atomic_fetch_add(&a.ctr[1], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (f == a.n_tiles - 1) {
      // last tile of the launch: every other workgroup has passed its waits;
      // leave the counters at zero for the next launch on the stream
      for (int i = 0; i < a.n_ops; ++i)
        __hip_atomic_store(&a.ctr[2 + i], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ctr[0], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ctr[1], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

int op_lds_bytes(const DevOp &op) {
  if (op.kind == DK_CONV) {
    TileShape s = tile_shape(op.tcfg);
    return s.wk * tile_bn(op.tcfg) * (tile_bm(op.tcfg) + 1) * (int)sizeof(float);
  }
  if (op.kind == DK_SEP) {
    int c = op.CinP > op.Npad ? op.CinP : op.Npad;
    return c * (kSepBM + 1) * (int)sizeof(float);
  }
  return 0;
}

hipError_t launch_stage(const StageArgs &args, int lds_bytes, hipStream_t stream) {
  hipLaunchKernelGGL(ios_stage_kernel, dim3(args.n_tiles), dim3(kThreads), lds_bytes, stream, args);
  return hipGetLastError();
}

}  // namespace ios
