// The stage kernel: one launch executes every operator of one schedule stage
// (Sec. 3, "Stage" and "Parallelization Strategy").  Each workgroup (512
// threads = 8 wave64) runs one tile; the stage's operators are stored in tile
// order and each owns a contiguous range of workgroup (tile) indices:
//   DK_CONV   implicit-GEMM convolution, M = output pixels, N = output
//             channels, K = taps x input channels (tap-major), on
//             v_mfma_f32_16x16x4_f32; the 8 waves split M, N and/or K and
//             reduce their partial sums through LDS; bias + ReLU are applied
//             in the epilogue, which writes each output channel to its
//             destination (a merged conv has several destinations).
//   DK_SEP    "Relu-SepConv" unit (Table 2): the sum of the inputs, ReLU and
//             the depthwise kxk filter are computed in registers, laid out as
//             the A operand of the pointwise 1x1, which runs on MFMA.
//   DK_POOL_* / DK_ADD / DK_MEAN   elementwise tiles on the vector ALUs.
// Operators of one group run in order (Sec. 3: a group is executed
// sequentially): a consumer tile waits until every tile of its producers has
// finished (see ios_stage_kernel for why the waits always end).
#pragma once
#include <utility>

#include "ios_internal.h"

namespace ios {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// s_waitcnt operand with vmcnt = 0 and the other counters at their maxima
// (gfx9 encoding: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] in [15:14])
constexpr int kWaitVmcnt0 = 0x0F70;
constexpr int kXcds = 8;   // accelerator complex dies of an MI355X

__device__ __forceinline__ floatx4 mfma16x16x4(float a, float b, floatx4 c) {
  // D[16x16] += A[16x4] * B[4x16]; lane l supplies A[l%16][l/16] and
  // B[l/16][l%16]; lane l, element j holds D[4*(l/16)+j][l%16].
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Pointers into the global address space (plain pointers are generic and
// would make the compiler emit flat loads).
typedef __attribute__((address_space(1))) const float gcfloat;
__device__ __forceinline__ gcfloat *gp(const float *p) { return (gcfloat *)p; }

// Raw buffer loads: SGPR resource + 32-bit VGPR offset + SGPR offset, no
// 64-bit address arithmetic per load; an offset at or past the resource's
// size returns 0 (used for padding taps).
constexpr int kBufFlags = 0x00020000;   // gfx9 descriptor word 3 (32-bit data)
// Buffers are smaller than 1 GiB, so a per-lane offset of 2^30 or more reads
// 0.  The range check covers the per-lane (VGPR) offset only, never the
// scalar one: every offset that may leave the buffer goes in the VGPR offset.
constexpr int kOOB = 1 << 30;           // masked pixel / padding tap
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, bytes, kBufFlags);
}
__device__ __forceinline__ float bld(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
__device__ __forceinline__ floatx4 bld4(__amdgpu_buffer_rsrc_t r, int voff) {
  return __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
}

// Biases of a 32x32 MFMA accumulator's channels: lane l holds the bias of
// channel base + l % 32, loaded before the tile's main loop so that its round
// trip overlaps the operand loads; element r of lane l belongs to channel
// base + 8 (r / 4) + 4 (l / 32) + r % 4, taken from that lane by a permute.
__device__ __forceinline__ float bias32_load(const float *bias, int base, int cout, int lane) {
  const int n = base + (lane & 31);
  return bld(rsrc(bias, cout * 4), n < cout ? n * 4 : kOOB, 0);
}
__device__ __forceinline__ float bias32_of(float bl, int r, int lane) {
  const int src = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src * 4, __builtin_bit_cast(int, bl)));
}

// Activation accesses.  COH = true for outputs consumed by another tile of
// the same launch: agent-coherent (sc1) stores, performed beyond the
// XCD-private caches, so no L2 writeback is needed before signalling.
template <bool COH>
__device__ __forceinline__ float ld(const float *p) {
  if constexpr (COH) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else return *p;
}
template <bool COH>
__device__ __forceinline__ void st(float *p, float v) {
  if constexpr (COH) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else *p = v;
}

// Operator descriptors and buffer pointers live in LDS (the workgroup copies
// them there when it starts).  U() reads a field that is the same for every
// lane and moves it to a scalar register, so that descriptors, loop bounds
// and buffer resources stay uniform.
template <class T>
__device__ __forceinline__ T U(const T &v) {
  static_assert(sizeof(T) == 4 || sizeof(T) == 8, "4- or 8-byte fields");
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, v)));
  } else {
    const uint64_t x = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((int)(uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((int)(uint32_t)(x >> 32));
    return __builtin_bit_cast(T, ((uint64_t)hi << 32) | lo);
  }
}

// A descriptor's fields in scalar registers: lane i reads words i, 64 + i,
// ... of the LDS copy, then v_readlane moves word w from lane w % 64 to
// a scalar register (fields the caller never reads are dropped by the
// compiler).  Every lane reading every word would be 64x the LDS traffic.
// Arrays indexed by a run-time value are read from the LDS copy instead
// (U(op.arr[k])), which keeps this copy in registers.
__device__ __forceinline__ DevOp op_scalars(const DevOp &op) {
  constexpr int NW = (kDevOpWords + 63) / 64;   // words per lane
  const int *src = (const int *)&op;
  const int lane = threadIdx.x & 63;
  int v[NW];
#pragma unroll
  for (int j = 0; j < NW; ++j) v[j] = lane + 64 * j < kDevOpWords ? src[lane + 64 * j] : 0;
  DevOp o;
  int *d = (int *)&o;
#pragma unroll
  for (int i = 0; i < kDevOpWords; ++i) d[i] = __builtin_amdgcn_readlane(v[i / 64], i & 63);
  return o;
}

// The launch's buffer pointers (slot -> pointer), staged in LDS.  [] takes a
// slot index that is the same for every lane (LDS read + readfirstlane, which
// stays correct where some lanes are switched off, unlike v_readlane of a
// lane that may be inactive); .p[] takes one that may differ between lanes.
struct Slots {
  float *const *p;
  __device__ __forceinline__ float *operator[](int i) const { return U(p[i]); }
};

// Destination of output column n (the column differs between lanes, so a
// merged conv's route arrays are read per lane; a single route is uniform).
__device__ __forceinline__ float *route_ptr(const Slots &sl, const DevOp &op, const DevOp &o, int n, int img,
                                            int pix, int howo) {
  const int nr = o.n_routes;
  if (nr == 1)
    return sl[o.route_slot[0]] +
           ((size_t)img * o.route_ctot[0] + o.route_coff[0] + n) * howo + pix;
  int r = 0;
  while (r + 1 < nr && n >= op.route_n0[r + 1]) ++r;
  return sl.p[op.route_slot[r]] +
         ((size_t)img * op.route_ctot[r] + op.route_coff[r] + (n - op.route_n0[r])) * howo + pix;
}

// ------------------------------------------------------------------ conv

// n / d for 0 <= n < 2^31 with f = FDiv of d.
__device__ __forceinline__ int fdiv(int n, FDiv f) {
  return (int)((__umulhi((uint32_t)n, f.mul) + (uint32_t)n) >> f.shr);
}

__device__ __forceinline__ floatx4 bld4(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// Implicit-GEMM convolution tile: BM output pixels x BN output channels.
// The reduction runs over k-steps of 4 input channels of one tap (tap-major),
// in groups of 4 k-steps; the WK waves of a column split the groups evenly.
// Per k-step a lane gathers one activation per 16-pixel block (pixel
// lane % 16, channel 4 * step + lane / 16; padding taps and masked pixels
// read 0 through the buffer range check), and per group one 16-byte load
// brings the B operands of four consecutive MFMAs (pack_conv_weights).  A
// wave keeps two chunks of CG groups in registers: the loads of chunk c + 1
// are in flight while chunk c runs on the MFMA unit, and every load is issued
// on a straight path so that each wait only covers the chunk it needs (a
// wave with a single chunk skips the groups past its range instead).
template <int FM, int FN, int WM, int WN, int WK, bool COH, bool RELU, bool FULLC>
__device__ __forceinline__ void conv_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  constexpr int BM = 16 * FM * WM, BN = 16 * FN * WN, LDM = BM + 1;
  constexpr int CG = FM * FN >= 2 ? 2 : 4;     // groups per register chunk
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
  const int wk = wave % WK, wmn = wave / WK, wm = wmn % WM, wn = wmn / WM;
  const int tm = fdiv(t, o.fd_tn), tn = t - tm * o.tiles_n;
  const int Wo = o.Wo, howo = o.Ho * Wo, M = o.N * howo;
  const int H = o.H, W = o.W, HW = H * W;
  const int row16 = lane & 15, kq = lane >> 4;

  // epilogue outputs of this thread; their biases are loaded up front
  constexpr int EPT = (BM * BN + kThreads - 1) / kThreads;
  float bpre[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    int idx = tid + e * kThreads, n = tn * BN + idx / BM;
    bpre[e] = (idx < BM * BN && n < o.Cout) ? o.bias[n] : 0.f;
  }

  // per 16-pixel block: offset of this lane's pixel (channel kq, tap 0,0)
  // and the taps whose input row / column lies inside the image
  const int kh = o.kh, kw = o.kw;
  int pix[FM], rv[FM], cv[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int m = tm * BM + wm * 16 * FM + fm * 16 + row16;
    const bool ok = m < M;
    const int mm = ok ? m : 0;
    const int img = fdiv(mm, o.fd_howo), r = mm - img * howo, oh = fdiv(r, o.fd_wo), ow = r - oh * Wo;
    const int ih0 = oh * o.sh - o.ph, iw0 = ow * o.sw - o.pw;
    pix[fm] = (img * o.in_ctot[0] + o.in_coff[0] + kq) * HW + ih0 * W + iw0;
    int rb = 0, cb = 0;
    for (int u = 0; u < kh; ++u) rb |= (ok && ih0 + u >= 0 && ih0 + u < H) << u;
    for (int v = 0; v < kw; ++v) cb |= (iw0 + v >= 0 && iw0 + v < W) << v;
    rv[fm] = rb;
    cv[fm] = cb;
  }

  floatx4 acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int spt = o.CinP >> 2, NG = o.NG;
  const int g0 = NG * wk / WK, g1 = NG * (wk + 1) / WK;
  const int nc = (g1 - g0 + CG - 1) / CG;
  const __amdgpu_buffer_rsrc_t xr = rsrc(sl[o.in_slot[0]], o.in_bytes[0]);
  const __amdgpu_buffer_rsrc_t wr = rsrc(o.wpk, o.w_bytes);
  const int HW16 = HW * 16;                        // bytes between k-steps (4 channels)
  const int cmax = o.Cin - kq;                    // channel 4 * cs + kq exists iff 4 * cs < cmax
  // per-lane byte offset of each 16-column block's groups (kOOB for blocks
  // past the packed ones, i.e. columns past Cout)
  const int nblk = o.Npad >> 4;
  int nbv[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int nb = (tn * WN + wn) * FN + fn;
    nbv[fn] = nb < nblk ? nb * NG * 1024 + lane * 16 : kOOB;
  }

  // walk of (tap row u, tap column v, channel step cs) over the k-steps, in
  // load order, starting at this wave's first group; toff[fm] is the byte
  // offset of this lane's input, channel kq, for the current tap (kOOB
  // outside the image and past the last tap) and w_ka the uniform offset of
  // channel step cs.  A load takes toff in its per-lane offset, which the
  // buffer range check covers, and w_ka in its scalar offset, which it does
  // not: a lane either reads inside the buffer (a valid tap and channel) or
  // has a per-lane offset past its end, so no unchecked address leaves it.
  int w_tap = fdiv(4 * g0, o.fd_spt);
  int w_cs = 4 * g0 - w_tap * spt;
  int w_u = fdiv(w_tap, o.fd_kw), w_v = w_tap - w_u * kw;
  int w_ka = w_cs * HW16;
  int toff[FM];
  auto set_tap = [&]() {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
      toff[fm] = (w_u < kh && ((rv[fm] >> w_u) & (cv[fm] >> w_v) & 1)) ? (pix[fm] + w_u * W + w_v) * 4 : kOOB;
  };
  set_tap();

  typedef float AChunk[4 * CG][FM];
  typedef floatx4 BChunk[CG][FN];
  // A of groups past the wave's range is loaded but never used (compute
  // stops at g1), and k-steps past the last tap read 0 (their B is 0 too).
  auto load = [&](AChunk &A, BChunk &B, int gb, bool last) {
#pragma unroll
    for (int gi = 0; gi < CG; ++gi) {
      const int g = gb + gi;
      const bool gok = g < g1;                     // uniform
      if (last && !gok) break;                     // nothing is loaded after this chunk
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
          int off = toff[fm];
          if constexpr (!FULLC) off = 4 * w_cs < cmax ? off : kOOB;   // channel past Cin
          A[gi * 4 + s][fm] = bld(xr, off, w_ka);
        }
        w_ka += HW16;
        if (++w_cs == spt) {
          w_cs = 0;
          w_ka = 0;
          if (++w_v == kw) { w_v = 0; ++w_u; }
          set_tap();
        }
      }
      const int kb = gok ? g * 1024 : kOOB;        // uniform
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) B[gi][fn] = bld4(wr, (int)((uint32_t)nbv[fn] + (uint32_t)kb), 0);
    }
  };
  auto compute = [&](const AChunk &A, const BChunk &B, int gb) {
#pragma unroll
    for (int gi = 0; gi < CG; ++gi) {
      if (gb + gi >= g1) break;                    // uniform
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
          const float a = RELU ? fmaxf(A[gi * 4 + s][fm], 0.f) : A[gi * 4 + s][fm];
#pragma unroll
          for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = mfma16x16x4(a, B[gi][fn][s], acc[fm][fn]);
        }
    }
  };
  AChunk A0, A1;
  BChunk B0, B1;
  if (nc == 1) {
    load(A0, B0, g0, true);
    compute(A0, B0, g0);
  } else if (nc > 1) {
    load(A0, B0, g0, false);
    load(A1, B1, g0 + CG, false);
    for (int c = 0;; c += 2) {
      compute(A0, B0, g0 + c * CG);
      if (c + 2 >= nc) {
        compute(A1, B1, g0 + (c + 1) * CG);
        break;
      }
      load(A0, B0, g0 + (c + 2) * CG, false);
      compute(A1, B1, g0 + (c + 1) * CG);
      if (c + 3 >= nc) {
        compute(A0, B0, g0 + (c + 2) * CG);
        break;
      }
      load(A1, B1, g0 + (c + 3) * CG, false);
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
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    int idx = tid + e * kThreads;
    int col = idx / BM, row = idx - col * BM;
    int m = tm * BM + row, n = tn * BN + col;
    if (idx >= BM * BN || m >= M || n >= o.Cout) continue;
    float v = bpre[e];
#pragma unroll
    for (int w = 0; w < WK; ++w) v += lds[(w * BN + col) * LDM + row];
    if (o.post_relu) v = fmaxf(v, 0.f);
    int img = fdiv(m, o.fd_howo), pix_ = m - img * howo;
    st<COH>(route_ptr(sl, op, o, n, img, pix_, howo), v);
  }
}

// ------------------------------------------------------------------ pipelined conv

// Direct global -> LDS load of one float per lane: lane i of the wave writes
// l[i] (l the same for every lane), through no register.  The compiler does
// not see this write: readers wait for vmcnt(0) (and a barrier) first.
typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ void lds_dma(__amdgpu_buffer_rsrc_t r, float *l, int voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)l, 4, voff, 0, 0, 0);
}


typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ floatx16 mfma32x32x2(float a, float b, floatx16 c) {
  // D[32x32] += A[32x2] * B[2x32]; lane l supplies A[l%32][l/32] and
  // B[l/32][l%32]; lane l, element r holds D[8 (r/4) + 4 (l/32) + r%4][l%32].
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// s_waitcnt with vmcnt = N (gfx9 encoding, see kWaitVmcnt0), other counters free.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}
// Workgroup barrier for loops that keep direct-to-LDS loads in flight across
// it.  __syncthreads() carries a release fence, for which the compiler waits
// for every load in flight (vmcnt(0)), which would drain the whole ring at
// each block.  Here each wave has already waited for its own loads of the
// block about to be read (explicit vmcnt), and its LDS reads are complete
// (lgkmcnt(0)); the memory clobber keeps the compiler from moving LDS
// accesses across the barrier.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Implicit-GEMM convolution tile with both operands staged in LDS through a
// ring of direct global -> LDS loads: BM = 32 WMW output pixels (over the
// whole batch, flattened) x BN = 32 WNW output channels, 8 waves of one
// 32x32 block each on v_mfma_f32_32x32x2_f32 (output channels as rows,
// pixels as columns).  The reduction index k = (u kw + v) Cin + c runs in
// blocks of KB = kPipeKB channels of one tap (Cin is a multiple of KB, so
// a block never spans two taps).  A ring of kPipeStages slots holds, per
// block, the weights [KB][BN] (rows of the packed [k][n] matrix) and the
// im2col'd input [KB][BM]; kPipeStages - 1 blocks are in flight while one
// is multiplied, one barrier per block.
//
// Every load's address is a per-lane part fixed for a tap (the pixel's tap
// offset, or an out-of-range marker where the tap falls outside the image,
// which the buffer range check turns into 0) plus a uniform part in the
// scalar offset (the channel row, or the block's weight rows), which the
// range check does not cover: a lane either reads an element of the input
// or 0.  The walk over (tap, channel) is scalar; per block a wave spends no
// vector instruction on addresses.  The writes to LDS go through no
// register and the compiler does not see them: every wave counts its own
// loads (vmcnt) and the barrier publishes them.
template <int WMW, bool COH>
__device__ __forceinline__ void conv_pipe_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  constexpr int WNW = kWaves / WMW, BM = 32 * WMW, BN = 32 * WNW, KB = kPipeKB, D = kPipeStages;
  constexpr int HB = BM / 64;                        // 64-pixel segments of a row of the input block
  constexpr int A_DMA = KB * BN / 64 / kWaves, B_DMA = KB * BM / 64 / kWaves, PER = A_DMA + B_DMA;
  static_assert(A_DMA * 64 * kWaves == KB * BN && B_DMA * 64 * kWaves == KB * BM, "whole copies");
  static_assert(B_DMA == 2 * HB, "each wave stages two rows of the input block");
  static_assert((D & (D - 1)) == 0 && (D - 2) * PER < 64, "ring of 2^n slots; vmcnt is 6 bits");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WMW, wn = wave / WMW;
  const int tm = fdiv(t, o.fd_tn), tn = t - tm * o.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int Wo = o.Wo, howo = o.Ho * Wo, M = o.N * howo, H = o.H, W = o.W;
  const int Cin = o.Cin, kw = o.kw, nkb = o.NG, ldw = o.pipe_ldw;
  const int hw4 = H * W * 4;
  float *aring = lds, *bring = lds + D * KB * BN;

  // this lane's pixels of the input block (segment h: pixel m0 + 64 h + lane):
  // offset of tap (0, 0) of channel 0, and the taps inside the image (bit u kw + v)
  int pbase[HB];
  uint32_t tmask[HB];
#pragma unroll
  for (int h = 0; h < HB; ++h) {
    const int m = m0 + 64 * h + lane;
    pbase[h] = 0;
    tmask[h] = 0;
    if (m < M) {
      const int img = fdiv(m, o.fd_howo), r = m - img * howo, oh = fdiv(r, o.fd_wo), ow = r - oh * Wo;
      const int ih0 = oh * o.sh - o.ph, iw0 = ow * o.sw - o.pw;
      pbase[h] = ((img * o.in_ctot[0] + o.in_coff[0]) * H + ih0) * W + iw0;
      uint32_t cm = 0;
      for (int v = 0; v < kw; ++v) cm |= (uint32_t)(iw0 + v >= 0 && iw0 + v < W) << v;
      for (int u = 0; u < o.kh; ++u)
        if (ih0 + u >= 0 && ih0 + u < H) tmask[h] |= cm << (u * kw);
    }
  }
  // per lane, byte offset of its weight element in each of its copies of a block
  int aoff[A_DMA];
#pragma unroll
  for (int i = 0; i < A_DMA; ++i) {
    const int f = (wave * A_DMA + i) * 64 + lane;
    aoff[i] = ((f / BN) * ldw + n0 + f % BN) * 4;
  }
  const __amdgpu_buffer_rsrc_t xr = rsrc(sl[o.in_slot[0]], o.in_bytes[0]);
  const __amdgpu_buffer_rsrc_t wr = rsrc(o.wpk, o.w_bytes);
  const float bl = bias32_load(o.bias, n0 + wn * 32, o.Cout, lane);

  // scalar walk of the next block to issue: tap (u, v), first channel c
  int tap = 0, tu = 0, tv = 0, c = 0;
  int toff[HB];
  auto set_tap = [&]() {
#pragma unroll
    for (int h = 0; h < HB; ++h) toff[h] = (tmask[h] >> tap) & 1 ? (pbase[h] + tu * W + tv) * 4 : kOOB;
  };
  set_tap();
  auto issue = [&](int kb) {
    const int slot = kb & (D - 1);
    float *a = aring + slot * KB * BN, *b = bring + slot * KB * BM;
    const int wsoff = kb * KB * ldw * 4;
#pragma unroll
    for (int i = 0; i < A_DMA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void *)(a + (wave * A_DMA + i) * 64), 4, aoff[i], wsoff, 0, 0);
#pragma unroll
    for (int i = 0; i < B_DMA; ++i) {
      const int r = 2 * wave + i / HB, h = i % HB;   // block row, 64-pixel segment
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void *)(b + r * BM + h * 64), 4, toff[h], (c + r) * hw4, 0, 0);
    }
    c += KB;
    if (c == Cin) {                                  // uniform: next tap
      c = 0;
      ++tap;
      if (++tv == kw) { tv = 0; ++tu; }
      set_tap();
    }
  };

  floatx16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  for (int kb = 0; kb < D - 1 && kb < nkb; ++kb) issue(kb);
  const float *a_l = aring + (lane >> 5) * BN + wn * 32 + (lane & 31);
  const float *b_l = bring + (lane >> 5) * BM + wm * 32 + (lane & 31);
  for (int kb = 0; kb < nkb; ++kb) {
    // this wave's loads of block kb have landed once at most those of the
    // blocks issued after it are in flight; the barrier makes every wave's
    // visible and guarantees that block kb - 1's slot is no longer read
    if (kb + D - 2 < nkb) wait_vmcnt<(D - 2) * PER>();
    else wait_vmcnt<0>();
    ring_barrier();
    if (kb + D - 1 < nkb) issue(kb + D - 1);
    const int slot = kb & (D - 1);
    const float *a = a_l + slot * KB * BN, *b = b_l + slot * KB * BM;
    float av[KB / 2], bv[KB / 2];
#pragma unroll
    for (int p = 0; p < KB / 2; ++p) {
      av[p] = a[2 * p * BN];
      bv[p] = b[2 * p * BM];
    }
    __builtin_amdgcn_sched_barrier(0);               // every read of the block in flight before the first MFMA
#pragma unroll
    for (int p = 0; p < KB / 2; ++p) acc = mfma32x32x2(av[p], bv[p], acc);
  }
  // epilogue: element r of lane l is channel n0 + 32 wn + 8 (r/4) + 4 (l/32) + r%4 of pixel m0 + 32 wm + l%32
  const int m = m0 + wm * 32 + (lane & 31);
  float bv16[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) bv16[r] = bias32_of(bl, r, lane);
  if (m < M) {
    const int img = fdiv(m, o.fd_howo), pix = m - img * howo;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int n = n0 + wn * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (n < o.Cout) {
        float v = acc[r] + bv16[r];
        if (o.post_relu) v = fmaxf(v, 0.f);
        st<COH>(route_ptr(sl, op, o, n, img, pix, howo), v);
      }
    }
  }
}

// Implicit-GEMM convolution tile in which every wave streams its own
// operands through a private ring in LDS: BM = 32 WMW output pixels (over
// the whole batch, flattened) x BN = 32 WNW output channels, 8 waves of one
// 32x32 block each on v_mfma_f32_32x32x2_f32 (output channels as rows,
// pixels as columns).  The reduction index k = (u kw + v) Cin + c runs in
// blocks of KB = kWaveKB channels of one tap (Cin is a multiple of KB, so a
// block never spans two taps).  Per block a wave copies, with direct
// global -> LDS loads, its weights A[32 ch][KB] and its im2col'd input
// B[KB][32 px]: one load per k-pair and operand, lane i fetching the element
// (k = 2 p + i / 32, ch or px = i % 32) that lane i of the MFMA of k-pair p
// supplies, so the operand reads are conflict-free.  Each wave keeps
// kWaveStages - 1 blocks in flight while it multiplies one and waits only for
// its own loads (vmcnt): there is no barrier in the reduction, and the two
// waves of a SIMD run independently, each hiding the other's waits.
//
// Every load's address is a per-lane part (the pixel's offset for the tap,
// or an out-of-range marker where the tap falls outside the image, which the
// buffer range check turns into 0; the weight column) plus a uniform part in
// the scalar offset (the channel row; the block's weight rows), which the
// range check does not cover: a lane reads an element of its tensor or 0.
// The walk over (tap, channel) is scalar, so a block costs a wave no vector
// instruction for addresses.  The writes to LDS go through no register and
// the compiler does not see them: the memory clobbers order the reads.
template <int WMW, bool COH>
__device__ __forceinline__ void conv_wave_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  constexpr int WNW = kWaves / WMW, BM = 32 * WMW, BN = 32 * WNW, KB = kWaveKB, D = kWaveStages;
  static_assert(kPipeKB % KB == 0, "weights packed in blocks of kPipeKB rows");
  constexpr int NP = KB / 2;                         // k-pairs (MFMAs) per block
  constexpr int SLOT = 2 * NP * 64;                  // floats per slot: A then B, 64 per k-pair
  static_assert((D - 2) * 2 * NP < 64, "vmcnt is 6 bits");
  const int tid = threadIdx.x, lane = tid & 63, kq = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WMW, wn = wave / WMW;
  const int tm = fdiv(t, o.fd_tn), tn = t - tm * o.tiles_n;
  const int Wo = o.Wo, howo = o.Ho * Wo, M = o.N * howo, H = o.H, W = o.W;
  const int Cin = o.Cin, kw = o.kw, nkb = o.NG * (kPipeKB / KB), ldw = o.pipe_ldw, hw4 = H * W * 4;
  const int m = tm * BM + wm * 32 + l32, n0 = tn * BN + wn * 32;
  float *ring = lds + wave * D * SLOT;

  // this lane's pixel: offset of tap (0, 0) in channel kq, taps inside the
  // image (bit u kw + v); its weight column in channel row kq
  int pbase = 0;
  uint32_t tmask = 0;
  if (m < M) {
    const int img = fdiv(m, o.fd_howo), r = m - img * howo, oh = fdiv(r, o.fd_wo), ow = r - oh * Wo;
    const int ih0 = oh * o.sh - o.ph, iw0 = ow * o.sw - o.pw;
    pbase = ((img * o.in_ctot[0] + o.in_coff[0] + kq) * H + ih0) * W + iw0;
    uint32_t cm = 0;
    for (int v = 0; v < kw; ++v) cm |= (uint32_t)(iw0 + v >= 0 && iw0 + v < W) << v;
    for (int u = 0; u < o.kh; ++u)
      if (ih0 + u >= 0 && ih0 + u < H) tmask |= cm << (u * kw);
  }
  const int aoff = (kq * ldw + n0 + l32) * 4;
  const __amdgpu_buffer_rsrc_t xr = rsrc(sl[o.in_slot[0]], o.in_bytes[0]);
  const __amdgpu_buffer_rsrc_t wr = rsrc(o.wpk, o.w_bytes);
  const float bl = bias32_load(o.bias, n0, o.Cout, lane);

  // scalar walk of the next block to issue: tap (u, v), first channel c
  int tap = 0, tu = 0, tv = 0, c = 0;
  int toff = tmask & 1 ? pbase * 4 : kOOB;
  auto issue = [&](int kb) {
    float *s = ring + (kb & (D - 1)) * SLOT;
    const int wrow = kb * KB * ldw * 4;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void *)(s + p * 64), 4, aoff, wrow + 2 * p * ldw * 4, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void *)(s + (NP + p) * 64), 4, toff, (c + 2 * p) * hw4, 0, 0);
    }
    c += KB;
    if (c == Cin) {                                  // uniform: next tap
      c = 0;
      ++tap;
      if (++tv == kw) { tv = 0; ++tu; }
      toff = (tmask >> tap) & 1 ? (pbase + tu * W + tv) * 4 : kOOB;
    }
  };

  floatx16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  for (int kb = 0; kb < D - 1 && kb < nkb; ++kb) issue(kb);
  for (int kb = 0; kb < nkb; ++kb) {
    // block kb has landed once at most the blocks issued after it are in
    // flight; its slot's reads below come after the wait
    if (kb + D - 2 < nkb) wait_vmcnt<(D - 2) * 2 * NP>();
    else wait_vmcnt<0>();
    asm volatile("" ::: "memory");
    // block kb - 1's slot was read (and consumed) in the previous round
    if (kb + D - 1 < nkb) issue(kb + D - 1);
    const float *s = ring + (kb & (D - 1)) * SLOT + lane;
    float av[NP], bv[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      av[p] = s[p * 64];
      bv[p] = s[(NP + p) * 64];
    }
    __builtin_amdgcn_sched_barrier(0);               // every read of the block in flight before the first MFMA
#pragma unroll
    for (int p = 0; p < NP; ++p) acc = mfma32x32x2(av[p], bv[p], acc);
    asm volatile("" ::: "memory");
  }
  // epilogue: element r of lane l is channel n0 + 8 (r/4) + 4 (l/32) + r%4 of pixel m
  float bv16[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) bv16[r] = bias32_of(bl, r, lane);
  if (m < M) {
    const int img = fdiv(m, o.fd_howo), pix = m - img * howo;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int n = n0 + 8 * (r >> 2) + 4 * kq + (r & 3);
      if (n < o.Cout) {
        float v = acc[r] + bv16[r];
        if (o.post_relu) v = fmaxf(v, 0.f);
        st<COH>(route_ptr(sl, op, o, n, img, pix, howo), v);
      }
    }
  }
}

// ------------------------------------------------------------------ sepconv

// One depthwise output from staged rows: tap (u, v) at column iw0 + v of row
// xrow + u W, columns outside the image counting zero.  Every LDS read of
// the window (inputs and weights) is issued before the first product: one
// LDS round trip per output.
template <int KH, int KW>
__device__ __forceinline__ float dw_point(const float *xrow, const float *w, int iw0, int W, float d = 0.f) {
  float x[KH * KW], c[KH * KW];
#pragma unroll
  for (int u = 0; u < KH; ++u)
#pragma unroll
    for (int v = 0; v < KW; ++v) {
      const int iw = iw0 + v;
      const bool ok = iw >= 0 && iw < W;
      x[u * KW + v] = xrow[u * W + (ok ? iw : 0)];
      c[u * KW + v] = ok ? w[u * KW + v] : 0.f;
    }
#pragma unroll
  for (int i = 0; i < KH * KW; ++i) d = fmaf(c[i], x[i], d);
  return d;
}

// The pointwise MFMAs of one SEPCONV chunk for a wave with NP (pixel block,
// channel block) pairs: per group of 4 k-steps, the NP A operands (16 bytes
// per lane each) and the 4 B values are read from LDS together, then the
// 4 NP MFMAs run (one LDS round trip per group, no branch between MFMAs).
template <int NP>
__device__ __forceinline__ void sep_mma(floatx4 *acc, const float *as, const float *bs, int c, int gpc, int NG,
                                        int pitch, int wave, int MB, int mb, int lane) {
  for (int gi = 0; gi < gpc; ++gi) {
    if (c * gpc + gi >= NG) break;                   // uniform: a short last chunk
    floatx4 a[NP];
    float b[4];
#pragma unroll
    for (int r = 0; r < NP; ++r) a[r] = *(const floatx4 *)(as + (((wave + r * kWaves) / MB) * gpc + gi) * 256 + lane * 4);
#pragma unroll
    for (int s = 0; s < 4; ++s) b[s] = bs[(gi * 16 + 4 * s + (lane >> 4)) * pitch + mb * 16 + (lane & 15)];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int r = 0; r < NP; ++r) acc[r] = mfma16x16x4(a[r][s], b[s], acc[r]);
  }
}

// "Relu-SepConv" unit (Table 2): sum of the inputs -> ReLU -> depthwise
// kh x kw (stride 1, no bias) -> pointwise 1x1 (+ bias), on BM = sep_bm
// consecutive output pixels of one image (flattened, so a tile may span
// image rows) x sep_nbt blocks of 16 output channels.  The reduction over
// input channels runs in chunks of CK = sep_ck channels.  Everything a chunk
// needs arrives in one batch of loads, issued while the previous chunk runs
// on the MFMA units:
//   - the input rows its pixels read (the window's halo included; rows
//     outside the image staged as zeros) and its depthwise weights:
//     coalesced loads to registers, stored to LDS once the previous chunk's
//     MFMAs are issued (one LDS buffer: the previous chunk's depthwise pass
//     has finished by then); the inputs after the first (a RandWire node's
//     other producers) are loaded and added at that point, then the sum is
//     ReLU'd;
//   - its pointwise weights (packed like a 1x1 conv's: per 16-channel output
//     block and group of 4 k-steps, 64 lanes x 4 floats): 16-byte loads to
//     registers, then LDS (two buffers, as the MFMAs read the previous
//     chunk's meanwhile).
// Then
//   dw      every (pixel, channel) of the chunk from LDS -> Bs[channel][pixel];
//   mfma    output channels as MFMA rows, pixels as columns:
//           D[16 ch][16 px] += A[16 ch][4 k] B[4 k][16 px], A and B both read
//           from LDS.  Wave w owns the (pixel block, channel block) pairs w,
//           w + 8, ...; as the tile's pixel-block count divides 8 they share
//           one pixel block, so one Bs read feeds every MFMA of the wave.
// A thread's staging elements and depthwise outputs sit at the same places
// of every chunk, so their index arithmetic is done once per tile.  The
// epilogue adds the bias (staged with the first chunk) and writes each
// accumulator row straight to the output: 16 lanes hold 16 consecutive
// pixels of one channel.
template <bool COH>
__device__ __forceinline__ void sep_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int BM = o.sep_bm, LBM = o.sep_lbm, MB = BM >> 4, CK = o.sep_ck, W = o.W, H = o.H;
  const int Wo = o.Wo, howo = o.Ho * Wo, kh = o.kh, kw = o.kw, KK = kh * kw, HW = H * W;
  const int tm = fdiv(t, o.fd_tn), tn = t - tm * o.tiles_n;
  const int img = fdiv(tm, o.fd_pimg), p0 = (tm - img * o.tiles_per_plane) * BM;
  const int oh0 = fdiv(p0, o.fd_wo), r_lo = oh0 - o.ph;   // first staged input row (may be < 0)
  const int RW = o.sep_rows * W, plane = CK * RW;   // staged floats per channel / per chunk
  const int n_chunks = o.sep_nck, NG = o.NG, gpc = CK >> 4, NBT = o.sep_nbt, Cin = o.Cin;
  const int nb0 = tn * NBT, nbc = min(NBT, (o.Npad >> 4) - nb0);
  const int ablk = NBT * gpc * 256;                  // pointwise weights of one chunk (floats)
  const int pitch = sep_pitch(BM);
  float *xs = lds, *wd = xs + plane;
  float *as0 = wd + CK * KK, *as1 = as0 + ablk;
  float *bs = as1 + ablk, *bias = bs + CK * pitch;
  const int mb = wave & (MB - 1);                   // this wave's pixel block
  int np = 0;                                        // pairs of this wave: channel blocks nb0 + (wave + 8 r) / MB
  for (int i = wave; i < MB * nbc && np < kSepPairs; i += kWaves) ++np;
  np = __builtin_amdgcn_readfirstlane(np);

  // staging: element e = tid + 512 j of a chunk's CK x rows x W block
  // (channel, staged row, column) lies at soff[j] of the chunk's first input
  // channel, or outside the image / block (-1)
  constexpr int SE = kSepStagePerThread;
  const int ne = (plane + kThreads - 1) >> 9, nw = (CK * KK + kThreads - 1) >> 9;
  int soff[SE];
#pragma unroll
  for (int j = 0; j < SE; ++j) {
    const int e = tid + j * kThreads;
    const int ch = fdiv(e, o.fd_rw), rem = e - ch * RW;
    const int sr = fdiv(rem, o.fd_w), col = rem - sr * W, ih = r_lo + sr;
    soff[j] = (j < ne && e < plane && ih >= 0 && ih < H) ? ch * HW + ih * W + col : -1;
  }
  float sv[SE], wv[kSepDwPerThread];
  auto issue = [&](int c, int k, float (&dst)[SE]) {
    const __amdgpu_buffer_rsrc_t xr = rsrc(sl[U(op.in_slot[k])], U(op.in_bytes[k]));
    const int base = (img * U(op.in_ctot[k]) + U(op.in_coff[k]) + c * CK) * HW;
    const int elim = min(plane, (Cin - c * CK) * RW);   // elements of channels that exist
#pragma unroll
    for (int jb = 0; jb < SE; jb += 4) {
      if (jb >= ne) break;                           // uniform
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int j = jb + jj, e = tid + j * kThreads;
        dst[j] = bld(xr, soff[j] >= 0 && e < elim ? (soff[j] + base) * 4 : kOOB, 0);
      }
    }
  };
  const __amdgpu_buffer_rsrc_t wr = rsrc(o.wpk, o.w_bytes), dr = rsrc(o.dw, o.dw_bytes);
  // pointwise weights of chunk c: float4 f = tid + 512 k of the chunk's
  // nbc x gpc blocks (nb, g) of 64 lanes x 4 floats, to registers now and to
  // LDS with the inputs (groups past the packed ones read 0, never used)
  const int na4 = nbc * gpc * 64;
  floatx4 av[kSepAPerThread];
  auto stage_issue = [&](int c) {
#pragma unroll
    for (int k = 0; k < kSepAPerThread; ++k) {
      const int f = tid + k * kThreads, bi = f >> 6, nbl = bi / gpc, gl = bi - nbl * gpc, g = c * gpc + gl;
      av[k] = bld4(wr, f < na4 && g < NG ? (((nb0 + nbl) * NG + g) * 64 + (f & 63)) * 16 : kOOB, 0);
    }
    issue(c, 0, sv);
#pragma unroll
    for (int j = 0; j < kSepDwPerThread; ++j) {
      if (j >= nw) break;
      const int e = tid + j * kThreads;
      wv[j] = bld(dr, e < CK * KK ? (c * CK * KK + e) * 4 : kOOB, 0);   // past the buffer: 0
    }
  };
  auto stage_store = [&](int c, float *as) {
    for (int k = 1; k < o.n_in; ++k) {              // a RandWire node's further producers
      float sx[SE];
      issue(c, k, sx);
#pragma unroll
      for (int j = 0; j < SE; ++j) sv[j] += sx[j];
    }
#pragma unroll
    for (int j = 0; j < SE; ++j) {
      if (j >= ne) break;
      const int e = tid + j * kThreads;
      if (e < plane) xs[e] = o.pre_relu ? fmaxf(sv[j], 0.f) : sv[j];
    }
#pragma unroll
    for (int j = 0; j < kSepDwPerThread; ++j) {
      if (j >= nw) break;
      const int e = tid + j * kThreads;
      if (e < CK * KK) wd[e] = wv[j];
    }
#pragma unroll
    for (int k = 0; k < kSepAPerThread; ++k) {
      const int f = tid + k * kThreads;
      if (f < na4) *(floatx4 *)(as + f * 4) = av[k];
    }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);        // the biases' copy to LDS has landed
  };

  // depthwise: this thread's pixel p (the same in every pass, as BM divides
  // 512) and channels ch0 + i 512 / BM of each chunk
  const int p = tid & (BM - 1), ch0 = tid >> LBM, chs = kThreads >> LBM;
  const int qd = p0 + p;
  const bool qv = qd < howo;
  int xq = 0, iw0 = 0;
  if (qv) {
    const int oh = fdiv(qd, o.fd_wo), ow = qd - oh * Wo;
    xq = (oh - oh0) * W;
    iw0 = ow - o.pw;
  }

  floatx4 acc[kSepPairs];
#pragma unroll
  for (int r = 0; r < kSepPairs; ++r) acc[r] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (wave == 0) {                                   // the tile's biases, with the first chunk
    const __amdgpu_buffer_rsrc_t br = rsrc(o.bias, o.Npad * 4);
    for (int e = 0; e < nbc * 16; e += 64) lds_dma(br, bias + e, (nb0 * 16 + e + lane) * 4);
  }
  stage_issue(0);
  stage_store(0, as0);
  __syncthreads();
  for (int c = 0; c < n_chunks; ++c) {
    const float *as = (c & 1) ? as1 : as0;
    for (int ch = ch0; ch < CK; ch += chs) {
      float d = 0.f;
      if (qv) {
        const float *xrow = xs + ch * RW + xq, *w = wd + ch * KK;
        if (kh == 3 && kw == 3) d = dw_point<3, 3>(xrow, w, iw0, W);
        else if (kh == 5 && kw == 5) {                // rows 0-2, then 3-4 (bounds the registers)
          d = dw_point<3, 5>(xrow, w, iw0, W);
          __builtin_amdgcn_sched_barrier(0);
          d = dw_point<2, 5>(xrow + 3 * W, w + 15, iw0, W, d);
        }
        else
          for (int u = 0; u < kh; ++u)
            for (int v = 0; v < kw; ++v)
              if (iw0 + v >= 0 && iw0 + v < W) d = fmaf(w[u * kw + v], xrow[u * W + iw0 + v], d);
      }
      bs[ch * pitch + p] = d;
    }
    __syncthreads();
    if (c + 1 < n_chunks) stage_issue(c + 1);        // in flight during the MFMAs
    // pointwise on MFMA over the chunk's groups of 4 k-steps (16 channels)
    static_assert(kSepPairs == 4, "one case per pair count");
    switch (np) {
      case 1: sep_mma<1>(acc, as, bs, c, gpc, NG, pitch, wave, MB, mb, lane); break;
      case 2: sep_mma<2>(acc, as, bs, c, gpc, NG, pitch, wave, MB, mb, lane); break;
      case 3: sep_mma<3>(acc, as, bs, c, gpc, NG, pitch, wave, MB, mb, lane); break;
      case 4: sep_mma<4>(acc, as, bs, c, gpc, NG, pitch, wave, MB, mb, lane); break;
      default: break;
    }
    if (c + 1 < n_chunks) stage_store(c + 1, (c & 1) ? as0 : as1);
    __syncthreads();
  }
  // epilogue: lane l, element j holds channel nb 16 + 4 (l / 16) + j of pixel mb 16 + l % 16
  const int q = p0 + mb * 16 + (lane & 15);
  float *out = sl[o.route_slot[0]];
#pragma unroll
  for (int r = 0; r < kSepPairs; ++r) {
    if (r >= np) break;
    const int nbl = (wave + r * kWaves) / MB;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int nl = nbl * 16 + 4 * (lane >> 4) + j, n = nb0 * 16 + nl;
      if (n < o.Cout && q < howo) {
        float v = acc[r][j] + bias[nl];
        if (o.post_relu) v = fmaxf(v, 0.f);
        st<COH>(out + ((size_t)img * o.route_ctot[0] + o.route_coff[0] + n) * howo + q, v);
      }
    }
  }
}


// Cross-lane moves inside each row of 16 lanes (DPP): lane i of a row takes
// the value of lane i + N (from_right) or lane i - N (from_left) of the same
// row, and 0 where that lane lies outside the row.
template <int N>
__device__ __forceinline__ float from_right(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                0x100 + N, 0xF, 0xF, true));
}
template <int N>
__device__ __forceinline__ float from_left(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                0x110 + N, 0xF, 0xF, true));
}

// Taps 1 .. K-1 of one window row: tap v of pixel j is column j + v of the
// row segment, i.e. lane j + v's first value or lane j + v - 16's second.
template <int... V>
__device__ __forceinline__ float dw_taps(const float *w, float xa, float xb, float d,
                                         std::integer_sequence<int, V...>) {
  ((d = fmaf(w[V + 1], from_right<V + 1>(xa) + from_left<15 - V>(xb), d)), ...);
  return d;
}

// Waits for this wave's direct-to-LDS loads (the compiler does not see
// their writes).
__device__ __forceinline__ void lds_dma_wait() {
  __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// "Relu-SepConv" unit, row tile (the alternative to the staged tile above,
// chosen per operator by measurement): 16 output pixels of one output row x
// sep_nbt blocks of 16 output channels.
//
// Lane l = 16 g + j of a wave computes the depthwise output of pixel j for
// channel 4 ks + g: exactly the A operand lane l gives the 16x16x4 MFMA at
// k-step ks, so depthwise results never leave registers.  Per window row a
// lane loads two inputs, columns j and 16 + j of the row segment the 16
// pixels read; the K taps of pixel j are then gathered from lanes j .. j+K-1
// of its row with DPP shifts.  The 8 waves split the input channels (k-steps
// of 4); each wave copies the depthwise and pointwise weights of its own
// channels straight into a private LDS region, and the waves' partial
// pointwise sums are added in LDS.  Every input value of a batch of KB
// k-steps is loaded before any is used (one memory round trip per batch);
// with several inputs the next input's loads are in flight while the current
// one is added.
template <int K, bool SINGLE, bool COH>
__device__ __forceinline__ void sep_row_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  constexpr int KB = SINGLE ? (K == 3 ? 8 : 6) : (K == 3 ? 4 : 2);   // k-steps per batch
  constexpr int KKP = (K * K + 3) & ~3;               // floats per channel of depthwise weights
  constexpr int NBT = kSepRowMaxNB;
  constexpr int LDR = 16 + 1;                         // reduction buffer row pitch
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int j = lane & 15, g = lane >> 4;
  const int tm = fdiv(t, o.fd_tn), tn = t - tm * o.tiles_n;
  const int H = o.H, W = o.W, Ho = o.Ho, Wo = o.Wo, howo = Ho * Wo;
  const int bpr = o.row_bpr, per_img = Ho * bpr;
  const int img = fdiv(tm, o.fd_pimg), rr = tm - img * per_img;
  const int oh = fdiv(rr, o.fd_rbpr), ow0 = (rr - oh * bpr) * 16;
  const int NKS = o.CinP >> 2;
  const int ks0 = NKS * wave / kWaves, nks = NKS * (wave + 1) / kWaves - ks0;
  const int nb0 = tn * o.sep_nbt, nbc = min(o.sep_nbt, (o.Npad >> 4) - nb0);
  const int pitch = nbc * 16;                         // pointwise weights row in LDS
  const int Cin = o.Cin, kh = o.kh, ph = o.ph;
  const int NC = nbc * 16;

  // (0) the tile's biases -> LDS past the weights and partial sums, copied
  //     first so that their round trip overlaps the weights' and inputs'
  float *bl = lds + sep_row_bias_offset(o.CinP, K, o.sep_nbt);
  if (wave == 0 && lane < NC) lds_dma(rsrc(o.bias, o.Npad * 4), bl, (nb0 * 16 + lane) * 4);

  // (1) this wave's weights -> its LDS region: depthwise [4 nks][KKP], then
  //     pointwise rows 4 ks0 .. 4 (ks0 + nks) - 1, columns of this tile
  float *wl = lds + wave * sep_row_wave_floats(o.CinP, K, o.sep_nbt);
  float *pl = wl + nks * 4 * KKP;
  {
    const __amdgpu_buffer_rsrc_t dr = rsrc(o.dw, o.dw_bytes);
    const int nd = nks * 4 * KKP, src = ks0 * 4 * KKP;
    for (int e = 0; e < nd; e += 64)
      if (e + lane < nd) lds_dma(dr, wl + e, (src + e + lane) * 4);
    const __amdgpu_buffer_rsrc_t wr = rsrc(o.wpk, o.w_bytes);
    const int np = nks * 4 * pitch;
    for (int e = 0; e < np; e += 64) {
      const int i = e + lane, row = i / pitch, col = i - row * pitch;
      if (i < np) lds_dma(wr, pl + e, ((4 * ks0 + row) * o.Npad + nb0 * 16 + col) * 4);
    }
  }

  // (2) input loads.  Lane column colA = ow0 - pw + j (and colA + 16 for the
  //     K - 1 lanes whose second value is needed); out-of-image rows and
  //     columns and channels past Cin read 0 (zero padding).
  const int colA = ow0 - o.pw + j, colB = colA + 16;
  const bool okA = colA >= 0 && colA < W, okB = j < K - 1 && colB >= 0 && colB < W;
  auto issue = [&](int b, int k, float (&X)[KB][K][2]) {
    const __amdgpu_buffer_rsrc_t xr = rsrc(sl[U(op.in_slot[k])], U(op.in_bytes[k]));
    const int cb = img * U(op.in_ctot[k]) + U(op.in_coff[k]) + 4 * ks0 + g;
#pragma unroll
    for (int s = 0; s < KB; ++s) {
      const int kr = b * KB + s;                      // k-step relative to ks0
      const bool cok = 4 * (ks0 + kr) + g < Cin;
#pragma unroll
      for (int u = 0; u < K; ++u) {
        const int ih = oh + u - ph;
        if (kr < nks && u < kh && ih >= 0 && ih < H) {   // uniform
          const int row = ((cb + 4 * kr) * H + ih) * W;
          X[s][u][0] = bld(xr, cok && okA ? (row + colA) * 4 : kOOB, 0);
          X[s][u][1] = bld(xr, cok && okB ? (row + colB) * 4 : kOOB, 0);
        } else {
          X[s][u][0] = 0.f;
          X[s][u][1] = 0.f;
        }
      }
    }
  };

  floatx4 acc[NBT];
#pragma unroll
  for (int nb = 0; nb < NBT; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};

  const bool relu_in = o.pre_relu != 0;
  // depthwise filter of batch b from the summed inputs S, then its MFMAs
  // (weights from LDS: the caller has waited for the copies)
  auto finish = [&](int b, float (&S)[KB][K][2]) {
#pragma unroll
    for (int s = 0; s < KB; ++s) {
      const int kr = b * KB + s;
      if (kr >= nks) break;
      const float *wc = wl + (kr * 4 + g) * KKP;
      float d = 0.f;
#pragma unroll
      for (int u = 0; u < K; ++u) {
        float xa = S[s][u][0], xb = S[s][u][1];
        if (relu_in) { xa = fmaxf(xa, 0.f); xb = fmaxf(xb, 0.f); }
        d = fmaf(wc[u * K], xa, d);
        d = dw_taps(wc + u * K, xa, xb, d, std::make_integer_sequence<int, K - 1>{});
      }
      const float *bp = pl + (4 * kr + g) * pitch + j;
#pragma unroll
      for (int nb = 0; nb < NBT; ++nb)
        if (nb < nbc) acc[nb] = mfma16x16x4(d, bp[nb * 16], acc[nb]);
    }
  };

  if constexpr (SINGLE) {
    float X[KB][K][2];
    for (int b = 0; b * KB < nks; ++b) {
      issue(b, 0, X);
      lds_dma_wait();
      finish(b, X);
    }
  } else {
    float S[KB][K][2], X0[KB][K][2], X1[KB][K][2];
    const int n_in = o.n_in;
    for (int b = 0; b * KB < nks; ++b) {
      issue(b, 0, X0);
      for (int k = 0; k < n_in; k += 2) {
        if (k + 1 < n_in) issue(b, k + 1, X1);
#pragma unroll
        for (int s = 0; s < KB; ++s)
#pragma unroll
          for (int u = 0; u < K; ++u)
#pragma unroll
            for (int p = 0; p < 2; ++p) S[s][u][p] = k == 0 ? X0[s][u][p] : S[s][u][p] + X0[s][u][p];
        if (k + 1 >= n_in) break;
        if (k + 2 < n_in) issue(b, k + 2, X0);
#pragma unroll
        for (int s = 0; s < KB; ++s)
#pragma unroll
          for (int u = 0; u < K; ++u)
#pragma unroll
            for (int p = 0; p < 2; ++p) S[s][u][p] += X1[s][u][p];
      }
      lds_dma_wait();
      finish(b, S);
    }
  }
  // a wave with no k-steps still waits for nothing in flight
  lds_dma_wait();

  // (3) partial sums of the 8 waves -> LDS [wave][column][pixel] (the region
  //     held the weights: every wave must be done with them)
  __syncthreads();
#pragma unroll
  for (int nb = 0; nb < NBT; ++nb)
    if (nb < nbc) {
#pragma unroll
      for (int e = 0; e < 4; ++e) lds[(wave * NBT * 16 + nb * 16 + j) * LDR + 4 * g + e] = acc[nb][e];
    }
  __syncthreads();
  for (int idx = tid; idx < NC * 16; idx += kThreads) {
    const int col = idx >> 4, px = idx & 15;
    const int n = nb0 * 16 + col, ow = ow0 + px;
    if (ow >= Wo || n >= o.Cout) continue;
    float v = bl[col];
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v += lds[(w * NBT * 16 + col) * LDR + px];
    if (o.post_relu) v = fmaxf(v, 0.f);
    st<COH>(route_ptr(sl, op, o, n, img, oh * Wo + ow, howo), v);
  }
}

// "Relu-SepConv" unit, line tile: R = line_r whole output rows (R Wo <= 32
// pixels) x 32 NB output channels per workgroup (NB = 1 or 2), 3 x 3 windows, rows of a
// multiple of 4 floats.  Every global load is 16 bytes wide, so that a
// workgroup issues few vector memory instructions for what it reads (at batch
// 1 the stage is bound by that issue rate, not by bytes):
//  (1) the R + 2 input rows of every channel (contiguous in memory) are
//      loaded by thread (channel cp + chp j, 16-byte piece q), the loads of up
//      to kLineInFlight inputs in flight at once; their sum, rectified, goes
//      to LDS with four zero columns on each side.  The depthwise weights, the
//      tile's pointwise weights and biases are loaded before the inputs.
//  (2) the depthwise output of (channel c, pixel p) goes to LDS word
//      32 c + p: k-step ks of v_mfma_f32_32x32x2_f32 (channels 2 ks, 2 ks + 1)
//      then reads its B operand [k = lane / 32][pixel = lane % 32] as the 64
//      words from 64 ks, and the pointwise weights are packed the same way
//      ([block][ks][lane], lane = 32 k + output channel).
//  (3) wave w multiplies output block w % NB over k-steps [kw KSW, (kw + 1)
//      KSW), kw = w / NB, and the 8 / NB waves of a block add their partial
//      sums in LDS before the bias and the store.
template <int NB, bool COH>
__device__ __forceinline__ void sep_line_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  constexpr int KW = kWaves / NB, IF = kLineInFlight, NLD = kLineMaxLoads;
  constexpr int MAXKS = (kLineMaxCin + 1) / 2;
  constexpr int AJ = (NB * MAXKS * 16 + kThreads - 1) / kThreads;     // 16-byte pointwise loads per thread
  constexpr int DJ = (2 * MAXKS * 12 / 4 + kThreads - 1) / kThreads;  // 16-byte depthwise loads per thread
  static_assert(kWaves % NB == 0, "waves split evenly over the output blocks");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tm = fdiv(t, o.fd_tn), tn = t - tm * o.tiles_n;
  const int img = fdiv(tm, o.fd_pimg), rb = tm - img * o.tiles_per_plane;
  const int H = o.H, W = o.W, Wo = o.Wo, Ho = o.Ho, howo = Ho * Wo, HW = H * W;
  LineGeom g;
  g.r = o.line_r; g.rows = o.line_rows; g.q = o.line_q; g.chp = o.line_chp; g.nks = o.line_nks;
  g.pitch = o.line_pitch;
  line_offsets(g, NB);
  const int R = g.r, ROWS = g.rows, PITCH = g.pitch, NKS = g.nks, CE = 2 * NKS;
  const int oh0 = rb * R, ih0 = oh0 - o.ph, cb0 = tn * NB, Cin = o.Cin;
  float *slab = lds, *dwb = lds + g.dwb, *dww = lds + g.dww, *al = lds + g.al, *bl = lds + g.bl;

  // (0) weights and biases: issued first, stored to LDS once the first
  //     inputs' loads are in flight
  if (tid < 32 * NB) lds_dma(rsrc(o.bias, o.Cout * 4), bl + wave * 64, (cb0 * 32 + tid) * 4);
  floatx4 av[AJ], dv[DJ];
  {
    const __amdgpu_buffer_rsrc_t wr = rsrc(o.wpk, o.w_bytes), dr = rsrc(o.dw, o.dw_bytes);
    const int na = NB * NKS * 16, nd = CE * 3;        // 16-byte pieces
#pragma unroll
    for (int j = 0; j < AJ; ++j) {
      const int f = tid + j * kThreads;
      av[j] = bld4(wr, f < na ? (cb0 * NKS * 64 + 4 * f) * 4 : kOOB);
    }
#pragma unroll
    for (int j = 0; j < DJ; ++j) {
      const int f = tid + j * kThreads;
      dv[j] = bld4(dr, f < nd ? 16 * f : kOOB);
    }
  }
  // zero columns of the staged rows
  for (int i = tid; i < CE * ROWS; i += kThreads) {
    *(floatx4 *)(slab + i * PITCH) = floatx4{0.f, 0.f, 0.f, 0.f};
    *(floatx4 *)(slab + i * PITCH + 4 + W) = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  // (1) this thread's piece: channel cp + chp j, staged row r, columns 4 c4 ..
  const int cp = fdiv(tid, o.fd_lq), qq = tid - cp * g.q;
  const int r = fdiv(qq, o.fd_lw4), c4 = qq - r * (W >> 2), ih = ih0 + r;
  const bool act = cp < g.chp && ih >= 0 && ih < H;
  const int pix4 = (ih * W + 4 * c4) * 4;
  floatx4 S[NLD];
#pragma unroll
  for (int j = 0; j < NLD; ++j) S[j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int n_in = o.n_in;
  for (int k0 = 0; k0 < n_in; k0 += IF) {
    floatx4 X[IF][NLD];
#pragma unroll
    for (int i = 0; i < IF; ++i) {
      const int k = k0 + i;
      if (k < n_in) {                                 // uniform
        const __amdgpu_buffer_rsrc_t xr = rsrc(sl[U(op.in_slot[k])], U(op.in_bytes[k]));
        const int base = (img * U(op.in_ctot[k]) + U(op.in_coff[k]) + cp) * HW * 4 + pix4;
#pragma unroll
        for (int j = 0; j < NLD; ++j)
          X[i][j] = bld4(xr, act && cp + g.chp * j < Cin ? base + g.chp * j * HW * 4 : kOOB);
      } else {
#pragma unroll
        for (int j = 0; j < NLD; ++j) X[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if (k0 == 0) {
      const int na = NB * NKS * 16, nd = CE * 3;
#pragma unroll
      for (int j = 0; j < AJ; ++j)
        if (tid + j * kThreads < na) *(floatx4 *)(al + 4 * (tid + j * kThreads)) = av[j];
#pragma unroll
      for (int j = 0; j < DJ; ++j)
        if (tid + j * kThreads < nd) *(floatx4 *)(dww + 4 * (tid + j * kThreads)) = dv[j];
    }
#pragma unroll
    for (int i = 0; i < IF; ++i)
#pragma unroll
      for (int j = 0; j < NLD; ++j) S[j] += X[i][j];
  }
  const bool relu_in = o.pre_relu != 0;
  if (cp < g.chp) {
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const int ch = cp + g.chp * j;
      if (ch < CE) {
        floatx4 v = S[j];
        if (relu_in) {
          v.x = fmaxf(v.x, 0.f); v.y = fmaxf(v.y, 0.f); v.z = fmaxf(v.z, 0.f); v.w = fmaxf(v.w, 0.f);
        }
        *(floatx4 *)(slab + (ch * ROWS + r) * PITCH + 4 + 4 * c4) = v;
      }
    }
  }
  lds_dma_wait();                                     // the biases' copy (wave 0, 1)
  __syncthreads();

  // (2) depthwise.  One output row per tile: item e = (channel e / 4,
  //     pixels 8 (e % 4) .. + 7), reading columns x0 - 4 .. x0 + 11 of each
  //     staged row (the second four pixels only where they are in the row)
  if (R == 1) {
    for (int e = tid; e < CE * 4; e += kThreads) {
      const int ch = e >> 2, x0 = (e & 3) * 8;
      const bool two = x0 + 4 < Wo;
      floatx4 d0{0.f, 0.f, 0.f, 0.f}, d1{0.f, 0.f, 0.f, 0.f};
      if (x0 < Wo) {
        float w[12];
#pragma unroll
        for (int q4 = 0; q4 < 3; ++q4) {
          const floatx4 t4 = *(const floatx4 *)(dww + ch * 12 + 4 * q4);
          w[4 * q4] = t4.x; w[4 * q4 + 1] = t4.y; w[4 * q4 + 2] = t4.z; w[4 * q4 + 3] = t4.w;
        }
#pragma unroll
        for (int u = 0; u < 3; ++u) {
          const float *row = slab + (ch * ROWS + u) * PITCH + x0;
          const floatx4 a0 = *(const floatx4 *)row, a1 = *(const floatx4 *)(row + 4),
                        a2 = *(const floatx4 *)(row + 8);
          const floatx4 a3 = two ? *(const floatx4 *)(row + 12) : floatx4{0.f, 0.f, 0.f, 0.f};
          const float v[16] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w,
                               a2.x, a2.y, a2.z, a2.w, a3.x, a3.y, a3.z, a3.w};
#pragma unroll
          for (int c = 0; c < 3; ++c) {
            const float wt = w[u * 3 + c];
            d0.x = fmaf(wt, v[3 + c], d0.x);
            d0.y = fmaf(wt, v[4 + c], d0.y);
            d0.z = fmaf(wt, v[5 + c], d0.z);
            d0.w = fmaf(wt, v[6 + c], d0.w);
            d1.x = fmaf(wt, v[7 + c], d1.x);
            d1.y = fmaf(wt, v[8 + c], d1.y);
            d1.z = fmaf(wt, v[9 + c], d1.z);
            d1.w = fmaf(wt, v[10 + c], d1.w);
          }
        }
        if (!two) d1 = floatx4{0.f, 0.f, 0.f, 0.f};
      }
      *(floatx4 *)(dwb + ch * 32 + x0) = d0;
      *(floatx4 *)(dwb + ch * 32 + x0 + 4) = d1;
    }
  } else
  // several rows per tile: item e = (channel e / 8, pixels 4 (e % 8) .. + 3)
  for (int e = tid; e < CE * 8; e += kThreads) {
    const int ch = e >> 3, p0 = (e & 7) * 4;
    const int ro = fdiv(p0, o.fd_wo), x0 = p0 - ro * Wo;
    floatx4 d{0.f, 0.f, 0.f, 0.f};
    if (ro < R) {
      float w[12];
#pragma unroll
      for (int q4 = 0; q4 < 3; ++q4) {
        const floatx4 t4 = *(const floatx4 *)(dww + ch * 12 + 4 * q4);
        w[4 * q4] = t4.x; w[4 * q4 + 1] = t4.y; w[4 * q4 + 2] = t4.z; w[4 * q4 + 3] = t4.w;
      }
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const float *row = slab + (ch * ROWS + ro + u) * PITCH + x0;   // columns x0 - 4 .. x0 + 7
        const floatx4 a0 = *(const floatx4 *)row, a1 = *(const floatx4 *)(row + 4),
                      a2 = *(const floatx4 *)(row + 8);
        const float v[12] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w, a2.x, a2.y, a2.z, a2.w};
#pragma unroll
        for (int c = 0; c < 3; ++c) {
          const float wt = w[u * 3 + c];
          d.x = fmaf(wt, v[3 + c], d.x);
          d.y = fmaf(wt, v[4 + c], d.y);
          d.z = fmaf(wt, v[5 + c], d.z);
          d.w = fmaf(wt, v[6 + c], d.w);
        }
      }
    }
    *(floatx4 *)(dwb + ch * 32 + p0) = d;
  }
  __syncthreads();

  // (3) pointwise on the matrix cores: wave w multiplies block w % NB over
  //     k-steps [kw KSW, (kw + 1) KSW), kw = w / NB; then the partial sums of
  //     the KW waves of each block through LDS (over the staged rows, which
  //     are no longer read)
  const int cbl = wave % NB, kw = wave / NB;
  const int ksw = (NKS + KW - 1) / KW, ks0 = kw * ksw, ks1 = min(NKS, ks0 + ksw);
  floatx16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  {
    const float *ap = al + cbl * NKS * 64 + lane, *bp = dwb + lane;
    int ks = ks0;
    for (; ks + 2 <= ks1; ks += 2) {
      const float a0 = ap[ks * 64], b0 = bp[ks * 64], a1 = ap[ks * 64 + 64], b1 = bp[ks * 64 + 64];
      acc = mfma32x32x2(a0, b0, acc);
      acc = mfma32x32x2(a1, b1, acc);
    }
    if (ks < ks1) acc = mfma32x32x2(ap[ks * 64], bp[ks * 64], acc);
  }
  float *red = lds;                                   // [kw][block][16][64]
#pragma unroll
  for (int i = 0; i < 16; ++i) red[((kw * NB + cbl) * 16 + i) * 64 + lane] = acc[i];
  __syncthreads();
  for (int idx = tid; idx < NB * 1024; idx += kThreads) {
    const int b = idx >> 10, i = (idx >> 6) & 15, l = idx & 63;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < KW; ++w) v += red[((w * NB + b) * 16 + i) * 64 + l];
    const int cl = b * 32 + 8 * (i >> 2) + 4 * (l >> 5) + (i & 3), n = cb0 * 32 + cl, p = l & 31;
    const int ro = fdiv(p, o.fd_wo), x = p - ro * Wo, oh = oh0 + ro;
    if (n < o.Cout && ro < R && oh < Ho) {
      v += bl[cl];
      if (o.post_relu) v = fmaxf(v, 0.f);
      st<COH>(route_ptr(sl, op, o, n, img, oh * Wo + x, howo), v);
    }
  }
}

// The loads of SEPCONV GEMM-tile chunk c into ring slot s: this wave's
// 64-float pieces of the input planes (per-lane offsets xoff, the chunk's
// first channel added), of the pointwise weights [16 k][BN] and of the
// depthwise weights [16][KK].  Offsets that may pass the end of their
// buffer are per-lane (the range check covers them): the planes of the last
// chunk past Cin, the copy of the last chunk's depthwise weights rounded up
// to 64 floats.
template <int COPIES, int ACOPIES>
__device__ __forceinline__ void sepg_issue(float *s, const __amdgpu_buffer_rsrc_t &xr, const __amdgpu_buffer_rsrc_t &wr,
                                           const __amdgpu_buffer_rsrc_t &dr, const int *xoff, const int *aoff, int c,
                                           int nx, int nw, int XS, int AS, int hw4, int ldw, int KK, int wave,
                                           int lane) {
  wave = __builtin_amdgcn_readfirstlane(wave);       // uniform loop bounds around the LDS loads
#pragma unroll
  for (int i = 0; i < COPIES; ++i) {
    const int j = wave + i * kWaves;
    if (j < nx)                                       // uniform
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void *)(s + j * 64), 4,
                                               xoff[i] == kOOB ? kOOB : xoff[i] + c * 16 * hw4, 0, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < ACOPIES; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void *)(s + XS + (wave * ACOPIES + i) * 64), 4, aoff[i],
                                             c * 16 * ldw * 4, 0, 0);
#pragma unroll
  for (int i = 0; i < 2; ++i) {                       // nw <= 16 (windows up to 5 x 5)
    const int j = wave + i * kWaves;
    if (j < nw)                                       // uniform
      __builtin_amdgcn_raw_ptr_buffer_load_lds(dr, (lds_void *)(s + XS + AS + j * 64), 4,
                                               (c * 16 * KK + j * 64 + lane) * 4, 0, 0, 0);
  }
}

// s_waitcnt vmcnt(n) for a uniform run-time n <= MAX.
template <int MAX>
__device__ __forceinline__ void wait_vmcnt_upto(int n) {
  if constexpr (MAX > 0) {
    if (n >= MAX) { wait_vmcnt<MAX>(); return; }
    wait_vmcnt_upto<MAX - 1>(n);
  } else {
    wait_vmcnt<0>();
  }
}

// max(v, 0) in one instruction (median of v, 0 and +inf)
__device__ __forceinline__ float relu1(float v) { return __builtin_amdgcn_fmed3f(v, 0.f, __builtin_inff()); }

// Depthwise outputs of one (channel, strip of 2 output columns) for RG
// output rows, from its staged plane (rows with the window's halo, columns
// with a zero halo of pw on each side: no column test), the input ReLU
// applied as each value is read; written to the B operand (row ch, column
// r Wo + col), zeros for a channel past Cin.
template <int K, int RG>
__device__ __forceinline__ void sepg_dw(const float *xp, const float *w, float *brow, int W2, int Wo, int col0, int rt,
                                        bool relu_in, bool cv) {
  float d[RG][2];
#pragma unroll
  for (int o = 0; o < RG; ++o) d[o][0] = d[o][1] = 0.f;
#pragma unroll
  for (int i = 0; i < RG + K - 1; ++i) {             // staged input row i feeds output rows i - K + 1 .. i
    float x[K + 1];
#pragma unroll
    for (int j = 0; j <= K; ++j) {
      const float v = xp[i * W2 + j];
      x[j] = relu_in ? relu1(v) : v;
    }
#pragma unroll
    for (int o = 0; o < RG; ++o) {
      const int u = i - o;
      if (u < 0 || u >= K) continue;                  // compile time
#pragma unroll
      for (int v = 0; v < K; ++v) {
        d[o][0] = fmaf(w[u * K + v], x[v], d[o][0]);
        d[o][1] = fmaf(w[u * K + v], x[v + 1], d[o][1]);
      }
    }
  }
#pragma unroll
  for (int o = 0; o < RG; ++o)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      if (o < rt && col0 + j < Wo) brow[o * Wo + col0 + j] = cv ? d[o][j] : 0.f;
}

// "Relu-SepConv" unit, GEMM tile: RG whole output rows of one image
// (BM = 32 WMW MFMA columns, RG Wo <= BM) x BN = 32 WNW output channels, 8
// waves of one 32x32 block each on v_mfma_f32_32x32x2_f32 (output channels
// as rows, pixels as columns).  The pointwise reduction runs over chunks of
// 16 input channels; per chunk
//   stage  direct global -> LDS loads, kSepgStages - 1 chunks in flight, of
//          the chunk's input planes (the tile's rows with the window's halo,
//          rows and columns outside the image as 0: one plane of
//          sepg_w2 = W + 2 pw columns per channel, pitch sepg_ps), its
//          depthwise weights and its pointwise weights [16 k][BN];
//   dw     every (channel, strip of 2 output columns) of the chunk over the
//          tile's rows -> the B operand [16 k][BM] in LDS (two buffers);
//   mfma   D[32 ch][32 px] += A[32 ch][2 k] B[2 k][32 px], 8 k-pairs, A
//          from the slot (read into registers a round early), B from the
//          depthwise results of the round before.
// One barrier per round: round c runs the depthwise of chunk c and the
// MFMAs of chunk c - 1; half the waves of each SIMD take the MFMAs first,
// the other half the depthwise, so that the SIMD's vector ALU works while
// the matrix core does.  B columns past RG Wo are never stored.
template <int WMW, int K, int RG, bool COH>
__device__ __forceinline__ void sep_gemm_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  constexpr int WNW = kWaves / WMW, BM = 32 * WMW, BN = 32 * WNW, D = kSepgStages, KK = K * K;
  constexpr int BMP = BM + 1;                        // B row pitch: the 16 channel rows on distinct banks
  constexpr int AC = 16 * BN / 64 / kWaves;          // 64-float pointwise-weight copies per wave
  static_assert(D == 3, "slot of chunk c + 2 = slot of chunk c - 1");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WMW, wn = wave / WMW;
  const int tm = fdiv(t, o.fd_tn), tn = t - tm * o.tiles_n;
  const int img = fdiv(tm, o.fd_pimg), rb = tm - img * o.tiles_per_plane;
  const int Wo = o.Wo, W = o.W, H = o.H, howo = o.Ho * Wo, W2 = o.sepg_w2;
  const int oh0 = rb * RG, rt = min(RG, o.Ho - oh0);                // rows of this tile
  const int R = o.sep_rows, PS = o.sepg_ps, ih0 = oh0 - o.ph;       // staged rows, plane pitch
  const int n0 = tn * BN, nck = o.sep_nck, ldw = o.pipe_ldw;
  const int XS = o.sepg_xs, AS = 16 * BN, WS = o.sepg_ws;            // floats per slot part
  const int SLOT = XS + AS + WS;
  float *ring = lds, *bsm = lds + D * SLOT;
  const int nx = XS >> 6, nw = WS >> 6;              // 64-float copies per slot part

  // per-lane offsets of this wave's copies of the input planes: element
  // e = 64 j + lane of the slot is channel e / PS, staged row (e % PS) / W2,
  // plane column (e % PS) % W2 = image column + pw; elements past a plane's
  // R W2 floats, rows and columns outside the image read 0; the chunk's
  // first channel is added per chunk
  const int cbase = img * o.in_ctot[0] + o.in_coff[0];
  int xoff[kSepgMaxCopies];
#pragma unroll
  for (int i = 0; i < kSepgMaxCopies; ++i) {
    const int e = (wave + i * kWaves) * 64 + lane;
    const int ch = fdiv(e, o.fd_ps), rem = e - ch * PS, r = fdiv(rem, o.fd_w2), col = rem - r * W2 - o.pw;
    const int ih = ih0 + r;
    xoff[i] = rem < R * W2 && ih >= 0 && ih < H && col >= 0 && col < W ? (((cbase + ch) * H + ih) * W + col) * 4
                                                                        : kOOB;
  }
  // pointwise weights of the slot: element f = k BN + col of [16 k][BN]
  int aoff[AC];
#pragma unroll
  for (int i = 0; i < AC; ++i) {
    const int f = (wave * AC + i) * 64 + lane;
    aoff[i] = ((f / BN) * ldw + n0 + f % BN) * 4;
  }
  const __amdgpu_buffer_rsrc_t xr = rsrc(sl[o.in_slot[0]], o.in_bytes[0]);
  const __amdgpu_buffer_rsrc_t wr = rsrc(o.wpk, o.w_bytes);
  const __amdgpu_buffer_rsrc_t dr = rsrc(o.dw, o.dw_bytes);
  const int hw4 = H * W * 4;
  const float bl = bias32_load(o.bias, n0 + wn * 32, o.Cout, lane);
  // loads per wave and chunk (the same for every chunk)
  int per = AC;
#pragma unroll
  for (int i = 0; i < kSepgMaxCopies; ++i) per += wave + i * kWaves < nx;
  per += (wave < nw) + (wave + kWaves < nw);
  per = __builtin_amdgcn_readfirstlane(per);

  // depthwise items: (channel ch, strip of columns 2 st, 2 st + 1)
  const int ch = tid & 15, strips = o.sepg_strips;
  const bool relu_in = o.pre_relu != 0;
  const bool mfma_first = (wave >> 2) & 1;           // waves w and w + 4 share a SIMD

  floatx16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  float avc[8];                                      // A of the chunk whose MFMAs run next
#pragma unroll
  for (int p = 0; p < 8; ++p) avc[p] = 0.f;
  sepg_issue<kSepgMaxCopies, AC>(ring, xr, wr, dr, xoff, aoff, 0, nx, nw, XS, AS, hw4, ldw, KK, wave, lane);
  if (nck > 1)
    sepg_issue<kSepgMaxCopies, AC>(ring + SLOT, xr, wr, dr, xoff, aoff, 1, nx, nw, XS, AS, hw4, ldw, KK, wave, lane);
  for (int c = 0; c <= nck; ++c) {
    // chunk c has landed once only chunk c + 1's loads (if any) are in
    // flight; the barrier publishes every wave's loads and the depthwise
    // results of round c - 1, and guarantees that round c - 1 no longer
    // reads chunk c - 1's slot (its A is in registers) or the B buffer that
    // round c writes
    if (c + 1 < nck) wait_vmcnt_upto<kSepgMaxCopies + 4 + 2>(per);
    else wait_vmcnt<0>();
    ring_barrier();
    if (c + 2 < nck)
      sepg_issue<kSepgMaxCopies, AC>(ring + ((c + 2) % D) * SLOT, xr, wr, dr, xoff, aoff, c + 2, nx, nw, XS, AS, hw4,
                                     ldw, KK, wave, lane);
    const float *s = ring + (c % D) * SLOT;
    float avn[8];
    if (c < nck) {
      const float *a = s + XS + (lane >> 5) * BN + wn * 32 + (lane & 31);
#pragma unroll
      for (int p = 0; p < 8; ++p) avn[p] = a[2 * p * BN];
    }
#pragma unroll
    for (int ph = 0; ph < 2; ++ph) {
      if ((ph == 0) == mfma_first) {
        if (c >= 1) {                                 // MFMAs of chunk c - 1
          const float *b = bsm + ((c - 1) & 1) * 16 * BMP + (lane >> 5) * BMP + wm * 32 + (lane & 31);
          float bv[8];
#pragma unroll
          for (int p = 0; p < 8; ++p) bv[p] = b[2 * p * BMP];
#pragma unroll
          for (int p = 0; p < 8; ++p) acc = mfma32x32x2(avc[p], bv[p], acc);
        }
      } else if (c < nck) {                           // depthwise of chunk c
        const bool cv = c * 16 + ch < o.Cin;          // channels past Cin (last chunk): zeros
        float *brow = bsm + (c & 1) * 16 * BMP + ch * BMP;
        float w[KK];
        const float *wp = s + XS + AS + ch * KK;
#pragma unroll
        for (int i = 0; i < KK; ++i) w[i] = wp[i];
        for (int st = tid >> 4; st < strips; st += kThreads / 16)
          sepg_dw<K, RG>(s + ch * PS + 2 * st, w, brow, W2, Wo, 2 * st, rt, relu_in, cv);
      }
    }
#pragma unroll
    for (int p = 0; p < 8; ++p) avc[p] = c < nck ? avn[p] : 0.f;
  }
  // epilogue: element i of lane l is channel n0 + 32 wn + 8 (i/4) + 4 (l/32) + i%4 of tile column 32 wm + l%32
  const int px = wm * 32 + (lane & 31);
  float bv16[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) bv16[i] = bias32_of(bl, i, lane);
  if (px < rt * Wo) {
    const int q = oh0 * Wo + px;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int n = n0 + wn * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
      if (n < o.Cout) {
        float v = acc[i] + bv16[i];
        if (o.post_relu) v = fmaxf(v, 0.f);
        st<COH>(route_ptr(sl, op, o, n, img, q, howo), v);
      }
    }
  }
}

// GEMM SEPCONV tile variants: waves along pixels (sep_nbt), window, rows per tile.
template <int WMW, int K, bool COH>
__device__ __forceinline__ void sep_gemm_rows(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  switch (o.sepg_rout) {
    case 2: sep_gemm_tile<WMW, K, 2, COH>(sl, op, o, t, lds); break;
    case 3: sep_gemm_tile<WMW, K, 3, COH>(sl, op, o, t, lds); break;
    default: sep_gemm_tile<WMW, K, 4, COH>(sl, op, o, t, lds); break;
  }
}
template <bool COH>
__device__ __forceinline__ void sep_gemm_dispatch(const Slots &sl, const DevOp &op, const DevOp &o, int t, float *lds) {
  if (o.sep_nbt == 4) {
    if (o.kh == 3) sep_gemm_rows<4, 3, COH>(sl, op, o, t, lds); else sep_gemm_rows<4, 5, COH>(sl, op, o, t, lds);
  } else {
    if (o.kh == 3) sep_gemm_rows<2, 3, COH>(sl, op, o, t, lds); else sep_gemm_rows<2, 5, COH>(sl, op, o, t, lds);
  }
}

// ------------------------------------------------------------------ elementwise

constexpr int kPoolBatch = 8;   // staging loads per thread in flight

// planes_per_tile whole (image, channel) planes of a pool whose planes are
// small: the planes' input rows are staged in LDS one plane after another
// (coalesced, each input value read once), then every output of the tile is
// reduced from LDS.  Planes run over images: plane = image * C + channel.
template <bool COH>
__device__ __forceinline__ void pool_planes_tile(const Slots &sl, const DevOp &o, int t, bool is_max,
                                                 float *lds) {
  const int tid = threadIdx.x;
  const int C = o.Cout, H = o.H, W = o.W, Wo = o.Wo, howo = o.Ho * Wo;
  const int p0 = t * o.planes_per_tile, np = min(o.planes_per_tile, o.N * C - p0);
  const int rows = o.pool_in_rows, n_pl = rows * W, n_in = np * n_pl;
  const __amdgpu_buffer_rsrc_t xr = rsrc(sl[o.in_slot[0]], o.in_bytes[0]);
  for (int base = 0; base < n_in; base += kPoolBatch * kThreads) {
    float v[kPoolBatch];
#pragma unroll
    for (int k = 0; k < kPoolBatch; ++k) {
      const int i = base + k * kThreads + tid;
      const int p = fdiv(i, o.fd_pin), j = i - p * n_pl;
      const int img = fdiv(p0 + p, o.fd_c), c = p0 + p - img * C;
      v[k] = bld(xr, i < n_in ? ((img * o.in_ctot[0] + o.in_coff[0] + c) * H * W + j) * 4 : kOOB, 0);
    }
#pragma unroll
    for (int k = 0; k < kPoolBatch; ++k) {
      const int i = base + k * kThreads + tid;
      if (i < n_in) lds[i] = v[k];
    }
  }
  __syncthreads();
  const float inv = 1.0f / (float)(o.kh * o.kw);
  for (int i = tid; i < np * howo; i += kThreads) {
    const int p = fdiv(i, o.fd_howo), r = i - p * howo;
    const int oh = fdiv(r, o.fd_wo), ow = r - oh * Wo;
    const float *pl = lds + p * n_pl;
    float acc = is_max ? -INFINITY : 0.f;
    for (int u = 0; u < o.kh; ++u) {
      const int ih = oh * o.sh + u - o.ph;
      if (ih < 0 || ih >= rows) continue;          // outside the image
      for (int q = 0; q < o.kw; ++q) {
        const int iw = ow * o.sw + q - o.pw;
        if (iw < 0 || iw >= W) continue;
        const float v = pl[ih * W + iw];
        acc = is_max ? fmaxf(acc, v) : acc + v;
      }
    }
    if (!is_max) acc *= inv;
    const int img = fdiv(p0 + p, o.fd_c), c = p0 + p - img * C;
    st<COH>(sl[o.route_slot[0]] + (size_t)(img * o.route_ctot[0] + o.route_coff[0] + c) * howo + r, acc);
  }
}

// One band of output rows of one (image, channel) plane: the input rows it
// needs are staged in LDS with coalesced loads (each input value is read from
// memory once), then every output is reduced from LDS.
template <bool COH>
__device__ __forceinline__ void pool_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, bool is_max,
                                          float *lds) {
  if (o.planes_per_tile > 1) {
    pool_planes_tile<COH>(sl, o, t, is_max, lds);
    return;
  }
  const int tid = threadIdx.x;
  const int C = o.Cout, H = o.H, W = o.W, Ho = o.Ho, Wo = o.Wo;
  const int plane = fdiv(t, o.fd_tpp), band = t - plane * o.tiles_per_plane;
  const int img = fdiv(plane, o.fd_c), c = plane - img * C;
  const int oh0 = band * o.rows_per_tile, oh1 = min(Ho, oh0 + o.rows_per_tile);
  const int ih_lo = max(0, oh0 * o.sh - o.ph);
  const int ih_hi = min(H, (oh1 - 1) * o.sh - o.ph + o.kh);
  const __amdgpu_buffer_rsrc_t xr = rsrc(sl[o.in_slot[0]], o.in_bytes[0]);
  const int src = ((img * o.in_ctot[0] + o.in_coff[0] + c) * H + ih_lo) * W;
  const int n_in = (ih_hi - ih_lo) * W;
  // batches of kPoolBatch loads per thread, all issued before any is
  // written to LDS: one memory round trip per batch
  for (int base = 0; base < n_in; base += kPoolBatch * kThreads) {
    float v[kPoolBatch];
#pragma unroll
    for (int k = 0; k < kPoolBatch; ++k) {
      const int i = base + k * kThreads + tid;
      v[k] = bld(xr, i < n_in ? (src + i) * 4 : kOOB, 0);
    }
#pragma unroll
    for (int k = 0; k < kPoolBatch; ++k) {
      const int i = base + k * kThreads + tid;
      if (i < n_in) lds[i] = v[k];
    }
  }
  __syncthreads();
  float *__restrict__ out = sl[o.route_slot[0]] +
                            (size_t)(img * o.route_ctot[0] + o.route_coff[0] + c) * Ho * Wo;
  const float inv = 1.0f / (float)(o.kh * o.kw);
  const int n_out = (oh1 - oh0) * Wo;
  for (int i = tid; i < n_out; i += kThreads) {
    const int q = fdiv(i, o.fd_wo), oh = oh0 + q, ow = i - q * Wo;
    float acc = is_max ? -INFINITY : 0.f;
    for (int u = 0; u < o.kh; ++u) {
      const int ih = oh * o.sh + u - o.ph;
      if (ih < ih_lo || ih >= ih_hi) continue;     // outside the image
      for (int q = 0; q < o.kw; ++q) {
        const int iw = ow * o.sw + q - o.pw;
        if (iw < 0 || iw >= W) continue;
        const float v = lds[(ih - ih_lo) * W + iw];
        acc = is_max ? fmaxf(acc, v) : acc + v;
      }
    }
    if (!is_max) acc *= inv;
    st<COH>(out + oh * Wo + ow, acc);
  }
}

// Up to kEltPerTile contiguous outputs of one (image, channel) plane.
template <bool COH>
__device__ __forceinline__ void sum_tile(const Slots &sl, const DevOp &op, const DevOp &o, int t, bool mean) {
  const int hw = o.Ho * o.Wo, C = o.Cout;
  const int plane = fdiv(t, o.fd_tpp), chunk = t - plane * o.tiles_per_plane;
  const int img = fdiv(plane, o.fd_c), c = plane - img * C;
  const int p0 = chunk * kEltPerTile;
  float *__restrict__ out = sl[o.route_slot[0]] +
                            (size_t)(img * o.route_ctot[0] + o.route_coff[0] + c) * hw;
  float s[kEltPerTile / kThreads];
#pragma unroll
  for (int e = 0; e < kEltPerTile / kThreads; ++e) s[e] = 0.f;
  // inputs two at a time: both inputs' loads are issued before either is added
  for (int i = 0; i < o.n_in; i += 2) {
    const int j = min(i + 1, o.n_in - 1);
    const __amdgpu_buffer_rsrc_t r0 = rsrc(sl[U(op.in_slot[i])], U(op.in_bytes[i]));
    const __amdgpu_buffer_rsrc_t r1 = rsrc(sl[U(op.in_slot[j])], U(op.in_bytes[j]));
    const int base0 = (img * U(op.in_ctot[i]) + U(op.in_coff[i]) + c) * hw;
    const int base1 = (img * U(op.in_ctot[j]) + U(op.in_coff[j]) + c) * hw;
    const bool two = j != i;                       // uniform
    float a[kEltPerTile / kThreads], b[kEltPerTile / kThreads];
#pragma unroll
    for (int e = 0; e < kEltPerTile / kThreads; ++e) {
      const int pix = p0 + e * kThreads + threadIdx.x;
      a[e] = bld(r0, pix < hw ? (base0 + pix) * 4 : kOOB, 0);
      b[e] = bld(r1, two && pix < hw ? (base1 + pix) * 4 : kOOB, 0);
    }
#pragma unroll
    for (int e = 0; e < kEltPerTile / kThreads; ++e) s[e] += a[e] + b[e];
  }
#pragma unroll
  for (int e = 0; e < kEltPerTile / kThreads; ++e) {
    const int pix = p0 + e * kThreads + threadIdx.x;
    if (pix < hw) st<COH>(out + pix, mean ? s[e] * o.inv_n : s[e]);
  }
}

// ------------------------------------------------------------------ kernel

// Kernel variants, chosen per stage by the host so that a stage only pays
// the registers of the tile kinds it contains:
//   KV_LIGHT   16x16 and 16x32 conv tiles, pooling, add / mean
//   KV_SEP     KV_LIGHT + staged SEPCONV tiles
//   KV_SEPROW  KV_LIGHT + row SEPCONV tiles
//   KV_PIPE    KV_LIGHT + pipelined conv tiles
//   KV_FULL    every tile kind and conv tile shape
// A conv tile with the input ReLU and the channel check resolved at compile
// time (no branch between its loads and MFMAs).
template <int FM, int FN, int WM, int WN, int WK, bool COH>
__device__ __forceinline__ void conv_any(const Slots &sl, const DevOp &op, const DevOp &o, int ti, float *lds) {
  const bool full = o.Cin == o.CinP;
  if (o.pre_relu) {
    if (full) conv_tile<FM, FN, WM, WN, WK, COH, true, true>(sl, op, o, ti, lds);
    else conv_tile<FM, FN, WM, WN, WK, COH, true, false>(sl, op, o, ti, lds);
  } else {
    if (full) conv_tile<FM, FN, WM, WN, WK, COH, false, true>(sl, op, o, ti, lds);
    else conv_tile<FM, FN, WM, WN, WK, COH, false, false>(sl, op, o, ti, lds);
  }
}

template <bool COH, int KV>
__device__ __forceinline__ void run_tile(const Slots &sl, const DevOp &op, const DevOp &o, int ti, float *lds) {
  switch (o.kind) {
    case DK_CONV:
      if constexpr (KV == KV_PIPE || KV == KV_FULL) {
        if (o.tcfg >= TC_P128x64) {
          switch (o.tcfg) {
            case TC_P128x64: conv_pipe_tile<4, COH>(sl, op, o, ti, lds); break;
            case TC_P256x32: conv_pipe_tile<8, COH>(sl, op, o, ti, lds); break;
            case TC_P64x128: conv_pipe_tile<2, COH>(sl, op, o, ti, lds); break;
            case TC_W128x64: conv_wave_tile<4, COH>(sl, op, o, ti, lds); break;
            case TC_W256x32: conv_wave_tile<8, COH>(sl, op, o, ti, lds); break;
            default: conv_wave_tile<2, COH>(sl, op, o, ti, lds); break;
          }
          break;
        }
      }
      if constexpr (KV != KV_FULL) {
        if (o.tcfg == TC_16x16_K8) conv_any<1, 1, 1, 1, 8, COH>(sl, op, o, ti, lds);
        else conv_any<1, 2, 1, 1, 8, COH>(sl, op, o, ti, lds);
        break;
      } else {
        switch (o.tcfg) {
          case TC_16x16_K8: conv_any<1, 1, 1, 1, 8, COH>(sl, op, o, ti, lds); break;
          case TC_16x32_K8: conv_any<1, 2, 1, 1, 8, COH>(sl, op, o, ti, lds); break;
          case TC_32x32_K8: conv_any<2, 2, 1, 1, 8, COH>(sl, op, o, ti, lds); break;
          case TC_32x64_K4: conv_any<2, 2, 1, 2, 4, COH>(sl, op, o, ti, lds); break;
          case TC_64x64_K2: conv_any<2, 2, 2, 2, 2, COH>(sl, op, o, ti, lds); break;
          default: conv_any<2, 2, 4, 2, 1, COH>(sl, op, o, ti, lds); break;
        }
        break;
      }
    case DK_SEP:
      if constexpr (KV == KV_SEP || KV == KV_SEPROW || KV == KV_FULL) {
        if (o.sep_row == 2) {
          if constexpr (KV != KV_SEPROW) sep_gemm_dispatch<COH>(sl, op, o, ti, lds);
        } else if (!o.sep_row) {
          if constexpr (KV != KV_SEPROW) sep_tile<COH>(sl, op, o, ti, lds);
        } else if constexpr (KV != KV_SEP) {
          if (o.sep_row == 3) {
            if (o.sep_nbt == 1) sep_line_tile<1, COH>(sl, op, o, ti, lds);
            else sep_line_tile<2, COH>(sl, op, o, ti, lds);
            break;
          }
          const bool one = o.n_in == 1;
          if (o.row_k == 3) {
            if (one) sep_row_tile<3, true, COH>(sl, op, o, ti, lds); else sep_row_tile<3, false, COH>(sl, op, o, ti, lds);
          } else {
            if (one) sep_row_tile<5, true, COH>(sl, op, o, ti, lds); else sep_row_tile<5, false, COH>(sl, op, o, ti, lds);
          }
        }
      }
      break;
    case DK_POOL_MAX: pool_tile<COH>(sl, op, o, ti, true, lds); break;
    case DK_POOL_AVG: pool_tile<COH>(sl, op, o, ti, false, lds); break;
    case DK_ADD: sum_tile<COH>(sl, op, o, ti, false); break;
    default: sum_tile<COH>(sl, op, o, ti, true); break;
  }
}

// Wait for in-stage producers, compute, signal (one tile of op `opi`, whose
// descriptor is `op` in LDS and `o` for uniform use).
template <int KV>
__device__ __forceinline__ void tile_body(const StageArgs &a, const Slots &sl, const DevOp *ops, const DevOp &op,
                                          const DevOp &o, int opi, int ti, float *lds) {
  const int tid = threadIdx.x;
  const int n_deps = o.n_deps, signal = o.signal;
  if (n_deps) {
    // one thread polls the producers' counters with coherent loads (its own
    // copy of each, so the pollers of a stage spread over kCtrCopies memory
    // channels), then invalidates stale cache lines once; the workgroup
    // reads the producers' outputs only after that (barrier)
    if (tid == 0) {
      int32_t *mine = a.ctr + 2 + kCtrStride * (blockIdx.x % kCtrCopies);
      for (int k = 0; k < n_deps; ++k) {
        const int d = op.dep[k];
        const int need = ops[d].n_tiles;
        int spins = 0;
        while (__hip_atomic_load(&mine[d], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < need) {
          __builtin_amdgcn_s_sleep(4);
          if (++spins > a.spin_limit) {
            __hip_atomic_fetch_or(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
        }
      }
      // drop lines of this CU / XCD that may predate the producers' stores
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
  }

  if (n_deps || signal) run_tile<true, KV>(sl, op, o, ti, lds);
  else run_tile<false, KV>(sl, op, o, ti, lds);

  if (signal) {
    // The tile's outputs were written with agent-coherent stores.  Every wave
    // waits until its stores have been performed, then one wave moves every
    // copy of the op's counter; a consumer reads the outputs only after
    // seeing the final count and invalidating its stale lines, so it sees
    // every value.  This orders like a release/acquire pair without a
    // per-tile L2 writeback.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
    if (tid < kCtrCopies)
      __hip_atomic_fetch_add(&a.ctr[2 + opi + kCtrStride * tid], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}


// One tile: find its op, then tile_body.
// `tab` is the stage table in LDS, `gtab` the same table in global memory.
template <int KV>
__device__ __forceinline__ void process_tile(const StageArgs &a, const Slots &sl, const int32_t *tab,
                                             const int4 *__restrict__ gtab, int t, float *lds) {
  const int tid = threadIdx.x, lane = tid & 63;
  // op_start is non-decreasing with op_start[0] = 0: the tile's op is the
  // last one starting at or before t.  Lane i holds op_start[i] and word
  // i % 4 of the header; the values are taken out with v_readlane.
  const int hv = tab[lane & 3], ov = tab[4 + lane];
  const int n_ops = __builtin_amdgcn_readlane(hv, 0);
  const int opi = __popcll(__ballot(lane < n_ops && t >= ov)) - 1;
  const int s0 = __builtin_amdgcn_readlane(ov, opi);
  int ti = t - s0;
  const int devop_off = __builtin_amdgcn_readlane(hv, 2);
  const DevOp *ops = (const DevOp *)(tab + devop_off);
  const DevOp &op = ops[opi];
  if (ti >= U(op.n_tiles)) return;                   // padding between ops' ranges (see the stage table)

  // The descriptor's fields for uniform use.  The light and pipelined
  // variants, which read few of them, move the LDS copy into scalar
  // registers at once (op_scalars); the SEPCONV and full variants, which
  // read many (a v_readlane per word and hundreds of spilled scalars), load
  // each field where it is used with scalar loads from the table in global
  // memory (read-only while the kernel runs, a uniform address).
  if constexpr (KV == KV_LIGHT || KV == KV_PIPE) {
    const DevOp o = op_scalars(op);
    tile_body<KV>(a, sl, ops, op, o, opi, ti, lds);
  } else {
    const DevOp &o = ((const DevOp *)((const int32_t *)gtab + devop_off))[opi];
    tile_body<KV>(a, sl, ops, op, o, opi, ti, lds);
  }
}

// Dynamic LDS of a launch: the buffer pointers (kSlotWords words), the stage
// table, then the tile's own scratch.  A workgroup fills the first two with
// one round of loads before its first tile: the table pointer and size are
// preloaded into scalar registers at dispatch, and every load (table words,
// pointer words from the kernel arguments) is issued before the first wait.
__device__ __forceinline__ float *stage_prologue(const int4 *__restrict__ table, int table_words,
                                                 const StageArgs &a, int32_t *meta) {
  const int tid = threadIdx.x, nv = table_words >> 2;
  const bool ht = tid < nv, hs = tid < kSlotWords;
  int4 tv{};
  int sv = 0;
  if (ht) tv = table[tid];
  if (hs) sv = ((const int32_t *)a.slot)[tid];
  int4 *dst = (int4 *)(meta + kSlotWords);
  if (ht) dst[tid] = tv;
  if (hs) meta[tid] = sv;
  for (int i = tid + kThreads; i < nv; i += kThreads) dst[i] = table[i];   // tables over 8 KB
  __syncthreads();
  return (float *)(meta + kSlotWords + table_words);
}

// A stage without in-stage dependencies runs one workgroup per tile.  A stage
// with dependencies runs G workgroups, G no more than fit on the GPU at once
// (occupancy of this kernel), so that all of them become resident even if
// other kernels hold CUs for a while.  Workgroup w takes tiles w, w + G,
// w + 2G, ... in tile order, which is topological: the smallest unfinished
// tile has finished producers and an owner that has reached it, so every wait
// ends, without a work queue or ticket atomics.  (A cooperative launch would
// guarantee the residency too, but costs about 20 us per launch here.)
// The table pointer and size come first so that they can be preloaded into
// scalar registers at dispatch.
// Workgroups are handed to the 8 XCDs in turn (workgroup b to XCD b % 8),
// and each XCD has its own L2.  Workgroup b of a launch of n tiles runs tile
// xcd_tile(b, n, lg) (a persistent launch does so per round of gridDim.x
// tiles): runs of 2^lg consecutive tiles land on one XCD, while the runs
// still start in tile order.  The host picks lg per stage (word 3 of the
// table header).  A permutation of [0, n); the last n % (8 2^lg) tiles keep
// their index, and lg = 0 is the plain order.
static_assert(kXcds == 8, "xcd_tile divides by the XCD count with shifts by 3");
__device__ __forceinline__ int xcd_tile(int b, int n, int lg) {
  const int full = (n >> (3 + lg)) << (3 + lg);
  if (b >= full) return b;
  const int xcd = b & 7, local = b >> 3;
  return ((((local >> lg) << 3) + xcd) << lg) + (local & ((1 << lg) - 1));
}

// The one-tile-per-workgroup kernels of the light, pipelined and row-SEPCONV
// variants keep two workgroups per CU (at most 128 VGPRs).
template <int KV, bool PERSIST>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(
    (!PERSIST && (KV == KV_LIGHT || KV == KV_PIPE || KV == KV_SEPROW)) ? 4 : 1))) void ios_stage_kernel(const int4 *__restrict__ table, int table_words,
                                                             StageArgs a) {
  extern __shared__ int4 lds_base[];
  int32_t *meta = (int32_t *)lds_base;
  float *lds = stage_prologue(table, table_words, a, meta);
  const Slots sl{(float *const *)meta};
  const int32_t *tab = meta + kSlotWords;
  if constexpr (!PERSIST) {
    process_tile<KV>(a, sl, tab, table, xcd_tile(blockIdx.x, gridDim.x, U(tab[3])), lds);
    return;
  }
  // round r takes tiles [r G, r G + G), permuted inside the round as above:
  // a workgroup still meets its tiles in increasing order, so the lowest
  // unfinished tile always has its producers done and its workgroup free
  const int n_tiles = U(tab[1]), n_ops = U(tab[0]), lg = U(tab[3]), G = gridDim.x, b = blockIdx.x;
  for (int base = 0; base + b < n_tiles; base += G) {
    process_tile<KV>(a, sl, tab, table, base + xcd_tile(b, min(G, n_tiles - base), lg), lds);
    __syncthreads();   // the next tile reuses LDS
  }
  if (threadIdx.x == 0) {
    // Thread 0 belongs to the wave that issued this workgroup's counter
    // increments (process_tile).  vmcnt(0) makes the wave wait until every
    // one of them (and every poll) has been performed before the increment
    // below is issued, so when the last workgroup sees gridDim.x - 1 every
    // increment of the launch has landed; the resets depend on the value it
    // returned, so they are issued after it was performed.  No increment of
    // this launch can therefore land after a reset and leave a counter
    // non-zero for the next launch.  (An agent-scope release would do the
    // same plus an L2 writeback, which the counters do not need: they are
    // only touched by agent-scope atomics.)
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    int f = __hip_atomic_fetch_add(&a.ctr[1], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (f == (int)gridDim.x - 1) {
      // last workgroup of the launch: leave the counters at zero for the
      // next launch on the stream
      for (int r = 0; r < kCtrCopies; ++r)
        for (int i = 0; i < n_ops; ++i)
          __hip_atomic_store(&a.ctr[2 + i + kCtrStride * r], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ctr[1], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

}  // namespace ios
