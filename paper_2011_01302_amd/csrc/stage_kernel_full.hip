// Stage kernel variant KV_FULL, one workgroup per tile: every tile kind and conv tile shape.  One translation unit per
// (variant, launch kind) so that the kernels build in parallel (see
// stage_kernel.h and stage_launch.cpp).
#include "stage_kernel.h"

namespace ios {

void *stage_kernel_fn_full() { return (void *)ios_stage_kernel<KV_FULL, false>; }

hipError_t stage_launch_full(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s) {
  hipLaunchKernelGGL((ios_stage_kernel<KV_FULL, false>), dim3(grid), dim3(kThreads), lds, s, t, words, a);
  return hipGetLastError();
}

}  // namespace ios
