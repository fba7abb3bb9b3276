// Stage kernel variant KV_LIGHT, persistent launch: 16x16 and 16x32 conv tiles, pooling, add / mean.  One translation unit per
// (variant, launch kind) so that the kernels build in parallel (see
// stage_kernel.h and stage_launch.cpp).
#include "stage_kernel.h"

namespace ios {

void *stage_kernel_fn_light_persist() { return (void *)ios_stage_kernel<KV_LIGHT, true>; }

hipError_t stage_launch_light_persist(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s) {
  hipLaunchKernelGGL((ios_stage_kernel<KV_LIGHT, true>), dim3(grid), dim3(kThreads), lds, s, t, words, a);
  return hipGetLastError();
}

}  // namespace ios
