// Stage kernel variant KV_SEP, one workgroup per tile: the light tiles plus staged SEPCONV tiles.  One translation unit per
// (variant, launch kind) so that the kernels build in parallel (see
// stage_kernel.h and stage_launch.cpp).
#include "stage_kernel.h"

namespace ios {

void *stage_kernel_fn_sep() { return (void *)ios_stage_kernel<KV_SEP, false>; }

hipError_t stage_launch_sep(const int4 *t, int words, const StageArgs &a, int grid, int lds, hipStream_t s) {
  hipLaunchKernelGGL((ios_stage_kernel<KV_SEP, false>), dim3(grid), dim3(kThreads), lds, s, t, words, a);
  return hipGetLastError();
}

}  // namespace ios
