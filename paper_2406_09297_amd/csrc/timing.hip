// Launch-overhead reference for the benchmarks' event timing: an empty
// kernel launched with an event pair recorded with its dispatch, the way the
// attention launches are timed.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace mlkv {

__global__ void empty_kernel() {}

hipError_t launch_empty_timed(int workgroups, int threads, hipStream_t stream, hipEvent_t start,
                              hipEvent_t stop) {
  hipExtLaunchKernelGGL(empty_kernel, dim3(workgroups), dim3(threads), 0, stream, start, stop, 0);
  return hipGetLastError();
}

}  // namespace mlkv
