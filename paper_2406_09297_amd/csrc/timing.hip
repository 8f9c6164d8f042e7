// References for the benchmarks' event timing: an empty kernel (the launch
// overhead) and a plain streaming read (the achievable read rate), each
// launched with an event pair recorded with its dispatch, the way the
// attention launches are timed.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "kernels.h"

namespace mlkv {

__global__ void empty_kernel() {}

hipError_t launch_empty_timed(int workgroups, int threads, hipStream_t stream, hipEvent_t start,
                              hipEvent_t stop) {
  hipExtLaunchKernelGGL(empty_kernel, dim3(workgroups), dim3(threads), 0, stream, start, stop, 0);
  return hipGetLastError();
}

// Streaming read of a buffer: every 16-byte piece loaded once (grid-stride,
// eight loads in flight per thread), folded into one value that is stored
// only if it equals an impossible pattern, so the loads cannot be dropped.
// The achievable read rate the attention kernels are compared with.
typedef uint32_t rd_u32x4 __attribute__((ext_vector_type(4)));
constexpr int kReadThreads = 256;
constexpr int kReadUnroll = 8;

__global__ __launch_bounds__(kReadThreads) void stream_read_kernel(const rd_u32x4* __restrict__ src,
                                                                   size_t n16, uint32_t* sink) {
  const size_t stride = static_cast<size_t>(gridDim.x) * kReadThreads;
  rd_u32x4 acc = {0u, 0u, 0u, 0u};
  size_t i = static_cast<size_t>(blockIdx.x) * kReadThreads + threadIdx.x;
  for (; i + (kReadUnroll - 1) * stride < n16; i += kReadUnroll * stride) {
    rd_u32x4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u];
  }
  for (; i < n16; i += stride) acc ^= __builtin_nontemporal_load(src + i);
  if ((acc[0] ^ acc[1] ^ acc[2] ^ acc[3]) == 0x9E3779B9u && acc[0] == 0x7F4A7C15u) sink[0] = acc[1];
}

hipError_t launch_stream_read_timed(const void* src, size_t bytes, uint32_t* sink, int workgroups,
                                    hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  hipExtLaunchKernelGGL(stream_read_kernel, dim3(workgroups), dim3(kReadThreads), 0, stream, start,
                        stop, 0, static_cast<const rd_u32x4*>(src), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace mlkv
