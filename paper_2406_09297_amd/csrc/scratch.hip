// The library's own device scratch for callers that cannot allocate (code
// under graph capture, serving loops that forbid allocation): a file-scope
// device array holding what a decode workspace holds (arrival counters, run
// counts, the step's run list, split-run partials), used by
// mlkv_decode_step_noalloc in place of a caller's workspace.
//
// Each device the library runs on has its own copy of the array, at its own
// address, kept until the process ends.  The address is looked up once per
// device (with that device current) and cached; the array's name is never
// used as an address on the host.  On that first lookup the array is zero
// filled on the caller's stream (the arrival counters must start at zero;
// every decode call leaves them at zero again).
#include <hip/hip_runtime.h>

#include <mutex>
#include <stdint.h>

#include "kernels.h"

namespace mlkv {

namespace {

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t scratch_for_current_device(hipStream_t stream, void** ptr) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    if (!p) return hipErrorInvalidSymbol;
    err = launch_fill(static_cast<uint32_t*>(p), kScratchBytes / 4, 0u, stream);
    if (err != hipSuccess) return err;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace mlkv
