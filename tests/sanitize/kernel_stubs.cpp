// Host-only stand-ins for the device side of the library, so that the C-ABI
// host code (map construction, argument validation, planning, workspace
// sizing) can be built by a plain C++ compiler with AddressSanitizer and
// UndefinedBehaviorSanitizer.  A launch reports an error: the sanitizer
// driver only exercises paths that stop before any launch, and an
// unexpected MLKV_ERR_HIP would show that one was reached.
#include "kernels.h"

namespace mlkv {

namespace {
hipError_t no_device() { return hipErrorInvalidDevice; }
}  // namespace

hipError_t launch_pack(const PackParams&, hipStream_t) { return no_device(); }
hipError_t launch_layer_in(const LayerInParams&, int, hipStream_t) { return no_device(); }
hipError_t launch_layer_out(const LayerOutParams&, hipStream_t) { return no_device(); }
hipError_t launch_norm2(const NormParams&, hipStream_t) { return no_device(); }
hipError_t launch_qkv_epilogue(const QkvEpilogueParams&, hipStream_t) { return no_device(); }
hipError_t launch_gelu(const GeluParams&, hipStream_t) { return no_device(); }
hipError_t launch_residual(const ResidualParams&, hipStream_t) { return no_device(); }
hipError_t launch_append(const AppendParams&, int, int, hipStream_t) { return no_device(); }
hipError_t launch_rope_table(const RopeTableParams&, hipStream_t) { return no_device(); }
hipError_t launch_cache_rows(const CacheRowsParams&, int, hipStream_t) { return no_device(); }
hipError_t launch_append_rows(const AppendRowsParams&, int, int, hipStream_t) { return no_device(); }
hipError_t launch_prefill(const PrefillParams&, int, hipStream_t, hipEvent_t, hipEvent_t) {
  return no_device();
}
hipError_t launch_attention_main(const AttnParams&, int, hipStream_t, hipEvent_t, hipEvent_t,
                                 const SideProduct*) {
  return no_device();
}
hipError_t launch_attention_merge(const AttnParams&, int, hipStream_t, hipEvent_t) {
  return no_device();
}
hipError_t launch_fill(uint32_t*, size_t, uint32_t, hipStream_t) { return no_device(); }
hipError_t launch_empty_timed(int, int, hipStream_t, hipEvent_t, hipEvent_t) { return no_device(); }
hipError_t launch_stream_read_timed(const void*, size_t, uint32_t*, int, hipStream_t, hipEvent_t,
                                    hipEvent_t) {
  return no_device();
}
hipError_t scratch_for_current_device(hipStream_t, void** ptr) {
  *ptr = nullptr;
  return no_device();
}
// The planner's device facts, fixed at MI355X's: 256 compute units, three
// four-wave attention workgroups resident per compute unit.
int max_batch() { return 2048; }
int stage_floats() { return 8192; }
int resident_workgroups(int) { return 768; }
int wide_waves() { return 8; }
int compute_units() { return 256; }
int default_waves() { return 4; }

}  // namespace mlkv
