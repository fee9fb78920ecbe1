// Test-only stand-ins for the GPU launchers, for host-only builds of the planner sources under the
// address, undefined-behaviour and thread sanitizers.  The host-side drivers never reach a launch
// (they exercise validation, planning, error paths and the host-only rows), so every stub reports
// that launching is unavailable in this build.
#include "internal.h"

namespace wavepp {

hipError_t launch_append(const DevPlan&, const void*, const void*, void*, void*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_attention(const DevPlan&, const void*, const void*, const void*, void*, float*, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_merge(const DevPlan&, void*, float*, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_upload(const void*, void*, size_t, hipStream_t) { return hipErrorNotSupported; }
hipError_t noalloc_scratch(void** ptr) {
  *ptr = nullptr;
  return hipErrorNotSupported;
}
hipError_t launch_kda_prefill(const KdaDevPlan&, const void*, const void*, const void*, const float*, const float*,
                              float*, void*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace wavepp
