// Stand-ins for the kernel launchers of cardan_kernels.hip, linked into the
// sanitizer build of the host code (argument validation, planning, workspace
// layout) so that build needs no device code. Every launcher reports a HIP
// error; the CPU tests that run against this build never reach one.
#include <hip/hip_runtime.h>

#include "../../paper_2609_21137_amd/csrc/cardan_plan.h"

namespace cardan {
const void* route_kernel() { return nullptr; }
const void* expert_kernel(const Plan&) { return nullptr; }
hipError_t launch_route(const Plan&, const Args&, const Chain&, int, size_t, hipStream_t, hipEvent_t, hipEvent_t) {
  return hipErrorInvalidDeviceFunction;
}
hipError_t launch_expert(const Plan&, const Args&, const Chain&, int, size_t, hipStream_t, hipEvent_t, hipEvent_t) {
  return hipErrorInvalidDeviceFunction;
}
hipError_t launch_route_reset(const Plan&, const Args&, hipStream_t) { return hipErrorInvalidDeviceFunction; }
hipError_t launch_zero(void*, size_t, hipStream_t) { return hipErrorInvalidDeviceFunction; }
hipError_t launch_rmsnorm(hipStream_t, int, int, const float*, float, uint16_t*, hipEvent_t, hipEvent_t) {
  return hipErrorInvalidDeviceFunction;
}
}  // namespace cardan
