// Test-only stand-ins for the gfx950 kernel launchers, so that the C-ABI
// layer (api.cpp) and the host planner can be built with host sanitizers
// without compiling the kernels.  Every launcher reports that no device
// code is present; the sanitizer driver only exercises paths that return
// before a launch, or treats HIP_ERROR as an expected outcome.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace splash {

hipError_t launch_plan(const PlanLaunch&, hipStream_t) { return hipErrorNoBinaryForGpu; }
hipError_t launch_attend(const AttendLaunch&, int32_t, hipStream_t) { return hipErrorNoBinaryForGpu; }
hipError_t launch_combine(const CombineLaunch&, hipStream_t) { return hipErrorNoBinaryForGpu; }
hipError_t launch_gather(const void*, const int32_t*, const int32_t*, int32_t, int32_t, int32_t, void*, hipStream_t) {
  return hipErrorNoBinaryForGpu;
}
hipError_t launch_topk_check(const int32_t*, const int32_t*, const int32_t*, const int32_t*, int32_t, int32_t, int32_t,
                             int32_t, int32_t, const void*, int32_t*, hipStream_t) {
  return hipErrorNoBinaryForGpu;
}
hipError_t launch_dop_pack_q(const void*, const void*, const int32_t*, int32_t, int32_t, void*, hipStream_t) {
  return hipErrorNoBinaryForGpu;
}
hipError_t launch_dop_unpack_q(const void*, int32_t, int32_t, int32_t, void*, hipStream_t) {
  return hipErrorNoBinaryForGpu;
}
hipError_t launch_dop_pack_out(const void*, int32_t, int32_t, int32_t, void*, hipStream_t) {
  return hipErrorNoBinaryForGpu;
}
hipError_t launch_dop_unpack_out(const void*, const int32_t*, int32_t, int32_t, void*, hipStream_t) {
  return hipErrorNoBinaryForGpu;
}
hipError_t launch_check(const int32_t*, const int32_t*, const void*, const int32_t*, const int32_t*, int32_t, int32_t,
                        int32_t, int32_t, int32_t*, hipStream_t) {
  return hipErrorNoBinaryForGpu;
}

}  // namespace splash
