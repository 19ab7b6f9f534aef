// Stand-ins for the HIP kernel launchers, so that the library's host code
// (argument validation, work splitting, workspace layout, the C ABI) can be
// built alone with the host sanitizers and exercised on a machine without a
// GPU. Every launch reports that no device is present.
#include "bifattn_internal.h"

namespace bifattn {
hipError_t launch_partials(const PartialsParams&, int, int, int, int, hipStream_t,
                           const LaunchEvents&) {
  return hipErrorNoDevice;
}
hipError_t launch_combine(const CombineParams&, int, hipStream_t, const LaunchEvents&) {
  return hipErrorNoDevice;
}
hipError_t launch_append(const AppendParams&, int, int, hipStream_t, const LaunchEvents&) {
  return hipErrorNoDevice;
}
hipError_t launch_standard(const PartialsParams&, int, int, int, hipStream_t,
                           const LaunchEvents&) {
  return hipErrorNoDevice;
}
hipError_t launch_ctx_large(const PartialsParams&, int, int, hipStream_t, const LaunchEvents&) {
  return hipErrorNoDevice;
}
hipError_t scratch_address(int, void**) { return hipErrorNoDevice; }
}  // namespace bifattn
