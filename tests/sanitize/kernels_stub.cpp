// Host-only stand-ins for the kernel launchers, for the sanitizer build of the
// library's host code (planner and C-ABI), which the CPU tests load instead of
// the HIP build: every launch reports hipErrorNotSupported, so a device call
// through the sanitizer build fails loudly instead of computing anything.
#include "kernels.h"

namespace mstar {
hipError_t launch_tiles(const KArgs&, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_cascade(const KArgs&, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_append(const AArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_few(const KArgs&, int, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_f32(const KArgs&, int, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_merge(const MArgs&, int, bool, hipStream_t) { return hipErrorNotSupported; }
hipError_t scratch_buffer(void** ptr) {
    *ptr = nullptr;
    return hipErrorNotSupported;
}
}  // namespace mstar
