// Launchers that enqueue nothing, linked in place of the kernels when the C ABI
// layer is built with host sanitizers for the CPU tests: every call those tests
// make fails validation or has no work, so no launcher is reached.
#include "ress_internal.h"

namespace ress {
hipError_t launch_pool(const PoolParams &, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_proj(const ProjParams &, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_select(const SelectParams &, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_attn(const AttnParams &, int, int, bool, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_drift_sq(const DriftSqParams &, hipStream_t) { return hipErrorInvalidValue; }
}  // namespace ress
