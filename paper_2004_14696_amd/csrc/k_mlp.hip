// MLP worker gradients (placeholder until the MFMA kernels land).
#include <hip/hip_runtime.h>

#include "dbw_internal.h"

namespace dbw {
hipError_t launch_mlp_grads(const MlpArgs&, hipStream_t) { return hipErrorNotSupported; }
}  // namespace dbw
