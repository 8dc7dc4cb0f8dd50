// Fused path: whole words resident in LDS, every layer in one launch.
#include <hip/hip_runtime.h>

#include "aecct_internal.h"
#include "device_common.h"

namespace aecct {

bool fused_supported(const Model &) { return false; }

hipError_t launch_fused(const Model &, const float *, int64_t, uint8_t *, float *, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace aecct
