// M = 1 decode kernels for 12-bit ids.
#include "fasq_gemv_m1_launch.h"

namespace fasq {
hipError_t launch_gemv_m1_u12(const Problem& p, const DeviceInfo& dev, hipStream_t stream) {
  return launch_gemv_m1_bits<12>(p, dev, stream);
}
}  // namespace fasq
