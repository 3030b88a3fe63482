// M = 1 decode kernels for 16-bit ids.
#include "fasq_gemv_m1_launch.h"

namespace fasq {
hipError_t launch_gemv_m1_u16(const Problem& p, const DeviceInfo& dev, hipStream_t stream) {
  return launch_gemv_m1_bits<16>(p, dev, stream);
}
}  // namespace fasq
