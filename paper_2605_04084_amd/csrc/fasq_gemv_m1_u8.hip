// M = 1 decode kernels for 8-bit ids.
#include "fasq_gemv_m1_launch.h"

namespace fasq {
hipError_t launch_gemv_m1_u8(const Problem& p, const DeviceInfo& dev, hipStream_t stream) {
  return launch_gemv_m1_bits<8>(p, dev, stream);
}
}  // namespace fasq
