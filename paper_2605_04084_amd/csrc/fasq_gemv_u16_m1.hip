// Decode GEMV kernels: 16-bit ids, one or two tokens (the row-streaming kernels).
#include "fasq_gemv_launch.h"

namespace fasq {
hipError_t launch_gemv_u16_m1(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream) {
  return launch_gemv_m1_bits<16>(ps, count, dev, stream);
}
}  // namespace fasq
