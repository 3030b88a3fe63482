// Decode GEMV kernels: 16-bit ids, 2 to 16 tokens.
#include "fasq_gemv_launch.h"

namespace fasq {
hipError_t launch_gemv_u16_m16(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream) {
  return launch_gemv_bits<16, 16>(ps, count, dev, stream);
}
}  // namespace fasq
