// fasq_pq_gemv_ex_noalloc: fasq_pq_gemv_ex with the library's own scratch
// memory, for callers that cannot allocate device memory.
//
// The scratch is one file-scope device array per GPU, loaded with the code
// object.  Host code never passes the array's name to a kernel (on the host
// it is only a stand-in for the symbol): its device address is looked up
// once per device with hipGetSymbolAddress and kept, and that address is the
// workspace every call on the device hands to the kernels.
#include "fasq.h"

#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "fasq_internal.h"

namespace fasq {

constexpr int64_t kScratchBytes = FASQ_NOALLOC_SCRATCH_BYTES;

// One copy per GPU, each at its own device address; host code uses only the
// address looked up below, never this name.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// The device address of the current device's scratch array, looked up on
// the first call on that device.
hipError_t scratch_of_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

}  // namespace fasq

extern "C" {

int64_t fasq_noalloc_scratch_bytes(void) { return fasq::kScratchBytes; }

fasq_status fasq_pq_gemv_ex_noalloc(const void* x, int64_t M, int64_t K, int64_t N, const void* idx, int idx_bits,
                                    int d, const void* codebook, int64_t C, int64_t cb_stride, void* y,
                                    hipStream_t stream) {
  // argument checks first (fasq_pq_gemv_ex repeats them; nothing is launched
  // before they pass)
  const int64_t need = fasq_pq_gemv_ex_workspace_bytes(M, K, N, idx_bits, d, C, cb_stride);
  if (need < 0) {
    // invalid sizes: let fasq_pq_gemv_ex name the failed check (it launches nothing)
    return fasq_pq_gemv_ex(x, M, K, N, idx, idx_bits, d, codebook, C, cb_stride, y, nullptr, 0, stream);
  }
  if (need > fasq::kScratchBytes) {
    fasq::set_last_error("these sizes need " + std::to_string(need) + " bytes of scratch, more than the " +
                         std::to_string(fasq::kScratchBytes) +
                         " bytes the library holds per device; call fasq_pq_gemv_ex with a workspace");
    return FASQ_ERR_INVALID_ARG;
  }
  void* ws = nullptr;
  if (need > 0) {
    const hipError_t e = fasq::scratch_of_current_device(&ws);
    if (e != hipSuccess) {
      fasq::set_last_error(std::string("looking up the scratch array: ") + hipGetErrorString(e));
      return FASQ_ERR_HIP;
    }
  }
  return fasq_pq_gemv_ex(x, M, K, N, idx, idx_bits, d, codebook, C, cb_stride, y, ws,
                         need > 0 ? fasq::kScratchBytes : 0, stream);
}

}  // extern "C"
