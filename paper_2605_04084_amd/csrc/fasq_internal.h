// Host-side declarations shared by the libfasq sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <initializer_list>
#include <memory>
#include <string>
#include <tuple>
#include <utility>
#include <vector>

namespace fasq {

// One validated call: y[M x N] = x[M x K] . W_hat^T.
struct Problem {
  const void* x;
  int64_t M, K, N;
  const void* idx;
  int idx_bits;
  int d;
  const void* codebook;
  int64_t C;
  void* y;
  int64_t S;  // sub-vectors per row, K / d
  int64_t R;  // bytes per packed index row
  int64_t cb_stride = 0;  // 0: one shared codebook; C * d: codebook s of subspace s at codebook + s * C * d
  // caller scratch the 16-row-tile decode kernel may split K with (fp32
  // partials; nullptr: no split)
  void* ws = nullptr;
  int64_t ws_bytes = 0;
};

// Properties of the current device, read once per device and cached.
struct DeviceInfo {
  int device = -1;
  int num_cus = 0;
  int lds_per_block = 0;  // bytes of LDS one workgroup may use
};
hipError_t device_info(DeviceInfo* out);

// Launchers.  Each returns hipSuccess or the launch error; none synchronizes.
hipError_t launch_reconstruct(const Problem& p, void* w, hipStream_t stream);
hipError_t launch_generic(const Problem& p, hipStream_t stream);

// Tuned decode kernel for M <= kGemvMaxTokens.  Returns hipErrorNotSupported
// (without launching) when no tuned variant applies.
hipError_t launch_gemv(const Problem& p, const DeviceInfo& dev, hipStream_t stream);

// Tuned decode kernels over one to kMaxBatchLaunch matrices in one launch,
// all with the same M <= kGemvMaxTokens, x, K, d and id width: the row-streaming kernel
// for M <= kM1MaxTokens where its codebook placement allows, else the
// 16-row-tile kernel.  hipErrorNotSupported (without launching) when
// neither applies.
hipError_t launch_gemv_group(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream);
constexpr int kMaxBatchLaunch = 8;  // matrices per grouped launch
constexpr int kM1MaxTokens = 2;     // tokens the row-streaming decode kernel takes at once
constexpr int kGemvMaxTokens = 16;  // tokens the 16-row-tile decode kernel takes at once

// Tuned MFMA prefill kernel.  hipErrorNotSupported when no variant applies.
// With a workspace of at least gemm_workspace_bytes() a grid too small for
// the CUs is also split along K (fp32 partials summed by a second kernel);
// otherwise the workspace is not touched.
hipError_t launch_gemm_mfma(const Problem& p, const DeviceInfo& dev, hipStream_t stream, void* workspace = nullptr,
                            int64_t workspace_bytes = 0);
int64_t gemm_workspace_bytes(const Problem& p, const DeviceInfo& dev);

// Whether the 16-row-tile decode kernel would stage x in slabs for p.
bool gemv_x_slabbed(const Problem& p);
// Whether a decode call that has a workspace is faster on the prefill GEMM
// with its K split (the measured crossover); see fasq_gemm.hip.
constexpr int kGemmFromTokens = 12;
bool decode_prefers_gemm(const Problem& p, const DeviceInfo& dev);
// Workspace bytes with which the 16-row-tile decode kernel splits K over
// workgroups for p (one matrix; 0 when it would not split).
int64_t gemv_split_workspace_bytes(const Problem& p);

// The paper's lookup-table GEMM (Alg. 3), kept for comparison with the MFMA
// GEMM.  hipErrorNotSupported when its tables do not fit in LDS.
hipError_t launch_gemm_lut(const Problem& p, hipStream_t stream);

// Per-subspace codebooks, one token: K split over workgroups whose codebooks
// fit in LDS, fp32 partials in `workspace`, then a fixed-order sum.
// hipErrorNotSupported when the tuned kernel does not apply.
int64_t gemv_sub_workspace_bytes(const Problem& p, const DeviceInfo& dev);
hipError_t launch_gemv_sub(const Problem& p, void* workspace, int64_t workspace_bytes, const DeviceInfo& dev,
                           hipStream_t stream);

// Once per device and kernel: check that the kernel declares no static LDS
// (its LDS-resident codebook is addressed from LDS address 0) and raise its
// dynamic-LDS limit to the 160 KB a gfx950 CU offers.  One bit per device
// ordinal; ordinals >= 64 repeat the set-up on every call.
template <typename K>
hipError_t prepare_kernel(K kernel) {
  static std::atomic<uint64_t> done{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? (uint64_t(1) << dev) : 0;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  hipFuncAttributes attr;
  e = hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(kernel));
  if (e != hipSuccess) return e;
  if (attr.sharedSizeBytes != 0) return hipErrorInvalidDeviceFunction;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                          160 * 1024);
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_acq_rel);
  return e;
}

// Calibration-free encoding of one weight matrix (validated arguments).
struct EncodeProblem {
  const void* w;  // fp16 [N x K]
  int64_t N, K;
  int d;
  int64_t C;
  int idx_bits;
  int64_t R;             // bytes per packed id row
  const void* init;      // fp16 [C x d]
  int iters;
  void* codebook;        // fp16 [C x d] out
  void* idx;             // packed ids out
  void* workspace;
};
int64_t encode_workspace_bytes(int64_t N, int64_t K, int d, int64_t C);
hipError_t launch_encode(const EncodeProblem& e, const DeviceInfo& dev, hipStream_t stream);

// Planning mode (per thread): while active, launchers record the name of the
// kernel instantiation they would launch instead of launching it.
struct Plan {
  bool active = false;
  char name[128] = {0};
};
Plan& plan();
// Record `base<params...>` as the planned kernel; returns true when planning.
bool plan_record(const char* base, std::initializer_list<int> params);

// ---------------------------------------------------------------------------
// Launch recording (fasq_launch_list_*).  While a list records on the calling
// thread, every kernel launch of the library is appended to it (kernel, grid,
// block, dynamic LDS bytes and a copy of the argument values) instead of
// being queued; fasq_launch_list_run queues the recorded launches later.
// ---------------------------------------------------------------------------
struct LaunchArgs {
  virtual ~LaunchArgs() = default;
  virtual void** pointers() = 0;  // one pointer per kernel parameter, as hipLaunchKernel takes them
};

// The argument values of one launch, held with the kernel's own parameter
// types (so each pointer addresses exactly the bytes of its parameter).
template <typename... T>
struct LaunchArgsOf final : LaunchArgs {
  std::tuple<T...> values;
  void* ptrs[sizeof...(T) > 0 ? sizeof...(T) : 1];
  explicit LaunchArgsOf(T... v) : values(v...) { point(std::index_sequence_for<T...>{}); }
  LaunchArgsOf(const LaunchArgsOf&) = delete;
  LaunchArgsOf& operator=(const LaunchArgsOf&) = delete;
  void** pointers() override { return ptrs; }

 private:
  template <size_t... I>
  void point(std::index_sequence<I...>) {
    ((ptrs[I] = static_cast<void*>(&std::get<I>(values))), ...);
  }
};

struct RecordedLaunch {
  const void* kernel;  // host-side handle of the __global__ function
  dim3 grid, block;
  size_t lds;
  std::unique_ptr<LaunchArgs> args;
};

// The launches the calling thread records into (nullptr: launches are queued).
std::vector<RecordedLaunch>*& recording_into();

// Queue kernel `kern` on `stream`, or record the launch when the calling
// thread records a launch list.  Returns the launch error (hipSuccess when
// recorded; hipErrorOutOfMemory when the host cannot hold the record).
template <typename... KArgs, typename... Args>
hipError_t launch_kernel(void (*kern)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t stream,
                         Args&&... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "one value per kernel parameter");
  if (std::vector<RecordedLaunch>* out = recording_into()) {
    try {
      out->push_back(RecordedLaunch{reinterpret_cast<const void*>(kern), grid, block, lds,
                                    std::make_unique<LaunchArgsOf<KArgs...>>(static_cast<KArgs>(args)...)});
    } catch (...) {
      return hipErrorOutOfMemory;
    }
    return hipSuccess;
  }
  hipLaunchKernelGGL(kern, grid, block, lds, stream, std::forward<Args>(args)...);
  return hipGetLastError();
}

// Sets the calling thread's fasq_last_error() text.
void set_last_error(const std::string& msg);

// Environment overrides used by tests and ablations: FASQ_FORCE_PATH=generic
// makes every call take the general kernel.
bool force_generic();

}  // namespace fasq
