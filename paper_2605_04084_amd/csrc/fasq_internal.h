// Host-side declarations shared by the libfasq sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <initializer_list>

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

// Tuned decode kernel for M <= 16.  Returns hipErrorNotSupported (without
// launching) when no tuned variant applies.
hipError_t launch_gemv(const Problem& p, const DeviceInfo& dev, hipStream_t stream);

// Tuned single-token kernel over several matrices in one launch (all with
// M = 1 and the same x, K, d and id width; at most 8).  hipErrorNotSupported
// (without launching) when the tuned kernel does not apply to the group.
hipError_t launch_gemv_m1_group(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream);
constexpr int kMaxBatchLaunch = 8;  // matrices per grouped launch

// Tuned MFMA prefill kernel.  hipErrorNotSupported when no variant applies.
hipError_t launch_gemm_mfma(const Problem& p, const DeviceInfo& dev, hipStream_t stream);

// Planning mode (per thread): while active, launchers record the name of the
// kernel instantiation they would launch instead of launching it.
struct Plan {
  bool active = false;
  char name[128] = {0};
};
Plan& plan();
// Record `base<params...>` as the planned kernel; returns true when planning.
bool plan_record(const char* base, std::initializer_list<int> params);

// Environment overrides used by tests and ablations: FASQ_FORCE_PATH=generic
// makes every call take the general kernel.
bool force_generic();

}  // namespace fasq
