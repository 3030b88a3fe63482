// libfasq C ABI: argument validation, kernel selection, error reporting.
#include "fasq.h"

#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>

#include "fasq_internal.h"

namespace fasq {

hipError_t launch_gemv_u8_m1(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream);
hipError_t launch_gemv_u12_m1(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream);
hipError_t launch_gemv_u16_m1(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream);
hipError_t launch_gemv_u8_m16(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream);
hipError_t launch_gemv_u12_m16(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream);
hipError_t launch_gemv_u16_m16(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream);

namespace {

hipError_t launch_gemv_m1_group(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream) {
  switch (ps[0].idx_bits) {
    case 8: return launch_gemv_u8_m1(ps, count, dev, stream);
    case 12: return launch_gemv_u12_m1(ps, count, dev, stream);
    default: return launch_gemv_u16_m1(ps, count, dev, stream);
  }
}

// Whether the row-streaming kernel would take matrix p alone (nothing is
// launched: the launcher runs in planning mode).
bool m1_takes_alone(const Problem& p, const DeviceInfo& dev) {
  Plan& pl = plan();
  const Plan saved = pl;
  pl.active = true;
  const hipError_t e = launch_gemv_m1_group(&p, 1, dev, nullptr);
  pl = saved;
  return e == hipSuccess;
}

}  // namespace

hipError_t launch_gemv_group(const Problem* ps, int count, const DeviceInfo& dev, hipStream_t stream) {
  const Problem& p = ps[0];
  if (p.M < 1 || p.M > kGemvMaxTokens) return hipErrorNotSupported;
  if (p.M <= kM1MaxTokens) {  // the row-streaming kernel when its codebook placement allows
    hipError_t e = launch_gemv_m1_group(ps, count, dev, stream);
    if (e != hipErrorNotSupported || p.M == 1) return e;
    // Two tokens and a group the two-token kernel cannot take (a codebook
    // too large for LDS).  A member that it would take alone must not run
    // on the 16-row-tile kernel here: the two kernels add their fp32
    // partials in different orders, and a grouped output has to equal the
    // single call's bit for bit.  The caller then runs the matrices one by
    // one.
    if (count > 1)
      for (int i = 0; i < count; ++i)
        if (m1_takes_alone(ps[i], dev)) return hipErrorNotSupported;
  }
  switch (p.idx_bits) {
    case 8: return launch_gemv_u8_m16(ps, count, dev, stream);
    case 12: return launch_gemv_u12_m16(ps, count, dev, stream);
    default: return launch_gemv_u16_m16(ps, count, dev, stream);
  }
}

hipError_t launch_gemv(const Problem& p, const DeviceInfo& dev, hipStream_t stream) {
  return launch_gemv_group(&p, 1, dev, stream);
}

namespace {

thread_local std::string t_last_error;

constexpr int kMaxDevices = 64;
std::mutex g_dev_mutex;
DeviceInfo g_dev[kMaxDevices];

fasq_status fail(fasq_status s, const std::string& msg) {
  t_last_error = msg;
  return s;
}

fasq_status hip_fail(const char* what, hipError_t e) {
  std::string m = what;
  m += ": ";
  m += hipGetErrorString(e);
  return fail(FASQ_ERR_HIP, m);
}

// Validation shared by the three compute entry points.  No HIP call is made.
fasq_status validate(int64_t M, int64_t K, int64_t N, int idx_bits, int d, int64_t C, const void* x,
                     const void* idx, const void* codebook, const void* y, bool need_x) {
  if (M < 1 || K < 1 || N < 1) return fail(FASQ_ERR_INVALID_ARG, "M, K and N must be >= 1");
  if (d < 1) return fail(FASQ_ERR_INVALID_ARG, "d must be >= 1");
  if (K % d != 0) return fail(FASQ_ERR_INVALID_ARG, "K must be a multiple of d");
  if (idx_bits != 8 && idx_bits != 12 && idx_bits != 16)
    return fail(FASQ_ERR_INVALID_ARG, "idx_bits must be 8, 12 or 16");
  if (C < 1 || C > (int64_t(1) << idx_bits))
    return fail(FASQ_ERR_INVALID_ARG, "C must lie in [1, 2^idx_bits]");
  if ((need_x && x == nullptr) || idx == nullptr || codebook == nullptr || y == nullptr)
    return fail(FASQ_ERR_INVALID_ARG, "a buffer pointer is NULL");
  // the largest flat index any kernel forms must fit in int64
  if (M > (int64_t(1) << 40) / K || N > (int64_t(1) << 40) / K)
    return fail(FASQ_ERR_INVALID_ARG, "problem too large");
  return FASQ_OK;
}

Problem make_problem(const void* x, int64_t M, int64_t K, int64_t N, const void* idx, int idx_bits, int d,
                     const void* codebook, int64_t C, void* y) {
  Problem p;
  p.x = x;
  p.M = M;
  p.K = K;
  p.N = N;
  p.idx = idx;
  p.idx_bits = idx_bits;
  p.d = d;
  p.codebook = codebook;
  p.C = C;
  p.y = y;
  p.S = K / d;
  p.R = (p.S * idx_bits + 7) / 8;
  return p;
}

enum class Regime { kGemv, kGemm };

fasq_status run(const Problem& p, Regime regime, hipStream_t stream, void* workspace = nullptr,
               int64_t workspace_bytes = 0) {
  DeviceInfo dev;
  hipError_t e = device_info(&dev);
  if (e != hipSuccess) return hip_fail("querying the current device", e);
  e = hipErrorNotSupported;
  if (!force_generic()) {
    // a decode call with a workspace goes to the GEMM where that is faster
    const bool to_gemm = regime == Regime::kGemv && workspace != nullptr && decode_prefers_gemm(p, dev) &&
                         workspace_bytes >= gemm_workspace_bytes(p, dev);
    if (regime == Regime::kGemv && !to_gemm) {
      // the workspace also lets the 16-row-tile decode kernel split K
      Problem q = p;
      q.ws = workspace;
      q.ws_bytes = workspace_bytes;
      e = launch_gemv(q, dev, stream);
    }
    if (e == hipErrorNotSupported) e = launch_gemm_mfma(p, dev, stream, workspace, workspace_bytes);
  }
  if (e == hipErrorNotSupported) e = launch_generic(p, stream);
  if (e != hipSuccess) return hip_fail("kernel launch", e);
  t_last_error.clear();
  return FASQ_OK;
}

}  // namespace

hipError_t device_info(DeviceInfo* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < kMaxDevices) {
    std::lock_guard<std::mutex> lock(g_dev_mutex);
    if (g_dev[dev].device == dev) {
      *out = g_dev[dev];
      return hipSuccess;
    }
  }
  DeviceInfo info;
  info.device = dev;
  e = hipDeviceGetAttribute(&info.num_cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&info.lds_per_block, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < kMaxDevices) {
    std::lock_guard<std::mutex> lock(g_dev_mutex);
    g_dev[dev] = info;
  }
  *out = info;
  return hipSuccess;
}

Plan& plan() {
  static thread_local Plan p;
  return p;
}

bool plan_record(const char* base, std::initializer_list<int> params) {
  Plan& p = plan();
  if (!p.active) return false;
  int n = std::snprintf(p.name, sizeof(p.name), "%s<", base);
  bool first = true;
  for (int v : params) {
    if (n < 0 || n >= (int)sizeof(p.name)) break;
    n += std::snprintf(p.name + n, sizeof(p.name) - n, first ? "%d" : ", %d", v);
    first = false;
  }
  if (n >= 0 && n < (int)sizeof(p.name) - 1) std::snprintf(p.name + n, sizeof(p.name) - n, ">");
  return true;
}

void set_last_error(const std::string& msg) { t_last_error = msg; }

bool force_generic() {
  const char* v = std::getenv("FASQ_FORCE_PATH");
  return v != nullptr && std::strcmp(v, "generic") == 0;
}

}  // namespace fasq

using fasq::Problem;

extern "C" {

fasq_status fasq_pq_gemv(const void* x, int64_t M, int64_t K, int64_t N, const void* idx, int idx_bits, int d,
                         const void* codebook, int64_t C, void* y, hipStream_t stream) {
  fasq_status s = fasq::validate(M, K, N, idx_bits, d, C, x, idx, codebook, y, true);
  if (s != FASQ_OK) return s;
  return fasq::run(fasq::make_problem(x, M, K, N, idx, idx_bits, d, codebook, C, y), fasq::Regime::kGemv, stream);
}

fasq_status fasq_pq_gemv_batched(const void* x, int64_t M, int64_t K, int count, const void* const* idx,
                                 const int64_t* N, const void* const* codebook, const int64_t* C, void* const* y,
                                 int idx_bits, int d, hipStream_t stream) {
  if (count < 1) return fasq::fail(FASQ_ERR_INVALID_ARG, "count must be >= 1");
  if (idx == nullptr || N == nullptr || codebook == nullptr || C == nullptr || y == nullptr)
    return fasq::fail(FASQ_ERR_INVALID_ARG, "a matrix array is NULL");
  for (int i = 0; i < count; ++i) {
    fasq_status s = fasq::validate(M, K, N[i], idx_bits, d, C[i], x, idx[i], codebook[i], y[i], true);
    if (s != FASQ_OK) {
      fasq::t_last_error = "matrix " + std::to_string(i) + ": " + fasq::t_last_error;
      return s;
    }
  }
  fasq::DeviceInfo dev;
  hipError_t e = fasq::device_info(&dev);
  if (e != hipSuccess) return fasq::hip_fail("querying the current device", e);
  Problem ps[fasq::kMaxBatchLaunch];
  for (int off = 0; off < count; off += fasq::kMaxBatchLaunch) {
    const int n = count - off < fasq::kMaxBatchLaunch ? count - off : fasq::kMaxBatchLaunch;
    for (int i = 0; i < n; ++i)
      ps[i] = fasq::make_problem(x, M, K, N[off + i], idx[off + i], idx_bits, d, codebook[off + i], C[off + i],
                                 y[off + i]);
    e = hipErrorNotSupported;
    if (!fasq::force_generic()) e = fasq::launch_gemv_group(ps, n, dev, stream);
    if (e == hipErrorNotSupported) {
      for (int i = 0; i < n; ++i) {
        fasq_status s = fasq::run(ps[i], fasq::Regime::kGemv, stream);
        if (s != FASQ_OK) return s;
      }
    } else if (e != hipSuccess) {
      return fasq::hip_fail("kernel launch", e);
    }
  }
  fasq::t_last_error.clear();
  return FASQ_OK;
}

fasq_status fasq_pq_gemm(const void* x, int64_t M, int64_t K, int64_t N, const void* idx, int idx_bits, int d,
                         const void* codebook, int64_t C, void* y, hipStream_t stream) {
  fasq_status s = fasq::validate(M, K, N, idx_bits, d, C, x, idx, codebook, y, true);
  if (s != FASQ_OK) return s;
  return fasq::run(fasq::make_problem(x, M, K, N, idx, idx_bits, d, codebook, C, y), fasq::Regime::kGemm, stream);
}

fasq_status fasq_pq_gemm_lut(const void* x, int64_t M, int64_t K, int64_t N, const void* idx, int idx_bits, int d,
                             const void* codebook, int64_t C, void* y, hipStream_t stream) {
  fasq_status s = fasq::validate(M, K, N, idx_bits, d, C, x, idx, codebook, y, true);
  if (s != FASQ_OK) return s;
  hipError_t e = fasq::launch_gemm_lut(fasq::make_problem(x, M, K, N, idx, idx_bits, d, codebook, C, y), stream);
  if (e == hipErrorNotSupported)
    return fasq::fail(FASQ_ERR_UNSUPPORTED, "the lookup-table GEMM needs d in {1, 2, 4, 8} and C <= 2048");
  if (e != hipSuccess) return fasq::hip_fail("kernel launch", e);
  fasq::t_last_error.clear();
  return FASQ_OK;
}

fasq_status fasq_pq_reconstruct(const void* idx, int64_t N, int64_t K, int idx_bits, int d, const void* codebook,
                                int64_t C, void* w, hipStream_t stream) {
  fasq_status s = fasq::validate(1, K, N, idx_bits, d, C, nullptr, idx, codebook, w, false);
  if (s != FASQ_OK) return s;
  Problem p = fasq::make_problem(nullptr, 1, K, N, idx, idx_bits, d, codebook, C, nullptr);
  hipError_t e = fasq::launch_reconstruct(p, w, stream);
  if (e != hipSuccess) return fasq::hip_fail("kernel launch", e);
  fasq::t_last_error.clear();
  return FASQ_OK;
}

int64_t fasq_idx_row_bytes(int64_t K, int d, int idx_bits) {
  if (K < 1 || d < 1 || K % d != 0) return -1;
  if (idx_bits != 8 && idx_bits != 12 && idx_bits != 16) return -1;
  return (K / d * idx_bits + 7) / 8;
}

const char* fasq_status_string(fasq_status s) {
  switch (s) {
    case FASQ_OK: return "FASQ_OK";
    case FASQ_ERR_INVALID_ARG: return "FASQ_ERR_INVALID_ARG";
    case FASQ_ERR_UNSUPPORTED: return "FASQ_ERR_UNSUPPORTED";
    case FASQ_ERR_HIP: return "FASQ_ERR_HIP";
    case FASQ_ERR_HOST_MEMORY: return "FASQ_ERR_HOST_MEMORY";
  }
  return "FASQ_UNKNOWN_STATUS";
}

const char* fasq_last_error(void) { return fasq::t_last_error.c_str(); }

int fasq_abi_version(void) { return FASQ_ABI_VERSION; }

int64_t fasq_pq_gemv_ex_workspace_bytes(int64_t M, int64_t K, int64_t N, int idx_bits, int d, int64_t C,
                                        int64_t cb_stride) {
  const void* fake = reinterpret_cast<const void*>(uintptr_t(1) << 20);
  if (fasq::validate(M, K, N, idx_bits, d, C, fake, fake, fake, fake, true) != FASQ_OK) return -1;
  if (cb_stride != 0 && cb_stride != C * d) return -1;
  Problem p = fasq::make_problem(fake, M, K, N, fake, idx_bits, d, fake, C, const_cast<void*>(fake));
  p.cb_stride = cb_stride;
  fasq::DeviceInfo dev;
  if (fasq::device_info(&dev) != hipSuccess) return -1;
  if (cb_stride != 0) return fasq::gemv_sub_workspace_bytes(p, dev);
  // one shared codebook: a workspace serves the GEMM when the decode kernels
  // hand it the call, or when the GEMM with its K split is the faster one,
  // and the 16-row-tile decode kernel when it splits K
  if (fasq::force_generic()) return 0;
  const char* plan = fasq_pq_plan(0, M, K, N, idx_bits, d, C);
  if (std::strncmp(plan, "k_gemm_mfma", 11) == 0 || fasq::decode_prefers_gemm(p, dev))
    return fasq::gemm_workspace_bytes(p, dev);
  if (std::strncmp(plan, "k_gemv<", 7) == 0) return fasq::gemv_split_workspace_bytes(p);
  return 0;
}

fasq_status fasq_pq_gemv_ex(const void* x, int64_t M, int64_t K, int64_t N, const void* idx, int idx_bits, int d,
                            const void* codebook, int64_t C, int64_t cb_stride, void* y, void* workspace,
                            int64_t workspace_bytes, hipStream_t stream) {
  fasq_status s = fasq::validate(M, K, N, idx_bits, d, C, x, idx, codebook, y, true);
  if (s != FASQ_OK) return s;
  if (cb_stride != 0 && cb_stride != C * d)
    return fasq::fail(FASQ_ERR_INVALID_ARG, "cb_stride must be 0 (one shared codebook) or C * d (one per subspace)");
  if (workspace_bytes < 0) return fasq::fail(FASQ_ERR_INVALID_ARG, "workspace_bytes must be >= 0");
  Problem p = fasq::make_problem(x, M, K, N, idx, idx_bits, d, codebook, C, y);
  if (cb_stride == 0) return fasq::run(p, fasq::Regime::kGemv, stream, workspace, workspace_bytes);
  p.cb_stride = cb_stride;
  fasq::DeviceInfo dev;
  hipError_t e = fasq::device_info(&dev);
  if (e != hipSuccess) return fasq::hip_fail("querying the current device", e);
  e = hipErrorNotSupported;
  if (!fasq::force_generic()) e = fasq::launch_gemv_sub(p, workspace, workspace_bytes, dev, stream);
  if (e == hipErrorNotSupported) e = fasq::launch_generic(p, stream);
  if (e != hipSuccess) return fasq::hip_fail("kernel launch", e);
  fasq::t_last_error.clear();
  return FASQ_OK;
}

int64_t fasq_pq_gemm_ex_workspace_bytes(int64_t M, int64_t K, int64_t N, int idx_bits, int d, int64_t C) {
  const void* fake = reinterpret_cast<const void*>(uintptr_t(1) << 20);
  if (fasq::validate(M, K, N, idx_bits, d, C, fake, fake, fake, fake, true) != FASQ_OK) return -1;
  Problem p = fasq::make_problem(fake, M, K, N, fake, idx_bits, d, fake, C, const_cast<void*>(fake));
  fasq::DeviceInfo dev;
  if (fasq::device_info(&dev) != hipSuccess) return -1;
  return fasq::gemm_workspace_bytes(p, dev);
}

fasq_status fasq_pq_gemm_ex(const void* x, int64_t M, int64_t K, int64_t N, const void* idx, int idx_bits, int d,
                            const void* codebook, int64_t C, void* y, void* workspace, int64_t workspace_bytes,
                            hipStream_t stream) {
  fasq_status s = fasq::validate(M, K, N, idx_bits, d, C, x, idx, codebook, y, true);
  if (s != FASQ_OK) return s;
  if (workspace_bytes < 0) return fasq::fail(FASQ_ERR_INVALID_ARG, "workspace_bytes must be >= 0");
  return fasq::run(fasq::make_problem(x, M, K, N, idx, idx_bits, d, codebook, C, y), fasq::Regime::kGemm, stream,
                   workspace, workspace_bytes);
}

int64_t fasq_pq_encode_workspace_bytes(int64_t N, int64_t K, int d, int64_t C) {
  if (N < 1 || K < 1 || d < 1 || K % d != 0 || C < 1 || C > (int64_t(1) << 16)) return -1;
  if (N > (int64_t(1) << 40) / K) return -1;
  return fasq::encode_workspace_bytes(N, K, d, C);
}

fasq_status fasq_pq_encode(const void* w, int64_t N, int64_t K, int d, int64_t C, int idx_bits,
                           const void* init_codebook, int iters, void* codebook, void* idx, void* workspace,
                           int64_t workspace_bytes, hipStream_t stream) {
  using fasq::fail;
  if (N < 1 || K < 1) return fail(FASQ_ERR_INVALID_ARG, "N and K must be >= 1");
  if (d < 1) return fail(FASQ_ERR_INVALID_ARG, "d must be >= 1");
  if (K % d != 0) return fail(FASQ_ERR_INVALID_ARG, "K must be a multiple of d");
  if (idx_bits != 8 && idx_bits != 12 && idx_bits != 16)
    return fail(FASQ_ERR_INVALID_ARG, "idx_bits must be 8, 12 or 16");
  if (C < 1 || C > (int64_t(1) << idx_bits)) return fail(FASQ_ERR_INVALID_ARG, "C must lie in [1, 2^idx_bits]");
  if (iters < 0) return fail(FASQ_ERR_INVALID_ARG, "iters must be >= 0");
  if (w == nullptr || init_codebook == nullptr || codebook == nullptr || idx == nullptr || workspace == nullptr)
    return fail(FASQ_ERR_INVALID_ARG, "a buffer pointer is NULL");
  if (N > (int64_t(1) << 40) / K) return fail(FASQ_ERR_INVALID_ARG, "problem too large");
  if ((reinterpret_cast<uintptr_t>(w) | reinterpret_cast<uintptr_t>(init_codebook) |
       reinterpret_cast<uintptr_t>(codebook)) & 1)
    return fail(FASQ_ERR_INVALID_ARG, "fp16 buffers must be 2-byte aligned");
  if (reinterpret_cast<uintptr_t>(workspace) & 7) return fail(FASQ_ERR_INVALID_ARG, "workspace must be 8-byte aligned");
  if (workspace_bytes < fasq::encode_workspace_bytes(N, K, d, C))
    return fail(FASQ_ERR_INVALID_ARG, "workspace smaller than fasq_pq_encode_workspace_bytes()");
  if (d > 16) return fail(FASQ_ERR_UNSUPPORTED, "the encoder handles d <= 16");
  fasq::DeviceInfo dev;
  hipError_t e = fasq::device_info(&dev);
  if (e != hipSuccess) return fasq::hip_fail("querying the current device", e);
  fasq::EncodeProblem ep;
  ep.w = w;
  ep.N = N;
  ep.K = K;
  ep.d = d;
  ep.C = C;
  ep.idx_bits = idx_bits;
  ep.R = (K / d * idx_bits + 7) / 8;
  ep.init = init_codebook;
  ep.iters = iters;
  ep.codebook = codebook;
  ep.idx = idx;
  ep.workspace = workspace;
  e = fasq::launch_encode(ep, dev, stream);
  if (e != hipSuccess) return fasq::hip_fail("kernel launch", e);
  fasq::t_last_error.clear();
  return FASQ_OK;
}

const char* fasq_pq_plan(int regime, int64_t M, int64_t K, int64_t N, int idx_bits, int d, int64_t C) {
  // Placeholder, suitably aligned, never dereferenced: nothing is launched.
  const void* fake = reinterpret_cast<const void*>(uintptr_t(1) << 20);
  fasq_status s = fasq::validate(M, K, N, idx_bits, d, C, fake, fake, fake, fake, true);
  if (s != FASQ_OK) return "";
  fasq::Plan& pl = fasq::plan();
  pl.active = true;
  pl.name[0] = 0;
  Problem p = fasq::make_problem(fake, M, K, N, fake, idx_bits, d, fake, C, const_cast<void*>(fake));
  if (regime == 2) {  // a grouped decode launch: two matrices of these sizes
    Problem ps[2] = {p, p};
    fasq::DeviceInfo dev;
    hipError_t e = fasq::device_info(&dev);
    if (e == hipSuccess && !fasq::force_generic()) e = fasq::launch_gemv_group(ps, 2, dev, nullptr);
    else e = hipErrorNotSupported;
    s = e == hipSuccess ? FASQ_OK : e == hipErrorNotSupported ? fasq::run(p, fasq::Regime::kGemv, nullptr)
                                                             : FASQ_ERR_HIP;
  } else {
    s = fasq::run(p, regime == 1 ? fasq::Regime::kGemm : fasq::Regime::kGemv, nullptr);
  }
  pl.active = false;
  if (s != FASQ_OK) return "";
  return pl.name;
}

}  // extern "C"
