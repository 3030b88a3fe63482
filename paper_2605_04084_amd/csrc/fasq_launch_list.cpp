// libfasq C ABI: launch lists, the kernel launches of a sequence of calls
// recorded once and queued again on any stream of the same device.
#include "fasq.h"

#include <hip/hip_runtime.h>

#include <atomic>
#include <new>
#include <string>
#include <vector>

#include "fasq_internal.h"

struct fasq_launch_list {
  std::vector<fasq::RecordedLaunch> launches;
  int device = -1;                     // device of the recorded launches (-1: none yet)
  std::atomic<bool> recording{false};  // some thread records into the list
};

namespace fasq {

namespace {

struct Recorder {
  fasq_launch_list* list = nullptr;
  std::vector<RecordedLaunch>* into = nullptr;
};

Recorder& recorder() {
  static thread_local Recorder r;
  return r;
}

fasq_status list_fail(fasq_status s, const std::string& msg) {
  set_last_error(msg);
  return s;
}

}  // namespace

std::vector<RecordedLaunch>*& recording_into() { return recorder().into; }

}  // namespace fasq

extern "C" {

fasq_status fasq_launch_list_create(fasq_launch_list** list) {
  if (list == nullptr) return fasq::list_fail(FASQ_ERR_INVALID_ARG, "list is NULL");
  *list = new (std::nothrow) fasq_launch_list();
  if (*list == nullptr) return fasq::list_fail(FASQ_ERR_HOST_MEMORY, "cannot allocate a launch list");
  fasq::set_last_error("");
  return FASQ_OK;
}

fasq_status fasq_launch_list_begin(fasq_launch_list* list) {
  if (list == nullptr) return fasq::list_fail(FASQ_ERR_INVALID_ARG, "list is NULL");
  fasq::Recorder& r = fasq::recorder();
  if (r.list != nullptr) return fasq::list_fail(FASQ_ERR_INVALID_ARG, "the calling thread already records a launch list");
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fasq::list_fail(FASQ_ERR_HIP, std::string("querying the current device: ") + hipGetErrorString(e));
  if (!list->launches.empty() && list->device != dev)
    return fasq::list_fail(FASQ_ERR_INVALID_ARG, "the list holds launches for device " + std::to_string(list->device) +
                                                     ", the current device is " + std::to_string(dev));
  bool expected = false;
  if (!list->recording.compare_exchange_strong(expected, true))
    return fasq::list_fail(FASQ_ERR_INVALID_ARG, "the list is recording on another thread");
  list->device = dev;
  r.list = list;
  r.into = &list->launches;
  fasq::set_last_error("");
  return FASQ_OK;
}

fasq_status fasq_launch_list_end(fasq_launch_list* list) {
  if (list == nullptr) return fasq::list_fail(FASQ_ERR_INVALID_ARG, "list is NULL");
  fasq::Recorder& r = fasq::recorder();
  if (r.list != list) return fasq::list_fail(FASQ_ERR_INVALID_ARG, "the list is not recording on the calling thread");
  r.list = nullptr;
  r.into = nullptr;
  list->recording.store(false);
  fasq::set_last_error("");
  return FASQ_OK;
}

fasq_status fasq_launch_list_run(const fasq_launch_list* list, hipStream_t stream) {
  if (list == nullptr) return fasq::list_fail(FASQ_ERR_INVALID_ARG, "list is NULL");
  if (list->recording.load()) return fasq::list_fail(FASQ_ERR_INVALID_ARG, "the list is recording");
  if (fasq::recorder().list != nullptr)
    return fasq::list_fail(FASQ_ERR_INVALID_ARG, "the calling thread records a launch list");
  if (list->launches.empty()) {
    fasq::set_last_error("");
    return FASQ_OK;
  }
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fasq::list_fail(FASQ_ERR_HIP, std::string("querying the current device: ") + hipGetErrorString(e));
  if (dev != list->device)
    return fasq::list_fail(FASQ_ERR_INVALID_ARG, "the list was recorded on device " + std::to_string(list->device) +
                                                     ", the current device is " + std::to_string(dev));
  const size_t n = list->launches.size();
  for (size_t i = 0; i < n; ++i) {
    const fasq::RecordedLaunch& l = list->launches[i];
    e = hipLaunchKernel(l.kernel, l.grid, l.block, l.args->pointers(), l.lds, stream);
    if (e != hipSuccess)
      return fasq::list_fail(FASQ_ERR_HIP, "launch " + std::to_string(i) + " of " + std::to_string(n) + ": " +
                                               hipGetErrorString(e));
  }
  fasq::set_last_error("");
  return FASQ_OK;
}

int64_t fasq_launch_list_size(const fasq_launch_list* list) {
  return list == nullptr ? -1 : (int64_t)list->launches.size();
}

void fasq_launch_list_destroy(fasq_launch_list* list) {
  if (list == nullptr) return;
  fasq::Recorder& r = fasq::recorder();
  if (r.list == list) {
    r.list = nullptr;
    r.into = nullptr;
  }
  delete list;
}

}  // extern "C"
