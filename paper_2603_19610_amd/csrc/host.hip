// Host-side helpers of the pvlm library: status strings, HIP error capture and
// the per-device compute-unit count used to size launches.
#include <map>
#include <mutex>
#include <tuple>
#include <set>
#include <string>
#include <utility>

#include "common.h"

namespace pvlm {

namespace {
thread_local std::string g_last_hip_error;
std::mutex g_info_mu;
constexpr int kMaxDevices = 64;
int g_cus[kMaxDevices] = {0};
int g_xcds[kMaxDevices] = {0};
std::mutex g_lds_mu;
std::set<std::pair<const void*, int>> g_lds_done;
std::mutex g_occ_mu;
std::map<std::tuple<int, const void*, int, int>, int> g_occ;  // (device, kernel, block, lds) -> per CU
std::mutex g_budget_mu;
std::map<std::pair<int, hipStream_t>, int> g_budget;  // (device, stream) -> compute units
}  // namespace

hipError_t allow_dynamic_lds(const void* kernel, int bytes) {
  std::lock_guard<std::mutex> lock(g_lds_mu);
  if (g_lds_done.count({kernel, bytes})) return hipSuccess;
  hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess) g_lds_done.insert({kernel, bytes});
  return e;
}

pvlm_status check_coresident(const void* kernel, int grid, int block, int lds,
                             hipStream_t stream) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_check(e);
  const std::tuple<int, const void*, int, int> key{dev, kernel, block, lds};
  int per_cu = 0;
  {
    std::lock_guard<std::mutex> lock(g_occ_mu);
    auto it = g_occ.find(key);
    if (it != g_occ.end()) per_cu = it->second;
  }
  if (per_cu == 0) {
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, block, (size_t)lds);
    if (e != hipSuccess) return hip_check(e);
    std::lock_guard<std::mutex> lock(g_occ_mu);
    g_occ[key] = per_cu;
  }
  DeviceInfo di;
  const pvlm_status st = device_info(&di, stream);
  if (st != PVLM_OK) return st;
  return (int64_t)per_cu * di.cus >= grid ? PVLM_OK : PVLM_ERR_UNSUPPORTED;
}

hipError_t launch_coresident(const void* kernel, dim3 grid, dim3 block, void** args, int lds,
                             hipStream_t stream) {
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cap);
  if (e != hipSuccess) return e;
  if (cap == hipStreamCaptureStatusNone) {
    DeviceInfo di;
    if (device_info(&di, stream) != PVLM_OK) return hipErrorInvalidDevice;
    if (!di.budgeted) return hipLaunchCooperativeKernel(kernel, grid, block, args, lds, stream);
  }
  return hipLaunchKernel(kernel, grid, block, args, lds, stream);
}

void set_hip_error(hipError_t e) {
  g_last_hip_error = std::string(hipGetErrorName(e)) + ": " + hipGetErrorString(e);
}

pvlm_status hip_check(hipError_t e) {
  if (e == hipSuccess) return PVLM_OK;
  set_hip_error(e);
  return PVLM_ERR_HIP;
}

pvlm_status device_info(DeviceInfo* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_check(e);
  if (dev < 0 || dev >= kMaxDevices) return PVLM_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_info_mu);
  if (g_cus[dev] == 0) {
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_check(e);
    if (cus <= 0) return PVLM_ERR_HIP;
    int xcds = 0;
    if (hipDeviceGetAttribute(&xcds, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || xcds < 1)
      xcds = 0;  // unknown: no exchange relies on sharing an XCD
    (void)hipGetLastError();
    g_xcds[dev] = xcds;
    g_cus[dev] = cus;
  }
  out->cus = g_cus[dev];
  out->xcds = g_xcds[dev];
  out->budgeted = false;
  return PVLM_OK;
}

pvlm_status device_info(DeviceInfo* out, hipStream_t stream) {
  const pvlm_status st = device_info(out);
  if (st != PVLM_OK) return st;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_check(e);
  std::lock_guard<std::mutex> lock(g_budget_mu);
  auto it = g_budget.find({dev, stream});
  if (it != g_budget.end() && it->second < out->cus) {
    out->cus = it->second;
    out->budgeted = true;
  }
  return PVLM_OK;
}

}  // namespace pvlm

extern "C" const char* pvlm_status_string(pvlm_status s) {
  switch (s) {
    case PVLM_OK: return "ok";
    case PVLM_ERR_NULL: return "a required pointer is NULL";
    case PVLM_ERR_SHAPE: return "inconsistent or out-of-range size argument";
    case PVLM_ERR_UNSUPPORTED: return "unsupported dtype, head dim or shape";
    case PVLM_ERR_WORKSPACE: return "workspace missing or too small";
    case PVLM_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

extern "C" const char* pvlm_last_hip_error(void) { return pvlm::g_last_hip_error.c_str(); }

extern "C" int pvlm_version(void) { return 1; }

extern "C" pvlm_status pvlm_set_stream_cu_budget(hipStream_t stream, int cus) {
  pvlm::DeviceInfo di;
  const pvlm_status st = pvlm::device_info(&di);
  if (st != PVLM_OK) return st;
  const int step = di.xcds > 0 ? di.xcds : 1;
  if (cus != 0 && (cus < step || cus > di.cus || cus % step != 0)) return PVLM_ERR_SHAPE;
  int dev = 0;
  PVLM_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lock(pvlm::g_budget_mu);
  if (cus == 0 || cus == di.cus) pvlm::g_budget.erase({dev, stream});
  else pvlm::g_budget[{dev, stream}] = cus;
  return PVLM_OK;
}

extern "C" int pvlm_stream_cu_budget(hipStream_t stream) {
  pvlm::DeviceInfo di;
  if (pvlm::device_info(&di, stream) != PVLM_OK) return 0;
  return di.budgeted ? di.cus : 0;
}
