// Status strings, per-thread error messages and the per-device error word.
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "../../include/agrl.h"
#include "common.hpp"

// One error word per device (a __device__ variable has one instance per GPU).
__device__ int agrl_device_error_word = 0;

namespace agrl {

static thread_local char g_last_error[256] = "";

void set_last_error(const char* msg) {
  snprintf(g_last_error, sizeof g_last_error, "%s", msg ? msg : "");
}

int hip_status(hipError_t e) {
  if (e == hipSuccess) return AGRL_OK;
  char buf[200];
  snprintf(buf, sizeof buf, "HIP: %s", hipGetErrorString(e));
  set_last_error(buf);
  return AGRL_E_HIP;
}

namespace {
constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
int* g_err_ptr[kMaxDevices];
int g_cu[kMaxDevices];
}  // namespace

static int current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return -1;
  return dev;
}

static void init_device(int dev) {
  void* p = nullptr;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(agrl_device_error_word)) == hipSuccess)
    g_err_ptr[dev] = (int*)p;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) == hipSuccess) g_cu[dev] = prop.multiProcessorCount;
  if (g_cu[dev] <= 0) g_cu[dev] = 256;
}

int* device_error_ptr() {
  int dev = current_device();
  if (dev < 0) return nullptr;
  std::call_once(g_once[dev], init_device, dev);
  return g_err_ptr[dev];
}

int device_cu_count() {
  int dev = current_device();
  if (dev < 0) return 256;
  std::call_once(g_once[dev], init_device, dev);
  return g_cu[dev];
}

}  // namespace agrl

extern "C" const char* agrl_status_string(int status) {
  switch (status) {
    case AGRL_OK: return "ok";
    case AGRL_E_NULL: return "a required pointer is NULL";
    case AGRL_E_SHAPE: return "invalid size";
    case AGRL_E_DTYPE: return "invalid dtype";
    case AGRL_E_FLAGS: return "invalid option or clip bound";
    case AGRL_E_WORKSPACE: return "workspace missing or too small";
    case AGRL_E_HIP: return "HIP runtime error";
    case AGRL_E_UNSUPPORTED: return "unsupported configuration";
    default: return "unknown status";
  }
}

extern "C" const char* agrl_last_error(void) { return agrl::g_last_error; }

__global__ void agrl_clear_error_kernel(int* err) { *err = 0; }

extern "C" int agrl_get_device_error(void* stream, int32_t* code) {
  if (!code) {
    agrl::set_last_error("agrl_get_device_error: code is NULL");
    return AGRL_E_NULL;
  }
  hipStream_t s = (hipStream_t)stream;
  int rc = agrl::hip_status(hipStreamSynchronize(s));
  if (rc) return rc;
  int* p = agrl::device_error_ptr();
  if (!p) return agrl::hip_status(hipErrorInvalidSymbol);
  int v = 0;
  rc = agrl::hip_status(hipMemcpyAsync(&v, p, sizeof v, hipMemcpyDeviceToHost, s));
  if (rc) return rc;
  rc = agrl::hip_status(hipStreamSynchronize(s));
  if (rc) return rc;
  hipLaunchKernelGGL(agrl_clear_error_kernel, dim3(1), dim3(1), 0, s, p);
  rc = agrl::hip_status(hipGetLastError());
  if (rc) return rc;
  rc = agrl::hip_status(hipStreamSynchronize(s));
  if (rc) return rc;
  *code = v;
  return AGRL_OK;
}
