// Status strings, per-thread error detail and cached device properties.
#include <stdarg.h>
#include <stdio.h>

#include <mutex>

#include "common.h"

namespace moe {

static thread_local char g_last_error[512] = "";

moe_status fail(moe_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

moe_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(MOE_ERROR_HIP, "%s: %s", what, hipGetErrorString(e));
  return MOE_SUCCESS;
}

int device_cu_count() {
  static std::mutex mu;
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

}  // namespace moe

extern "C" const char* moe_status_string(moe_status s) {
  switch (s) {
    case MOE_SUCCESS: return "success";
    case MOE_ERROR_INVALID_VALUE: return "invalid value";
    case MOE_ERROR_NOT_SUPPORTED: return "not supported";
    case MOE_ERROR_WORKSPACE: return "workspace too small";
    case MOE_ERROR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

extern "C" const char* moe_last_error(void) { return moe::g_last_error; }
