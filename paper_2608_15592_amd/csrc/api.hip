// Library-wide entry points: version, status text and the per-thread error message.
#include <stdarg.h>
#include <stdio.h>

#include <atomic>

#include "estp_common.h"

namespace estp {

static thread_local char g_last_error[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
}

void clear_error() { g_last_error[0] = '\0'; }

int current_device_cu_count() {
  static std::atomic<int> cache[kMaxDevices];  // 0 = not yet asked
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
  if (dev < kMaxDevices) {
    const int n = cache[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) return 0;
  if (dev < kMaxDevices) cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

}  // namespace estp

extern "C" {

int estp_version(void) { return 100; }

const char* estp_status_string(int status) {
  switch (status) {
    case ESTP_OK: return "ESTP_OK";
    case ESTP_ERR_INVALID_ARG: return "ESTP_ERR_INVALID_ARG: invalid argument";
    case ESTP_ERR_UNSUPPORTED: return "ESTP_ERR_UNSUPPORTED: valid but unsupported configuration";
    case ESTP_ERR_WORKSPACE: return "ESTP_ERR_WORKSPACE: workspace too small";
    case ESTP_ERR_HIP: return "ESTP_ERR_HIP: HIP runtime error";
    default: return "unknown estp status";
  }
}

const char* estp_last_error(void) { return estp::g_last_error; }

}  // extern "C"
