// Library-wide entry points: version, status text and the per-thread error message.
#include <stdarg.h>
#include <stdio.h>

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
