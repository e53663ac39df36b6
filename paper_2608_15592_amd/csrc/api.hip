// Library-wide entry points: version, status text and the per-thread error message.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

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

bool debug_checks_enabled() {
  static const bool on = [] {
    const char* v = getenv("ESTP_DEBUG_CHECKS");
    return v != nullptr && v[0] == '1' && v[1] == '\0';
  }();
  return on;
}

int debug_check_cu(const char* fn, const int32_t* cu_dev, int32_t B, int64_t n_tok, int32_t max_seqlen,
                   hipStream_t s, std::vector<int>* cu_out) {
  std::vector<int> cu(size_t(B) + 1);
  hipError_t e = hipMemcpyAsync(cu.data(), cu_dev, cu.size() * sizeof(int), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    set_error("%s: debug check: copying cu_seqlens back: %s", fn, hipGetErrorString(e));
    return ESTP_ERR_HIP;
  }
  ESTP_REQUIRE(cu[0] == 0, ESTP_ERR_INVALID_ARG, "%s: debug check: cu_seqlens[0] = %d, must be 0", fn, cu[0]);
  for (int32_t b = 0; b < B; ++b) {
    const int64_t N = int64_t(cu[b + 1]) - cu[b];
    ESTP_REQUIRE(N >= 1 && N <= max_seqlen, ESTP_ERR_INVALID_ARG,
                 "%s: debug check: prompt %d has %lld tokens, must be in [1, max_seqlen = %d]", fn, b, (long long)N,
                 max_seqlen);
  }
  ESTP_REQUIRE(n_tok < 0 || cu[B] == n_tok, ESTP_ERR_INVALID_ARG, "%s: debug check: cu_seqlens[B] = %d, n_tok = %lld",
               fn, cu[B], (long long)n_tok);
  if (cu_out) *cu_out = std::move(cu);
  return ESTP_OK;
}

int debug_check_list(const char* fn, const int2* list_dev, const std::vector<int2>& expect, hipStream_t s) {
  std::vector<int2> got(expect.size());
  hipError_t e = hipMemcpyAsync(got.data(), list_dev, got.size() * sizeof(int2), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    set_error("%s: debug check: copying the work list back: %s", fn, hipGetErrorString(e));
    return ESTP_ERR_HIP;
  }
  for (size_t i = 0; i < got.size(); ++i) {
    ESTP_REQUIRE(got[i].x == expect[i].x && got[i].y == expect[i].y, ESTP_ERR_HIP,
                 "%s: debug check: work list entry %zu is (%d, %d), its definition gives (%d, %d)", fn, i, got[i].x,
                 got[i].y, expect[i].x, expect[i].y);
  }
  return ESTP_OK;
}

}  // namespace estp

extern "C" {

int estp_debug_checks(void) { return estp::debug_checks_enabled() ? 1 : 0; }

int estp_version(void) { return ESTP_VERSION; }

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
