// abi.cpp -- status reporting and version of the C ABI (no device code).
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <string>

#include "common.h"

namespace fast {

static thread_local std::string g_last_error;

fast_status_t fail(fast_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

fast_status_t ok() {
  g_last_error.clear();
  return FAST_OK;
}

fast_status_t check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

}  // namespace fast

extern "C" const char* fast_last_error(void) { return fast::g_last_error.c_str(); }

extern "C" const char* fast_version(void) { return "fast-mi355x 0.1 gfx950"; }
