// Library-wide pieces of the C ABI: error reporting and the version query.
#include <stdarg.h>
#include <stdio.h>

#include "common.hpp"

static thread_local char g_last_error[512] = "";

local_status_t local_fail(local_status_t code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return code;
}

local_status_t local_check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return local_fail(LOCAL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return LOCAL_OK;
}

extern "C" const char* local_last_error(void) { return g_last_error; }

extern "C" int32_t local_version(void) { return 200; }  // 0.2.0
