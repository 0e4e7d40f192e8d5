// Error state and version of the C ABI.
#include <stdarg.h>
#include <stdio.h>

#include "common.h"

namespace avits {

static thread_local char g_last_error[512] = "";

int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

// Status of the launches just enqueued by this thread.
int launch_status(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(AVITS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return AVITS_OK;
}

}  // namespace avits

extern "C" const char* avits_version(void) { return "0.1.0"; }

extern "C" const char* avits_last_error(void) { return avits::g_last_error; }
