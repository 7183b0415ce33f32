// Error reporting and version query of the C ABI.
#include <stdarg.h>
#include <stdio.h>

#include "dvs_common.h"

namespace dvs {

static thread_local char g_msg[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
}

void clear_error() { g_msg[0] = 0; }

int launch_status(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("%s: launch failed: %s", what, hipGetErrorString(e));
    return DVS_EHIP;
  }
  return DVS_OK;
}

}  // namespace dvs

extern "C" int dvs_version(void) { return 100; }

extern "C" const char* dvs_last_error(void) { return dvs::g_msg; }
