// Per-thread error state behind diffopt_last_error().
#include <cstdarg>
#include <cstdio>

#include "common.hpp"

namespace diffopt {

namespace {
thread_local char g_msg[512] = "";
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_msg[0] = '\0'; }

int launch_status(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    return fail(DIFFOPT_EHIP, "%s: kernel launch failed: %s", what, hipGetErrorString(e));
  }
  return DIFFOPT_OK;
}

}  // namespace diffopt

extern "C" const char* diffopt_last_error(void) { return diffopt::g_msg; }
