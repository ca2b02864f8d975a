// C-ABI plumbing: thread-local error reporting shared by every entry point.
#include <cstdio>
#include <string>

#include "tq_internal.hpp"

namespace tq {

static thread_local std::string g_error;

tq_status fail(tq_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return st;
}

void clear_error() { g_error.clear(); }

tq_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TQ_ERR_DEVICE, "%s: launch failed: %s", what, hipGetErrorString(e));
  return TQ_OK;
}

}  // namespace tq

extern "C" const char* tq_last_error(void) { return tq::g_error.c_str(); }
