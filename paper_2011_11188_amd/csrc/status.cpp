// Error state of the C ABI: a thread-local message of the last failure.
#include <string>

#include "internal.h"

namespace mdnn {

static thread_local std::string g_last_error;

mdnn_status_t fail(mdnn_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

void clear_error() { g_last_error.clear(); }

mdnn_status_t check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(MDNN_ERR_LAUNCH, "%s: %s", what, hipGetErrorString(e));
  return MDNN_SUCCESS;
}

}  // namespace mdnn

extern "C" const char* mdnn_last_error(void) { return mdnn::g_last_error.c_str(); }
extern "C" const char* mdnn_version(void) { return "mdnn 0.1 (gfx950)"; }
