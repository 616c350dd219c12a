// kf_last_error() and the helper every entry point uses to set it.
#include "error.h"

#include <cstdarg>
#include <cstdio>
#include <string>

static thread_local std::string g_err;

namespace kf {
kf_status fail(kf_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}
void clear_error() { g_err.clear(); }
}  // namespace kf

extern "C" const char* kf_last_error(void) { return g_err.c_str(); }
