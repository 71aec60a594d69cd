// Thread-local error text behind dp_last_error().
#include "common.h"

namespace dpool {

static thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

void clear_error() { g_last_error.clear(); }

}  // namespace dpool

extern "C" const char* dp_last_error(void) { return dpool::g_last_error.c_str(); }

extern "C" const char* dp_version(void) { return "dpool 0.1.0 (gfx950)"; }
