// Thread-local error messages and the library version (host only).
#include <cstdio>
#include <string>

#include "dcp_internal.h"

namespace dcp {

namespace {
thread_local std::string g_last_error;
}

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

}  // namespace dcp

extern "C" const char* dcp_last_error(void) { return dcp::g_last_error.c_str(); }

extern "C" const char* dcp_version(void) { return "dcp-mi355x 0.2 (gfx950)"; }
