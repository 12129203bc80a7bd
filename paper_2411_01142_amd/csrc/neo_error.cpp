// Thread-local error message of the C ABI (host code, shared by the device
// and host halves of the library).
#include "neo_error.h"

#include <stdarg.h>
#include <stdio.h>

#include <string>

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace neo {

neo_status set_error(neo_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

neo_status clear_error() {
  g_last_error.clear();
  return NEO_OK;
}

}  // namespace neo

extern "C" const char* neo_last_error(void) { return g_last_error.c_str(); }
