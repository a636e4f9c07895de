// Thread-local last-error message behind pa_last_error().
#include <cstdio>

#include "internal.h"

namespace {
thread_local std::string g_last_error;
}

namespace pa {

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

void clear_error() { g_last_error.clear(); }

}  // namespace pa

extern "C" const char* pa_last_error(void) { return g_last_error.c_str(); }
extern "C" int32_t pa_abi_version(void) { return 2; }
