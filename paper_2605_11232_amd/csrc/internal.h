// Internal declarations shared by the host-side translation units of libpa.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <string>

#include "pa.h"

namespace pa {

// Record a formatted message as the calling thread's last error and return code.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace pa
