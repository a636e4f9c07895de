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

// Tokens per block of a pool (the pool must not be NULL).
int32_t pool_block_size(const pa_pool* pool);

}  // namespace pa
