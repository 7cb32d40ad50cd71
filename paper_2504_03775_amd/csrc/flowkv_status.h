// Status plumbing shared by the host-side translation units of the library:
// every ABI entry point returns a code and leaves a per-thread message.
#pragma once

#include <cstdarg>
#include <cstdint>

#include "flowkv.h"

namespace flowkv {

// Record a formatted message for flowkv_last_error() and return `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clear the calling thread's message and return FLOWKV_OK.
int ok();

}  // namespace flowkv
