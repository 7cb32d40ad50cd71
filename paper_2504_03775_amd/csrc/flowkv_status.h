// Status plumbing shared by the host-side translation units of the library:
// every ABI entry point returns a code and leaves a per-thread message.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <new>

#include "flowkv.h"

namespace flowkv {

// Record a formatted message for flowkv_last_error() and return `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clear the calling thread's message and return FLOWKV_OK.
int ok();

// Run an entry point's body so that no exception crosses the C ABI: the
// standard containers of the host code can only raise std::bad_alloc, which
// becomes FLOWKV_ENOMEM.
template <class F>
int guarded(F&& body) {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(FLOWKV_ENOMEM, "out of host memory");
  } catch (...) {
    return fail(FLOWKV_EINVAL, "unexpected host exception");
  }
}

}  // namespace flowkv
