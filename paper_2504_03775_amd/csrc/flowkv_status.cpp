#include "flowkv_status.h"

#include <cstdio>

namespace flowkv {
namespace {
thread_local char g_msg[512] = "";
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_msg, sizeof g_msg, fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_msg[0] = '\0';
  return FLOWKV_OK;
}

}  // namespace flowkv

extern "C" const char* flowkv_last_error(void) { return flowkv::g_msg; }

extern "C" const char* flowkv_strerror(int code) {
  switch (code) {
    case FLOWKV_OK: return "ok";
    case FLOWKV_EINVAL: return "invalid argument";
    case FLOWKV_ENOSPC: return "not enough free blocks";
    case FLOWKV_ERANGE: return "block ID out of range";
    case FLOWKV_EDUP: return "block ID repeated, already free or already in use";
    case FLOWKV_ECAP: return "output capacity too small";
    case FLOWKV_EHIP: return "HIP runtime error";
    case FLOWKV_ENOMEM: return "out of host memory";
    default: return "unknown status code";
  }
}
