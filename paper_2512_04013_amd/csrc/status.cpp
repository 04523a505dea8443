#include "status.h"

#include <cstdarg>
#include <cstdio>

namespace {
thread_local char g_last_error[512] = "";
}

namespace aug {

aug_status fail(aug_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

}  // namespace aug

extern "C" const char* aug_status_string(aug_status s) {
  switch (s) {
    case AUG_OK: return "AUG_OK";
    case AUG_ERR_INVALID: return "AUG_ERR_INVALID";
    case AUG_ERR_UNSUPPORTED: return "AUG_ERR_UNSUPPORTED";
    case AUG_ERR_NO_SPACE: return "AUG_ERR_NO_SPACE";
    case AUG_ERR_HIP: return "AUG_ERR_HIP";
  }
  return "AUG_UNKNOWN_STATUS";
}

extern "C" const char* aug_last_error(void) { return g_last_error; }

extern "C" int32_t aug_abi_version(void) { return (3 << 16) | 1; }
