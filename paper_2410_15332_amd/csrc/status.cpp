// Status strings and the thread-local detail of the last failure.
#include "status.h"

#include <cstdio>

namespace {
thread_local std::string g_last_error;
}

namespace epic {

epic_status fail(epic_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

void clear_error() { g_last_error.clear(); }

}  // namespace epic

extern "C" const char* epic_status_string(int status) {
  switch (status) {
    case EPIC_OK: return "ok";
    case EPIC_ERR_INVALID_ARG: return "invalid argument";
    case EPIC_ERR_UNSUPPORTED: return "unsupported shape";
    case EPIC_ERR_NO_PRIVATE_BLOCKS: return "not enough free blocks for private copies";
    case EPIC_ERR_WORKSPACE: return "workspace too small";
    case EPIC_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

extern "C" const char* epic_last_error(void) { return g_last_error.c_str(); }

extern "C" const char* epic_version(void) { return "epic_link 0.1 gfx950"; }
