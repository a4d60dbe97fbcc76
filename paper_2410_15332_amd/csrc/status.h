// Internal helpers shared by the host sources of libepic_link: error reporting.
#pragma once

#include <cstdarg>
#include <string>

#include "epic_link.h"

namespace epic {

// Records a formatted detail message for epic_last_error() and returns `st`.
epic_status fail(epic_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace epic

#define EPIC_CHECK_ARG(cond, ...)                                   \
  do {                                                              \
    if (!(cond)) return ::epic::fail(EPIC_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)
