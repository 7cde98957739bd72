// Internal error reporting shared by the host planner and the HIP launchers.
#pragma once

#include <cstdarg>
#include <cstdio>
#include <string>

#include "libra.h"

namespace libra {

// Thread-local text of the last failure, returned by libra_last_error().
std::string &last_error_text();

// Record a formatted message and return `code` (a negative LIBRA_E* value).
inline int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  last_error_text() = buf;
  return code;
}

}  // namespace libra
