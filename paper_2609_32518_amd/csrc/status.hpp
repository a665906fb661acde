// Status codes and the thread-local message of the last failed call (unstep_last_error),
// shared by the host sources of the C ABI.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "unstep.h"

namespace unstep {

inline thread_local std::string g_err;

inline int ok() {
  g_err.clear();
  return UNSTEP_OK;
}

inline int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

inline int fail_msg(int code, const char* where, const std::string& why) {
  return fail(code, "%s: %s", where, why.c_str());
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace unstep
