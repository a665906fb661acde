// Status codes and the thread-local message of the last failed call (unstep_last_error),
// shared by the host sources of the C ABI.  No C++ exception crosses the ABI: every entry
// point runs its body inside guarded(), which turns an escaping exception (e.g. out of host
// memory) into UNSTEP_E_HOST.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <exception>
#include <new>
#include <string>

#include "unstep.h"

namespace unstep {

// The message lives in a fixed buffer, so recording an error never allocates.
constexpr size_t kErrBytes = 512;
inline thread_local char g_err[kErrBytes] = "";

inline int ok() {
  g_err[0] = '\0';
  return UNSTEP_OK;
}

inline int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, kErrBytes, fmt, ap);
  va_end(ap);
  return code;
}

inline int fail_msg(int code, const char* where, const std::string& why) {
  return fail(code, "%s: %s", where, why.c_str());
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Run the body of an entry point; an exception that escapes it becomes an error status.
template <class F>
int guarded(const char* where, F&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(UNSTEP_E_HOST, "%s: out of host memory", where);
  } catch (const std::exception& e) {
    return fail(UNSTEP_E_HOST, "%s: %s", where, e.what());
  } catch (...) {
    return fail(UNSTEP_E_HOST, "%s: unexpected host failure", where);
  }
}

}  // namespace unstep
