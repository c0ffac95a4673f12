// Host-side helpers shared by the C ABI sources: the thread-local error
// message and the status helpers.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/compresskv.h"

namespace ckv_api {

inline thread_local std::string g_last_error;

inline int fail(int status, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

inline int ok() {
  g_last_error.clear();
  return CKV_OK;
}

inline bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace ckv_api
