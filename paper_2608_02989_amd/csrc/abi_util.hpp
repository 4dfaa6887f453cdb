// Error reporting and argument helpers shared by the C ABI translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "acceptmoe.h"

namespace amoe {
namespace abi {

// thread-local text returned by acceptmoe_last_error (one object for the whole library)
inline thread_local char g_err[512] = "";

inline int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

inline void clear_err() { g_err[0] = '\0'; }

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

inline int hip_fail(hipError_t e, const char* what) {
  return fail(ACCEPTMOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace abi
}  // namespace amoe
