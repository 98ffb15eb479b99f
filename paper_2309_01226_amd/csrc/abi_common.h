// Error plumbing shared by the C-ABI translation units: a thread-local last
// error message and macros that turn HIP failures into sat_status codes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include "../../include/saturn.h"

void sat_set_error(const char* fmt, ...);

#define SAT_CHECK_ARG(cond, ...)        \
  do {                                  \
    if (!(cond)) {                      \
      sat_set_error(__VA_ARGS__);       \
      return SAT_EINVAL;                \
    }                                   \
  } while (0)

#define SAT_HIP(call)                                                              \
  do {                                                                             \
    hipError_t e_ = (call);                                                        \
    if (e_ != hipSuccess) {                                                        \
      sat_set_error("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, \
                    __LINE__);                                                     \
      return SAT_EHIP;                                                             \
    }                                                                              \
  } while (0)
