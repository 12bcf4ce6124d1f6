// Host-side error reporting shared by the C-ABI translation units.
#pragma once
#include <hip/hip_runtime_api.h>

int jolt_fail(int code, const char *fmt, ...);
int jolt_hip_fail(hipError_t e, const char *what, const char *file, int line);

#define HIP_OK(expr)                                                        \
  do {                                                                      \
    hipError_t _e = (expr);                                                 \
    if (_e != hipSuccess) return jolt_hip_fail(_e, #expr, __FILE__, __LINE__); \
  } while (0)
