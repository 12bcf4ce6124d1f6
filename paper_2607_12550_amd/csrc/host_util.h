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

// Makes a context's device current for the guard's lifetime and restores the device the
// caller had current when the guard leaves scope (every entry point that queues device
// work holds one, so a call never changes the caller's current device).
struct DeviceGuard {
  int prev = -1;
  hipError_t enter(int dev) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur == dev) return hipSuccess;
    prev = cur;
    return hipSetDevice(dev);
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
  DeviceGuard() = default;
  DeviceGuard(const DeviceGuard &) = delete;
  DeviceGuard &operator=(const DeviceGuard &) = delete;
};
