// Test double of the HIP runtime declarations that the library's C-ABI layer
// uses, for a host-only build of that layer under AddressSanitizer and
// UndefinedBehaviorSanitizer (tests/test_host_sanitize.py). It reports one
// gfx950 device; no GPU code is built or run. The kernel launchers are
// replaced by recording stubs (launch_stubs.cpp).
#pragma once

#include <cstring>

typedef int hipError_t;
constexpr hipError_t hipSuccess = 0;
typedef struct ihipStream_t* hipStream_t;

struct hipDeviceProp_t {
  char gcnArchName[256];
};

inline hipError_t hipGetDevice(int* dev) {
  *dev = 0;
  return hipSuccess;
}

inline hipError_t hipGetDeviceProperties(hipDeviceProp_t* prop, int) {
  std::memset(prop, 0, sizeof(*prop));
  std::strcpy(prop->gcnArchName, "gfx950:sramecc+:xnack-");
  return hipSuccess;
}

inline const char* hipGetErrorString(hipError_t) { return "hip test double"; }
