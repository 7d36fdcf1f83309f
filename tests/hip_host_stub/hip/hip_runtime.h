// Host-only stand-in for <hip/hip_runtime.h> (test infrastructure): lets the
// library's host builder (api.cpp) compile with a plain C++ compiler under
// the sanitizers.  There is no device: every device call fails, so a load
// runs the host expansion and stops at its first device call.
#pragma once
#include <cstddef>
#include <cstdint>

typedef int hipError_t;
typedef void *hipStream_t;
enum { hipSuccess = 0, hipErrorNoDevice = 100 };
enum hipMemcpyKind { hipMemcpyHostToDevice = 1, hipMemcpyDeviceToHost = 2 };
enum hipDeviceAttribute_t { hipDeviceAttributeMultiprocessorCount = 0 };
struct uint4 { unsigned x, y, z, w; };

inline hipError_t hipGetDevice(int *) { return hipErrorNoDevice; }
inline hipError_t hipDeviceGetAttribute(int *, hipDeviceAttribute_t, int) { return hipErrorNoDevice; }
inline hipError_t hipMalloc(void **p, size_t) { *p = nullptr; return hipErrorNoDevice; }
inline hipError_t hipFree(void *) { return hipSuccess; }
inline hipError_t hipMemcpy(void *, const void *, size_t, hipMemcpyKind) { return hipErrorNoDevice; }
inline const char *hipGetErrorString(hipError_t) { return "no device (host-only build)"; }
