// Host-only stand-in for <hip/hip_runtime.h>, used to build the host planner and C ABI with
// g++ under AddressSanitizer / UndefinedBehaviorSanitizer on a machine without a GPU.  It
// declares only what psattn_host.cpp, psattn_noalloc.hip and psattn_launch.h use; every device
// call fails with hipErrorNotSupported (the host tests never reach one), and a __device__ array
// becomes a plain host array.
#pragma once
#include <cstddef>

typedef int hipError_t;
enum { hipSuccess = 0, hipErrorInvalidValue = 1, hipErrorNotSupported = 801 };
typedef struct ihipStream_t* hipStream_t;
typedef struct ihipEvent_t* hipEvent_t;
typedef enum { hipMemcpyHostToDevice = 1 } hipMemcpyKind;

#define __device__
#define __align__(n) __attribute__((aligned(n)))
#define HIP_SYMBOL(x) (&(x))

inline const char* hipGetErrorString(hipError_t) { return "HIP unavailable in the sanitizer build"; }
inline hipError_t hipMemcpyAsync(void*, const void*, size_t, hipMemcpyKind, hipStream_t) { return hipErrorNotSupported; }
inline hipError_t hipStreamSynchronize(hipStream_t) { return hipErrorNotSupported; }
inline hipError_t hipEventCreate(hipEvent_t*) { return hipErrorNotSupported; }
inline hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipErrorNotSupported; }
inline hipError_t hipEventSynchronize(hipEvent_t) { return hipErrorNotSupported; }
inline hipError_t hipEventElapsedTime(float*, hipEvent_t, hipEvent_t) { return hipErrorNotSupported; }
inline hipError_t hipGetDevice(int*) { return hipErrorNotSupported; }
inline hipError_t hipGetSymbolAddress(void**, const void*) { return hipErrorNotSupported; }
