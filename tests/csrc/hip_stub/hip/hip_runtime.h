// A host-only stand-in for <hip/hip_runtime.h>: just the types, constants and
// functions the library's host sources (validation, geometry, planning, JPEG
// entropy decoding) use, so that they build with g++ and the sanitizers. The
// functions (host_stub.cpp) report that no device exists, so any call that
// passes validation ends with SMOL_ERR_HIP before it would touch a device.
#pragma once

#include <stddef.h>

typedef enum hipError_t { hipSuccess = 0, hipErrorInvalidValue = 1, hipErrorNoDevice = 100,
                          hipErrorInvalidDevice = 101 } hipError_t;
typedef struct ihipStream_t *hipStream_t;
typedef struct ihipEvent_t *hipEvent_t;
typedef enum hipMemcpyKind { hipMemcpyHostToHost = 0, hipMemcpyHostToDevice = 1,
                             hipMemcpyDeviceToHost = 2, hipMemcpyDeviceToDevice = 3 }
    hipMemcpyKind;
typedef enum hipDeviceAttribute_t { hipDeviceAttributeMultiprocessorCount = 1,
                                    hipDeviceAttributeMaxSharedMemoryPerMultiprocessor = 2,
                                    hipDeviceAttributeMaxSharedMemoryPerBlock = 3 }
    hipDeviceAttribute_t;
#define hipEventDisableTiming 0x2
#define hipStreamNonBlocking 0x1
#define hipHostMallocDefault 0x0

hipError_t hipGetDevice(int *device);
hipError_t hipDeviceGetAttribute(int *value, hipDeviceAttribute_t attr, int device);
hipError_t hipMemcpyAsync(void *dst, const void *src, size_t bytes, hipMemcpyKind kind,
                          hipStream_t stream);
hipError_t hipEventSynchronize(hipEvent_t e);
hipError_t hipEventRecord(hipEvent_t e, hipStream_t s);
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned flags);
const char *hipGetErrorString(hipError_t e);
hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned flags);
hipError_t hipStreamCreateWithFlags(hipStream_t *s, unsigned flags);
hipError_t hipMalloc(void **p, size_t bytes);
hipError_t hipFree(void *p);
hipError_t hipHostMalloc(void **p, size_t bytes, unsigned flags);
hipError_t hipHostFree(void *p);
hipError_t hipHostGetDevicePointer(void **dev, void *host, unsigned flags);
