// A host-only HIP runtime with working streams and events, for running the
// library's pipeline (smol_pipeline.cpp) and host code on the CPU: each stream
// is a worker thread that executes its operations in order (copies are
// memcpy, kernels are tasks of a fixed duration, event waits block the
// worker), events complete when their stream reaches them, and host waits
// block on them. Device memory is host memory. Implemented in
// tests/csrc/fake_hip.cpp.
#pragma once

#include <stddef.h>

typedef enum hipError_t { hipSuccess = 0, hipErrorInvalidValue = 1, hipErrorNotReady = 600,
                          hipErrorNoDevice = 100, hipErrorInvalidDevice = 101 } hipError_t;
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
hipError_t hipSetDevice(int device);
hipError_t hipDeviceGetAttribute(int *value, hipDeviceAttribute_t attr, int device);
hipError_t hipMemcpyAsync(void *dst, const void *src, size_t bytes, hipMemcpyKind kind,
                          hipStream_t stream);
hipError_t hipEventSynchronize(hipEvent_t e);
hipError_t hipEventQuery(hipEvent_t e);
hipError_t hipEventRecord(hipEvent_t e, hipStream_t s);
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned flags);
hipError_t hipStreamSynchronize(hipStream_t s);
const char *hipGetErrorString(hipError_t e);
hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned flags);
hipError_t hipEventDestroy(hipEvent_t e);
hipError_t hipStreamCreateWithFlags(hipStream_t *s, unsigned flags);
hipError_t hipStreamDestroy(hipStream_t s);
hipError_t hipMalloc(void **p, size_t bytes);
hipError_t hipFree(void *p);
hipError_t hipHostMalloc(void **p, size_t bytes, unsigned flags);
hipError_t hipHostFree(void *p);
hipError_t hipHostGetDevicePointer(void **dev, void *host, unsigned flags);

// Test hooks (not HIP): enqueue a task on a stream (the stand-in for a kernel)
// and read how many operations are queued and not yet finished, over all
// streams.
void fake_hip_enqueue_task(hipStream_t s, unsigned microseconds);
long fake_hip_pending(void);
