// Host-only stand-ins for the HIP runtime and for the library's kernel files
// (launchers, occupancy queries, the fixed descriptor array), so that the
// host sources build with g++ and the sanitizers. Every runtime call reports
// that there is no device.
#include <hip/hip_runtime.h>

#include "smol_internal.h"

hipError_t hipGetDevice(int *) { return hipErrorNoDevice; }
hipError_t hipDeviceGetAttribute(int *, hipDeviceAttribute_t, int) { return hipErrorNoDevice; }
hipError_t hipMemcpyAsync(void *, const void *, size_t, hipMemcpyKind, hipStream_t)
{
    return hipErrorNoDevice;
}
hipError_t hipEventSynchronize(hipEvent_t) { return hipErrorNoDevice; }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipErrorNoDevice; }
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned) { return hipErrorNoDevice; }
const char *hipGetErrorString(hipError_t) { return "no device (host-only build)"; }
hipError_t hipEventCreateWithFlags(hipEvent_t *, unsigned) { return hipErrorNoDevice; }
hipError_t hipStreamCreateWithFlags(hipStream_t *, unsigned) { return hipErrorNoDevice; }
hipError_t hipMalloc(void **, size_t) { return hipErrorNoDevice; }
hipError_t hipFree(void *) { return hipSuccess; }
hipError_t hipHostMalloc(void **, size_t, unsigned) { return hipErrorNoDevice; }
hipError_t hipHostFree(void *) { return hipSuccess; }
hipError_t hipHostGetDevicePointer(void **, void *, unsigned) { return hipErrorNoDevice; }

namespace smol {
int launch_jpeg_idct(const JpegArgs &, int, void *) { return hipErrorNoDevice; }
int scratch_table(int, void **) { return hipErrorNoDevice; }
int launch_table_copy(const void *, void *, size_t, void *) { return hipErrorNoDevice; }
int launch_rgb_direct(const BatchArgs &, int, void *, void *) { return hipErrorNoDevice; }
int launch_rgb_lds(const BatchArgs &, int, size_t, void *, void *) { return hipErrorNoDevice; }
int launch_rgb_gather(const BatchArgs &, int, size_t, void *, void *) { return hipErrorNoDevice; }
int launch_rgb_rows(const BatchArgs &, int, size_t, void *, void *) { return hipErrorNoDevice; }
int occupancy_rgb_rows(const BatchArgs &, int, size_t, int *) { return hipErrorNoDevice; }
int occupancy_rgb_gather(int, size_t, int *) { return hipErrorNoDevice; }
int occupancy_rgb_lds(int, size_t, int *) { return hipErrorNoDevice; }
int launch_yuv_direct(const BatchArgs &, int, void *, void *) { return hipErrorNoDevice; }
int launch_yuv_rows(const BatchArgs &, int, size_t, void *, void *) { return hipErrorNoDevice; }
int occupancy_yuv_rows(const BatchArgs &, int, size_t, int *) { return hipErrorNoDevice; }
}  // namespace smol
