// smol_scratch.hip -- the fixed device array behind smol_preprocess_batch_noalloc:
// the per-image descriptor table of a ragged batch, which the other entry
// points keep in device memory the library allocates (and grows) per stream.
//
// `scratch` is a file-scope device array: every device the library runs on
// holds its own copy until the process ends. Host code never uses its name
// as an address (in host code it names a host-side stand-in); it asks
// scratch_table() for the device address, which hipGetSymbolAddress looks up
// once per device with that device current.
#include <hip/hip_runtime.h>

#include <mutex>

#include "smol_internal.h"

namespace smol {
namespace {

static __device__ __align__(256) uint8_t scratch[kNoallocTableBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_addr[kMaxDevices];

}  // namespace

int scratch_table(int device, void **table)
{
    if (device < 0 || device >= kMaxDevices)
        return (int)hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_addr[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return (int)e;
        g_scratch_addr[device] = p;
    }
    *table = g_scratch_addr[device];
    return (int)hipSuccess;
}

}  // namespace smol
