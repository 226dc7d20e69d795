// Static scratch of the allocation-free decode entry point
// (bdlora_forward_layer_static): a file-scope device array that every GPU
// the library runs on holds from module load to process end, so a forward
// that uses it makes no allocation at all.
//
// In host code `scratch` is a host-side stand-in for the array, not a device
// address: the address of each device's copy comes from hipGetSymbolAddress,
// taken once per device at set-up (pool creation, with that device current)
// and kept here; host code only ever hands that address to kernels.
#include <mutex>

#include "bdl_launch.h"

namespace bdl {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
std::mutex g_mu;
void* g_addr[kMaxDevices] = {};
}  // namespace

hipError_t static_scratch_init(int device) {
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_addr[device]) return hipSuccess;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_addr[device] = p;
    return hipSuccess;
}

void* static_scratch(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_mu);
    return g_addr[device];
}

}  // namespace bdl
