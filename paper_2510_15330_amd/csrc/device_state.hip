// Per-device memory the library holds without allocating: the sticky error
// word every kernel reports into, and the fixed scratch array of the
// no-allocation decode entry point.  Both are file-scope device variables;
// each GPU the library runs on holds its own copy (loaded with the code
// object) until the process ends.  Host code never passes their names to a
// kernel or a copy: it asks the runtime for the current device's address
// once per device (hipGetSymbolAddress) and uses that.
#include <mutex>

#include "../../include/bellman.h"
#include "internal.h"

static __device__ __align__(256) int32_t err_word[64];            // [0]: error bits; rest padding
static __device__ __align__(256) char scratch[bellman::kScratchBytes];   // no-allocation decode workspace

namespace bellman {
namespace {

struct DeviceAddrs {
    bool ready = false;   // guarded by g_addrs_mutex
    int32_t* err = nullptr;
    char* scratch = nullptr;
};
DeviceAddrs g_addrs[kMaxDevices];
std::mutex g_addrs_mutex;

// Both addresses on device `dev`, which must be current; resolved on the
// first call for the device.
int resolve(int dev, DeviceAddrs* out) {
    if (dev < 0 || dev >= kMaxDevices) return set_error(BELLMAN_ERR_UNSUPPORTED, "device index %d", dev);
    std::lock_guard<std::mutex> lock(g_addrs_mutex);
    DeviceAddrs& d = g_addrs[dev];
    if (d.ready) {
        *out = d;
        return BELLMAN_OK;
    }
    void* pe = nullptr;
    void* ps = nullptr;
    hipError_t e = hipGetSymbolAddress(&pe, HIP_SYMBOL(err_word));
    if (e != hipSuccess || !pe) return set_error(BELLMAN_ERR_HIP, "hipGetSymbolAddress(error word): %s", hipGetErrorString(e));
    e = hipGetSymbolAddress(&ps, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ps) return set_error(BELLMAN_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    d.err = (int32_t*)pe;
    d.scratch = (char*)ps;
    d.ready = true;
    *out = d;
    return BELLMAN_OK;
}

}  // namespace

int device_error_word(int dev, int32_t** p) {
    DeviceAddrs d;
    const int rc = resolve(dev, &d);
    if (rc == BELLMAN_OK) *p = d.err;
    return rc;
}

int device_scratch(int dev, char** p) {
    DeviceAddrs d;
    const int rc = resolve(dev, &d);
    if (rc == BELLMAN_OK) *p = d.scratch;
    return rc;
}

}  // namespace bellman
