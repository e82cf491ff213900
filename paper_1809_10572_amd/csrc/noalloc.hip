// samd_conv2d_noalloc: samd_conv2d with its workspace in a file-scope device array instead
// of a caller buffer, for callers that cannot allocate device memory.
//
// The array is allocated by the HIP runtime when this code object is loaded on a device
// and is held until the process ends; each device holds its own copy.  Host code never
// passes the array's name to a kernel (in host code it is a host-side stand-in, not a
// device address): on the first call on a device its device address is looked up with
// hipGetSymbolAddress, with that device current, and kept per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "hip_util.hpp"

namespace samd {

namespace {

static __device__ __align__(256) unsigned char scratch[SAMD_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of the array (looked up once per device).
int scratch_address(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        set_error(std::string("samd_conv2d_noalloc: hipGetDevice: ") + hipGetErrorString(e));
        return SAMD_EHIP;
    }
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("samd_conv2d_noalloc: device index beyond the library's table");
        return SAMD_EUNSUPPORTED;
    }
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            set_error(std::string("samd_conv2d_noalloc: hipGetSymbolAddress: ") + hipGetErrorString(e));
            return SAMD_EHIP;
        }
        scratch_ptr[dev] = p;
    }
    *out = scratch_ptr[dev];
    return SAMD_OK;
}

}  // namespace

int launch_conv2d_noalloc(const uint32_t *x, const uint32_t *w, const Conv2dGeom &g, int32_t *y, hipStream_t s) {
    if (conv2d_workspace_bytes(g) > (size_t)SAMD_NOALLOC_SCRATCH_BYTES) {
        set_error("samd_conv2d_noalloc: the layer needs a larger workspace than the library's scratch array");
        return SAMD_ENOSPC;
    }
    void *ws = nullptr;
    int st = scratch_address(&ws);
    if (st) return st;
    // the kernel-word preparation also zeroes the multiply kernel's ticket counters, so
    // every call starts from a cleared scratch whatever the previous call left
    st = launch_conv2d_prepare(w, g, ws, s);
    if (st) return st;
    return launch_conv2d_samd(x, g, y, ws, s);
}

}  // namespace samd
