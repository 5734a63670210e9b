// Device scratch for the entry point that allocates nothing (tfk_conv2d_bwd_filter_noalloc):
// one file-scope array per GPU, in place of a caller workspace.
//
// The array's name is a host-side stand-in in host code; its device address on the current
// GPU is looked up once per device with hipGetSymbolAddress and kept, and only that address
// is ever handed to kernels.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "kernels.h"

namespace tfk {

namespace {

constexpr size_t kScratchBytes = size_t(128) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::atomic<void *> g_scratch[kMaxDevices];
std::mutex g_scratch_lock;

}  // namespace

size_t noalloc_scratch_bytes() { return kScratchBytes; }

// The scratch array's device address on the current device (looked up on the first call on
// that device), which must be the device of `stream`.  Returns the HIP error of the lookup,
// or hipErrorInvalidDevice when the stream belongs to another device.
hipError_t noalloc_scratch(void **ptr, hipStream_t stream) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    // the work is enqueued on `stream`: the scratch used must be that stream's GPU's copy
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return e;
    if (sdev != dev) return hipErrorInvalidDevice;
    void *p = g_scratch[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> g(g_scratch_lock);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (p == nullptr) {
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (p == nullptr) return hipErrorInvalidSymbol;
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *ptr = p;
    return hipSuccess;
}

}  // namespace tfk
