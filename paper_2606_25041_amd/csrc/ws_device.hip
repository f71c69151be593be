// Host-side device queries of the library: the compute-unit count the step
// planner sizes its launches for, and the per-device scratch array behind
// the allocation-free step entry point.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "ws_kernels.h"

namespace ws {

// Scratch for the allocation-free step entry point: the split-KV partials of
// one call live here instead of in a caller workspace.  One copy per device
// (each device's code object holds its own), kept until the process ends.
__device__ __align__(256) char scratch[NOALLOC_SCRATCH_BYTES];

int scratch_address(void **ptr) {
    constexpr int MAX_DEV = 64;
    static std::atomic<void *> addr[MAX_DEV];   // nullptr until looked up
    int dev = -1;
    if (hipError_t e = hipGetDevice(&dev)) return (int)e;
    if (dev < 0 || dev >= MAX_DEV) return (int)hipErrorInvalidDevice;
    void *p = addr[dev].load(std::memory_order_acquire);
    if (!p) {
        // host code must never pass `scratch` itself to a kernel: in host code
        // it names a host-side stand-in; this is its address on the device
        if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) return (int)e;
        if (!p) return (int)hipErrorInvalidSymbol;
        addr[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return 0;
}

int current_device_cus(int *cus) {
    constexpr int MAX_DEV = 64;
    static std::atomic<int> cached[MAX_DEV];   // 0 until queried
    int dev = -1;
    if (hipError_t e = hipGetDevice(&dev)) return (int)e;
    if (dev >= 0 && dev < MAX_DEV) {
        const int c = cached[dev].load(std::memory_order_relaxed);
        if (c > 0) {
            *cus = c;
            return 0;
        }
    }
    int n = 0;
    if (hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev)) return (int)e;
    if (n <= 0) return (int)hipErrorInvalidDevice;
    if (dev >= 0 && dev < MAX_DEV) cached[dev].store(n, std::memory_order_relaxed);
    *cus = n;
    return 0;
}

}  // namespace ws
