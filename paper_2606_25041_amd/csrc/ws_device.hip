// Host-side device queries of the library: the compute-unit count the step
// planner sizes its launches for.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "ws_kernels.h"

namespace ws {

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
