// Static device scratch for callers that cannot allocate (code under HIP
// graph capture, tight serving loops): recblr_bdlru_scan_backward_noalloc
// runs the scan backward's kernels on this buffer instead of a caller's
// workspace.  It holds the look-back state words and ticket counter and the
// per-tile dLambda partials of one call; the kernels clear what must start
// at zero (the look-back reset kernel) and overwrite the rest, so nothing
// carries over from the previous call.  Every GPU the library runs on holds
// its own copy until the process ends; calls that overlap on one GPU share it
// and race.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "launch.hpp"

static __device__ __align__(256) char scratch[recblr::kStaticScratchBytes];

namespace recblr {

namespace {
constexpr int kMaxDevices = 256;
// Device address of `scratch` per device.  The array's name is only a
// host-side stand-in for it, so host code uses these addresses, never the name.
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_lookup;
}  // namespace

hipError_t static_scratch(void** ptr, size_t* bytes) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void* p = g_scratch[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lock(g_lookup);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (p == nullptr) {
            // Once per device, with that device current.
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (p == nullptr) return hipErrorInvalidSymbol;
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *ptr = p;
    *bytes = kStaticScratchBytes;
    return hipSuccess;
}

}  // namespace recblr
