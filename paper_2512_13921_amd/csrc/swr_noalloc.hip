// swr_noalloc.hip -- the exact recurrence's forward on a workspace that the
// library owns: a static device array, for callers that cannot allocate
// device memory.  The kernels and the validation are those of
// swr_exact_forward; only where the workspace lives differs.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "../../include/swr.h"
#include "swr_internal.h"

namespace {

// The workspace, one copy per GPU.  In host code `scratch` names a host-side
// stand-in, not device memory: host code only ever uses the device address
// that hipGetSymbolAddress returns for the device in question.
static __device__ __align__(256) unsigned char scratch[SWR_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_scratch[kMaxDevices];   // per device ordinal: the device address of `scratch`, once known

// The device address of `scratch` on the device that runs `stream`, looked up
// (with that device current) on the first call for the device.
void* scratch_address(void* stream) {
    int dev = -1;
    if (stream) {
        hipDevice_t d;
        if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &d) != hipSuccess) return nullptr;
        dev = static_cast<int>(d);
    } else if (hipGetDevice(&dev) != hipSuccess) {
        return nullptr;
    }
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> hold(g_lock);
    if (!g_scratch[dev]) {
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return nullptr;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return nullptr;
        void* ptr = nullptr;
        const hipError_t err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != dev && hipSetDevice(cur) != hipSuccess) return nullptr;
        if (err != hipSuccess || !ptr) return nullptr;
        g_scratch[dev] = ptr;
    }
    return g_scratch[dev];
}

}  // namespace

extern "C" int swr_exact_forward_noalloc(const swr_problem_t* problem, const void* x, const void* a,
                                         const void* b, const void* c, const float* h0, void* y,
                                         float* carriers, float* h_last, void* stream) {
    return swr::exact_forward_impl(problem, x, a, b, c, h0, y, carriers, h_last, nullptr, scratch_address,
                                   SWR_NOALLOC_SCRATCH_BYTES, stream);
}
