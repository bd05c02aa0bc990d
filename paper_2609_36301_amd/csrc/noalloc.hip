// The low-rank router without a workspace argument, for callers that cannot allocate (code
// under HIP graph capture, serving loops, harnesses that forbid hipMalloc).
//
// The scratch the routing kernels need lives in `scratch`, a static device array of
// MORE_NOALLOC_SCRATCH_BYTES bytes.  It is the only object of this translation unit's code
// object, so it is placed on a device when this entry point first asks for its address there,
// and that device holds it until the process ends.  In host code the name `scratch` is only a
// host-side stand-in: its device address is looked up once per device with
// hipGetSymbolAddress, and only that address is ever passed on.
//
// Every call on one device shares that device's array.  The routing kernels initialise every
// part of the scratch they read (counters and histograms are cleared by the kernels
// themselves, never by a memset), so consecutive calls need no clearing; calls that overlap in
// time on one device race.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "more.h"

namespace {

static __device__ __align__(256) unsigned char scratch[MORE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_mu;

// Device address of `scratch` on the current device (looked up once per device), or nullptr
// with *err set.
void* device_scratch(hipError_t* err) {
    int dev = 0;
    *err = hipGetDevice(&dev);
    if (*err != hipSuccess) return nullptr;
    if (dev < 0 || dev >= kMaxDevices) {
        *err = hipErrorInvalidDevice;
        return nullptr;
    }
    void* p = g_scratch[dev].load(std::memory_order_acquire);
    if (p) return p;
    std::lock_guard<std::mutex> lock(g_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
        *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (*err != hipSuccess || !p) {
            if (*err == hipSuccess) *err = hipErrorInvalidSymbol;
            return nullptr;
        }
        g_scratch[dev].store(p, std::memory_order_release);
    }
    return p;
}

}  // namespace

extern "C" more_status more_route_lowrank_noalloc(const uint16_t* x, const uint16_t* R1t,
                                                  const uint16_t* R2t, int64_t T, int32_t h,
                                                  int32_t r, int32_t M, int32_t k, int32_t* idx,
                                                  float* gate, float* topval, int32_t* counts,
                                                  void* stream) {
    // Arguments and the scratch size are checked on the host before anything else.
    size_t need = 0;
    more_status s = more_route_lowrank_workspace_size(T, h, r, M, k, &need);
    if (s != MORE_OK) return s;
    if (need > MORE_NOALLOC_SCRATCH_BYTES) return MORE_ERR_WORKSPACE;
    void* ws = nullptr;
    if (need > 0 && x && R1t && R2t && idx && gate) {
        hipError_t e;
        ws = device_scratch(&e);
        if (!ws) return MORE_ERR_HIP;
    }
    return more_route_lowrank(x, R1t, R2t, T, h, r, M, k, idx, gate, topval, counts, ws,
                              ws ? MORE_NOALLOC_SCRATCH_BYTES : 0, stream);
}
