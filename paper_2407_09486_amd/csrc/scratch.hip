// Fixed device scratch of the allocation-free scoring entry point (enova_detect_score_noalloc).
//
// The array below is a file-scope device variable: every GPU that loads this library holds its
// own copy, at its own address, until the process ends. In host code the name `scratch` is a
// host-side stand-in, never a device address: host code uses only the pointer that
// hipGetSymbolAddress returns for the current device, looked up once per device at detector
// set-up (enova_detect_init) and kept here.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace enova {

namespace {
constexpr int kScratchDevices = 64;
}

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
std::mutex g_scratch_mu;
void *g_scratch_ptr[kScratchDevices] = {};
}  // namespace

hipError_t scratch_setup(int device, void **out)
{
    *out = nullptr;
    if (device < 0 || device >= kScratchDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        int cur = -1;
        hipError_t e = hipGetDevice(&cur);
        if (e != hipSuccess)
            return e;
        if (cur != device)
            return hipErrorInvalidDevice;     // the caller makes `device` current first
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (!p)
            return hipErrorInvalidSymbol;
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return hipSuccess;
}

}  // namespace enova
