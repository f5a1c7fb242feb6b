// noalloc.hip -- rubiconv_packed_conv_noalloc: the packed convolution with its scratch
// (the transform grid and the prescale words) taken from a fixed device array instead
// of a caller's workspace, for callers that cannot allocate device memory.
//
// The array lives in this file as a static __device__ object: every device that loads
// the library holds one copy of kNoAllocScratchBytes until the process ends.  In host
// code its name is only a host-side stand-in, so the device address of each device's
// copy is looked up once per device (hipGetSymbolAddress, with that device current) and
// only that address is handed to the kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "rubiconv.h"

namespace {

constexpr size_t kNoAllocScratchBytes = RUBICONV_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (looked up on first use).
rubiconv_status_t scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return RUBICONV_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return RUBICONV_ERR_HIP;
        }
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return RUBICONV_OK;
}

}  // namespace

extern "C" {

rubiconv_status_t rubiconv_packed_conv_noalloc(rubiconv_plan_t plan, const void* x, const void* spectrum,
                                               void* y, hipStream_t stream) {
    if (!plan || !x || !spectrum || !y) return RUBICONV_ERR_ARG;
    if (rubiconv_workspace_bytes(plan) > kNoAllocScratchBytes) return RUBICONV_ERR_UNSUPPORTED;
    void* ws = nullptr;
    const rubiconv_status_t st = scratch_address(&ws);
    if (st != RUBICONV_OK) return st;
    return rubiconv_packed_conv(plan, x, spectrum, y, ws, stream);
}

}  // extern "C"
