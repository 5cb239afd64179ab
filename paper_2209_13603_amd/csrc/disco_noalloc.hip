// disco_noalloc.hip -- disco_forward_noalloc: the forward op with every
// kernel's scratch memory (spectral transforms, fp32 partial outputs of
// channel groups and split patterns) taken from one fixed device array
// instead of the stream-ordered pool, for callers that cannot allocate
// (code under HIP graph capture, tight serving loops).
//
// The array lives in the library's code object: each GPU the library runs on
// holds its own copy, at its own address, until the process ends.  In host
// code the array's name is only a host-side stand-in, so the device address
// is looked up once per device with hipGetSymbolAddress (with that device
// current) and only that address is handed to the kernels.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "disco.h"
#include "disco_internal.h"

namespace {

// 64 MiB: the 2048 x 4096 forward op with 8 -> 8 channels needs about 43 MB
// (the spectral rings' transforms).
constexpr size_t kScratchBytes = (size_t)64 << 20;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on `device` (looked up on the first call there).
disco_status_t scratch_on(int device, void** out) {
    if (device < 0 || device >= kMaxDevices)
        return disco::set_last_error(DISCO_ERR_DEVICE, "device index beyond the non-allocating entry point's table");
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[device]) {
        int cur = 0;
        if (hipGetDevice(&cur) != hipSuccess) return disco::set_last_error(DISCO_ERR_DEVICE, "hipGetDevice failed");
        if (cur != device && hipSetDevice(device) != hipSuccess)
            return disco::set_last_error(DISCO_ERR_DEVICE, "hipSetDevice failed");
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != device) (void)hipSetDevice(cur);
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return disco::set_last_error(DISCO_ERR_DEVICE, (std::string("hipGetSymbolAddress(scratch): ") +
                                                            hipGetErrorString(e)).c_str());
        }
        g_scratch[device] = p;
    }
    *out = g_scratch[device];
    return DISCO_OK;
}

}  // namespace

extern "C" disco_status_t disco_forward_noalloc(disco_plan_t plan, const disco_tensor_t* x,
                                                const disco_tensor_t* w, disco_tensor_t* y,
                                                hipStream_t stream) {
    if (!plan) return disco::set_last_error(DISCO_ERR_INVALID_ARGUMENT, "plan is NULL");
    void* p = nullptr;
    const disco_status_t s = scratch_on(disco::plan_device(plan), &p);
    if (s != DISCO_OK) return s;
    return disco::forward_with_scratch(plan, x, w, y, stream, p, kScratchBytes);
}
