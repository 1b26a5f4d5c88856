// noalloc.hip -- the fixed device array behind sar_form_image_noalloc, the
// SAR entry point for callers that cannot allocate device memory (code under
// graph capture, tight serving loops).
//
// `scratch` is a file-scope device array: every GPU the library runs on holds
// its own copy, at its own address, until the process ends.  In host code its
// name is only a stand-in for the symbol, never a device address: the address
// comes from hipGetSymbolAddress, looked up once per device (with that device
// current, on the entry point's first call there) and kept per device; host
// code passes that address, and only that, to kernels and copies.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "fft_launch.h"

namespace mi355fft {

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {

std::mutex g_scratch_mutex;
std::map<int, void *> g_scratch;  // device -> its copy of `scratch`

}  // namespace

hipError_t noalloc_scratch(int device, void **ptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    auto it = g_scratch.find(device);
    if (it != g_scratch.end()) {
        *ptr = it->second;
        return hipSuccess;
    }
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch[device] = p;
    *ptr = p;
    return hipSuccess;
}

}  // namespace mi355fft
