// Fixed device scratch for the allocation-free backward (tbe_backward_noalloc):
// the backward's workspace lives in a file-scope device array instead of a
// caller buffer, so a caller that cannot allocate (code under HIP graph
// capture, tight serving loops) needs no workspace.
//
// The array exists once per GPU that loads the library and is held until the
// process ends.  Its device address differs per GPU, so it is looked up once
// per device, with that device current, when a plan is created there; host
// code only ever uses the looked-up address.

#include <mutex>

#include "tbe_internal.h"

namespace tbe {
namespace {

static __device__ __align__(256) char scratch[TBE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device, once looked up

}  // namespace

hipError_t noalloc_scratch_init(int device) {
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[device]) return hipSuccess;
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[device] = ptr;
    return hipSuccess;
}

void *noalloc_scratch(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
}

}  // namespace tbe
