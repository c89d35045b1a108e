// Scratch of dyad_forward_noalloc: a fixed device array instead of the
// library's per-stream pool buffer, for callers that cannot allocate.
//
// `scratch` below is a file-scope device array.  In host code its name is
// only a host-side stand-in: every host use goes through the device address
// hipGetSymbolAddress returns for it, looked up once per device (with that
// device current) and kept.  Each GPU the library runs on holds its own copy
// of the array until the process ends.
#include <mutex>

#include "dyad_internal.h"

namespace dyad {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch` per device, once looked up

thread_local const ScratchScope *t_scope = nullptr;

}  // namespace

hipError_t noalloc_scratch(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

ScratchScope::ScratchScope(void *p, size_t b) : ptr(p), bytes(b), prev(t_scope) { t_scope = this; }
ScratchScope::~ScratchScope() { t_scope = prev; }

const ScratchScope *current_scratch() { return t_scope; }

}  // namespace dyad
