// Scratch memory of stage_decode_noalloc (include/stage.h): one fixed array in device memory per
// GPU, from which that entry point carves the workspaces of its decode kernels (row metadata, the
// rotated queries, attention split partials and output, the SwiGLU output and the split-K partials
// of the matrix-core projections), so that the call allocates nothing.
//
// The array is a file-scope device variable of the library's code object: every GPU the library
// runs on holds its own copy, at its own address, from the module's load until the process ends.
// Host code must not use the array's name as a device address (on the host it names a stand-in);
// the device address comes from hipGetSymbolAddress, looked up once per device, with that device
// current, and kept.  Calls on one GPU share its copy: calls that overlap on one GPU race, and
// every call leaves its contents behind (no kernel reads a byte of it that the same call did not
// write first, so nothing needs clearing).
#include <mutex>

#include "stage_kernels.h"

static __device__ __align__(256) unsigned char scratch[stg::kScratchBytes];

namespace stg {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices] = {};
}  // namespace

hipError_t scratch_setup(int device, void **out) {
    *out = nullptr;
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[device]) {
        int cur = -1;
        hipError_t e = hipGetDevice(&cur);
        if (e != hipSuccess) return e;
        if (cur != device) return hipErrorInvalidDevice;  // the caller makes `device` current
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch[device] = p;
    }
    *out = g_scratch[device];
    return hipSuccess;
}

}  // namespace stg
