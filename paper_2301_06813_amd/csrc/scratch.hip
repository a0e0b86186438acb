// scratch.hip -- the library's own split-reduction scratch, for callers that
// cannot allocate device memory (sbp_linear_bwd_noalloc).
//
// The array below is the workspace of every such call on a device: one copy
// per device, placed by the code-object loader and held until the process
// ends. Host code never passes the array's name to a kernel (on the host it
// is only a stand-in for the symbol); it asks the runtime for the array's
// address on the current device once and keeps that per device.
#include <mutex>

#include "gemm.h"

static __device__ __align__(256) float scratch[sbpi::WS_FLOATS_PREFERRED];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
float *g_ptr[kMaxDevices] = {};
}  // namespace

namespace sbpi {

hipError_t static_scratch(float **ptr, size_t *floats) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_ptr[dev] = static_cast<float *>(p);
    }
    *ptr = g_ptr[dev];
    *floats = WS_FLOATS_PREFERRED;
    return hipSuccess;
}

}  // namespace sbpi
