// bf16 GEMM instances for the fwd orientation (see gemm_bf16_kernel.h).
#include "gemm_bf16_launch.h"

namespace sbpi {
hipError_t launch_bf16_fwd(const Gemm &g, const Plan &p, float *ws, hipStream_t s) {
    return launch_orient<true, false>(g, p, ws, s);
}
}  // namespace sbpi
