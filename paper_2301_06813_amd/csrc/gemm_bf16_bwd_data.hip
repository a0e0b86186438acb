// bf16 GEMM instances for the bwd_data orientation (see gemm_bf16_kernel.h).
#include "gemm_bf16_launch.h"

namespace sbpi {
hipError_t launch_bf16_bwd_data(const Gemm &g, const Plan &p, float *ws, hipStream_t s) {
    return launch_orient<true, true>(g, p, ws, s);
}
}  // namespace sbpi
