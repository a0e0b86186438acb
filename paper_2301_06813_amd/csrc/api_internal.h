// api_internal.h -- host helpers shared by the C-ABI translation units.
#pragma once

#include <hip/hip_runtime.h>

#include "gemm.h"

namespace sbpa {

// Plans and launches one product (bf16 kernels, or the fp32 kernel for fp32
// inputs) on stream s; SBP_OK, or SBP_ERR_HIP with the HIP error recorded
// for sbp_last_hip_error(). An empty product launches nothing.
int run_gemm(const sbpi::Gemm &g, hipStream_t s);

}  // namespace sbpa
