// split_reduce.hip -- second half of the split reduction.
//
// A GEMM launched with S > 1 reduction splits leaves S fp32 partial
// products in a workspace, slice s holding the m x n output of split s
// (row-major, ld n). This kernel adds the slices in split order
// 0, 1, ..., S-1 -- the same order whatever the schedule, so results are
// deterministic -- and writes the output as fp32, or as bf16 rounded to
// nearest even. Each thread owns 4 consecutive columns of one row: 16-byte
// loads of every slice when n is a multiple of 4, and stores that are
// contiguous across the threads of a wave.
#include "gemm.h"
#include "profile.h"

namespace sbpk {

typedef float f32x4v __attribute__((ext_vector_type(4)));

template <bool OUT_F32>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float *ws, int m, int n, int S,
                                                           void *C, int64_t ldc) {
    const int groups_per_row = (n + 3) / 4;
    const int64_t gidx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gidx >= (int64_t)m * groups_per_row) return;
    const int row = (int)(gidx / groups_per_row);
    const int col = (int)(gidx % groups_per_row) * 4;
    const size_t slice = (size_t)m * (size_t)n;
    const float *p = ws + (size_t)row * n + col;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if ((n & 3) == 0) {
        for (int s = 0; s < S; ++s) {
            const f32x4v x = __builtin_nontemporal_load(reinterpret_cast<const f32x4v *>(p + s * slice));
            v[0] += x[0];
            v[1] += x[1];
            v[2] += x[2];
            v[3] += x[3];
        }
    } else {
        for (int s = 0; s < S; ++s)
            for (int e = 0; e < 4; ++e)
                if (col + e < n) v[e] += p[s * slice + e];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (col + e >= n) break;
        if constexpr (OUT_F32) {
            reinterpret_cast<float *>(C)[(int64_t)row * ldc + col + e] = v[e];
        } else {
            __bf16 h = (__bf16)v[e];
            reinterpret_cast<uint16_t *>(C)[(int64_t)row * ldc + col + e] =
                __builtin_bit_cast(uint16_t, h);
        }
    }
}

}  // namespace sbpk

namespace sbpi {

hipError_t launch_split_reduce(const Gemm &g, int splits, const float *ws, hipStream_t s) {
    const int64_t groups = g.m * ((g.n + 3) / 4);
    const unsigned blocks = (unsigned)((groups + 255) / 256);
    if (g.out_dtype == DT_F32)
        return launch_kernel(sbpk::split_reduce_kernel<true>, "split_reduce_kernel<true>",
                             dim3(blocks), dim3(256), s, ws, (int)g.m, (int)g.n, splits, g.C,
                             g.ldc);
    return launch_kernel(sbpk::split_reduce_kernel<false>, "split_reduce_kernel<false>",
                         dim3(blocks), dim3(256), s, ws, (int)g.m, (int)g.n, splits, g.C, g.ldc);
}

}  // namespace sbpi
