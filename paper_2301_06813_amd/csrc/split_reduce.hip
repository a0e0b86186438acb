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

// Sums the S slices of one product's 4-column group gidx (row gidx /
// groups_per_row) in split order and stores it; out-of-range ids do nothing.
template <bool OUT_F32>
__device__ __forceinline__ void reduce_group(const float *ws, int m, int n, int S, void *C,
                                             int64_t ldc, int64_t gidx) {
    const int groups_per_row = (n + 3) / 4;
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

template <bool OUT_F32>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float *ws, int m, int n, int S,
                                                           void *C, int64_t ldc) {
    reduce_group<OUT_F32>(ws, m, n, S, C, ldc, (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

// The split reductions of the two backward products of one linear in one
// launch: blocks [0, blocks_d) reduce the backward-data product, the rest the
// backward-weight product.
struct ReduceJob {
    const float *ws;
    int m, n, S;
    void *C;
    int64_t ldc;
};

template <bool OD, bool OW>
__global__ __launch_bounds__(256) void split_reduce_pair_kernel(ReduceJob d, ReduceJob w,
                                                                int blocks_d) {
    const int b = blockIdx.x;
    if (b < blocks_d)
        reduce_group<OD>(d.ws, d.m, d.n, d.S, d.C, d.ldc, (int64_t)b * blockDim.x + threadIdx.x);
    else
        reduce_group<OW>(w.ws, w.m, w.n, w.S, w.C, w.ldc,
                         (int64_t)(b - blocks_d) * blockDim.x + threadIdx.x);
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

static unsigned reduce_blocks(const Gemm &g) {
    const int64_t groups = g.m * ((g.n + 3) / 4);
    return (unsigned)((groups + 255) / 256);
}

hipError_t launch_split_reduce_pair(const Gemm &gd, int sd, const float *wsd, const Gemm &gw,
                                    int sw, const float *wsw, hipStream_t s) {
    const sbpk::ReduceJob d{wsd, (int)gd.m, (int)gd.n, sd, gd.C, gd.ldc};
    const sbpk::ReduceJob w{wsw, (int)gw.m, (int)gw.n, sw, gw.C, gw.ldc};
    const unsigned bd = reduce_blocks(gd), bw = reduce_blocks(gw);
    const bool od = gd.out_dtype == DT_F32, ow = gw.out_dtype == DT_F32;
#define SBP_PAIR(OD_, OW_, NAME)                                                             \
    if (od == OD_ && ow == OW_)                                                              \
        return launch_kernel(sbpk::split_reduce_pair_kernel<OD_, OW_>, NAME, dim3(bd + bw),  \
                             dim3(256), s, d, w, (int)bd);
    SBP_PAIR(true, true, "split_reduce_pair_kernel<true, true>")
    SBP_PAIR(true, false, "split_reduce_pair_kernel<true, false>")
    SBP_PAIR(false, true, "split_reduce_pair_kernel<false, true>")
    SBP_PAIR(false, false, "split_reduce_pair_kernel<false, false>")
#undef SBP_PAIR
    return hipErrorInvalidValue;
}

}  // namespace sbpi
