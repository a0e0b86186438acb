// gemm_f32.hip -- fp32-input path of the local matmul and the bf16 dispatch
// by orientation.
//
// The fp32 path serves fp32 workloads (small layers trained in single
// precision). It is a plain LDS-tiled fp32 FMA kernel: 64 x 64 output tile,
// reduction step 16, 256 threads each owning a 4 x 4 strided sub-block, so
// that global loads and stores are coalesced for every operand orientation.
// Products and sums are single fp32 FMAs; the reduction order is
// increasing k.
#include "gemm.h"
#include "profile.h"

namespace sbpk {

constexpr int F_BM = 64, F_BN = 64, F_BK = 16;

struct F32Args {
    const float *A;
    const float *B;
    float *C;
    int64_t lda, ldb, ldc;
    int32_t m, n, k;
    int32_t tiles_n;
    int32_t accumulate;   // add the product to C's contents
};

template <bool A_KMAJ, bool B_KMAJ>
__global__ __launch_bounds__(256) void gemm_f32_kernel(F32Args g) {
    __shared__ float As[F_BK][F_BM + 1];
    __shared__ float Bs[F_BK][F_BN + 1];
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int tm = blockIdx.x / g.tiles_n, tn = blockIdx.x % g.tiles_n;
    const int m0 = tm * F_BM, n0 = tn * F_BN;
    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

    for (int k0 = 0; k0 < g.k; k0 += F_BK) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + 256 * q;
            int i, kk;
            if (A_KMAJ) { i = e / F_BK; kk = e % F_BK; } else { kk = e / F_BM; i = e % F_BM; }
            const int gi = m0 + i, gk = k0 + kk;
            float v = 0.f;
            if (gi < g.m && gk < g.k)
                v = A_KMAJ ? g.A[(int64_t)gi * g.lda + gk] : g.A[(int64_t)gk * g.lda + gi];
            As[kk][i] = v;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + 256 * q;
            int j, kk;
            if (B_KMAJ) { j = e / F_BK; kk = e % F_BK; } else { kk = e / F_BN; j = e % F_BN; }
            const int gj = n0 + j, gk = k0 + kk;
            float v = 0.f;
            if (gj < g.n && gk < g.k)
                v = B_KMAJ ? g.B[(int64_t)gj * g.ldb + gk] : g.B[(int64_t)gk * g.ldb + gj];
            Bs[kk][j] = v;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < F_BK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = m0 + ty + 16 * i;
        if (row >= g.m) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = n0 + tx + 16 * j;
            if (col >= g.n) continue;
            float *c = g.C + (int64_t)row * g.ldc + col;
            *c = g.accumulate ? *c + acc[i][j] : acc[i][j];
        }
    }
}

}  // namespace sbpk

namespace sbpi {

hipError_t launch_bf16_fwd(const Gemm &, const Plan &, float *, hipStream_t);
hipError_t launch_bf16_bwd_data(const Gemm &, const Plan &, float *, hipStream_t);
hipError_t launch_bf16_bwd_weight(const Gemm &, const Plan &, float *, hipStream_t);

hipError_t launch_bf16(const Gemm &g, const Plan &p, float *ws, hipStream_t s) {
    switch (g.orient) {
        case OR_FWD: return launch_bf16_fwd(g, p, ws, s);
        case OR_BWD_DATA: return launch_bf16_bwd_data(g, p, ws, s);
        case OR_BWD_WEIGHT: return launch_bf16_bwd_weight(g, p, ws, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_f32(const Gemm &g, hipStream_t s) {
    sbpk::F32Args a;
    a.A = static_cast<const float *>(g.A);
    a.B = static_cast<const float *>(g.B);
    a.C = static_cast<float *>(g.C);
    a.lda = g.lda;
    a.ldb = g.ldb;
    a.ldc = g.ldc;
    a.m = (int32_t)g.m;
    a.n = (int32_t)g.n;
    a.k = (int32_t)g.k;
    a.accumulate = g.accumulate;
    const int tiles_m = (int)((g.m + sbpk::F_BM - 1) / sbpk::F_BM);
    a.tiles_n = (int)((g.n + sbpk::F_BN - 1) / sbpk::F_BN);
    const int grid = tiles_m * a.tiles_n;
    switch (g.orient) {
        case OR_FWD:
            return launch_kernel(sbpk::gemm_f32_kernel<true, false>,
                                 "gemm_f32_kernel<true, false>", dim3(grid), dim3(256), s, a);
        case OR_BWD_DATA:
            return launch_kernel(sbpk::gemm_f32_kernel<true, true>,
                                 "gemm_f32_kernel<true, true>", dim3(grid), dim3(256), s, a);
        case OR_BWD_WEIGHT:
            return launch_kernel(sbpk::gemm_f32_kernel<false, false>,
                                 "gemm_f32_kernel<false, false>", dim3(grid), dim3(256), s, a);
    }
    return hipErrorInvalidValue;
}

}  // namespace sbpi
