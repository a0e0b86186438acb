// gemm_bf16_launch.h -- host-side launch of one orientation of the bf16 GEMM.
// Included by one translation unit per orientation so the tile instances of
// the three orientations compile in parallel.
#pragma once

#include "gemm.h"
#include "gemm_bf16_dma.h"

namespace sbpi {

template <bool AK, bool BK_, bool OUTF>
static hipError_t launch_tile(int bm, int bn, bool dma, const sbpk::GemmArgs &a, int grid,
                              hipStream_t s) {
#define SBP_TILE(BM_, BN_)                                                                  \
    if (!dma && bm == BM_ && bn == BN_) {                                                   \
        hipLaunchKernelGGL((sbpk::gemm_bf16_kernel<BM_, BN_, AK, BK_, OUTF>), dim3(grid),   \
                           dim3(sbpk::NT), 0, s, a);                                        \
        return hipGetLastError();                                                           \
    }
#define SBP_DMA_TILE(BM_, BN_, BKD_, NS_, WGM_, WGN_)                                       \
    if (dma && bm == BM_ && bn == BN_) {                                                    \
        hipLaunchKernelGGL(                                                                 \
            (sbpk::gemm_bf16_dma_kernel<BM_, BN_, BKD_, NS_, WGM_, WGN_, AK, BK_, OUTF>),   \
            dim3(grid), dim3(64 * WGM_ * WGN_), 0, s, a);                                   \
        return hipGetLastError();                                                           \
    }
    SBP_TILE(256, 128)
    SBP_TILE(128, 256)
    SBP_TILE(128, 128)
    SBP_TILE(128, 64)
    SBP_TILE(64, 128)
    SBP_TILE(64, 64)
    SBP_DMA_TILE(256, 256, 64, 2, 2, 4)
    SBP_DMA_TILE(256, 128, 64, 3, 2, 2)
    SBP_DMA_TILE(128, 256, 64, 3, 2, 2)
    SBP_DMA_TILE(128, 128, 64, 4, 2, 2)
    SBP_DMA_TILE(128, 64, 64, 4, 2, 2)
    SBP_DMA_TILE(64, 128, 64, 4, 2, 2)
    SBP_DMA_TILE(64, 64, 64, 4, 2, 2)
#undef SBP_TILE
#undef SBP_DMA_TILE
    return hipErrorInvalidValue;
}

template <bool AK, bool BK_>
static hipError_t launch_orient(const Gemm &g, const Plan &p, float *ws, hipStream_t s) {
    sbpk::GemmArgs a;
    a.A = static_cast<const uint16_t *>(g.A);
    a.B = static_cast<const uint16_t *>(g.B);
    a.C = g.C;
    a.lda = g.lda;
    a.ldb = g.ldb;
    a.ldc = g.ldc;
    a.m = (int32_t)g.m;
    a.n = (int32_t)g.n;
    a.k = (int32_t)g.k;
    a.tiles_m = (int32_t)((g.m + p.bm - 1) / p.bm);
    a.tiles_n = (int32_t)((g.n + p.bn - 1) / p.bn);
    a.splits = p.splits;
    a.kchunk = p.kblk_per_split * 64;
    a.ws = ws;
    a.vec_a = ((reinterpret_cast<uintptr_t>(g.A) & 15) == 0) && (g.lda % 8 == 0);
    a.vec_b = ((reinterpret_cast<uintptr_t>(g.B) & 15) == 0) && (g.ldb % 8 == 0);
    const int grid = a.tiles_m * a.tiles_n * a.splits;
    // with splits the GEMM writes fp32 partials, whatever the output dtype
    hipError_t e = (g.out_dtype == DT_F32 || p.splits > 1)
                       ? launch_tile<AK, BK_, true>(p.bm, p.bn, p.dma, a, grid, s)
                       : launch_tile<AK, BK_, false>(p.bm, p.bn, p.dma, a, grid, s);
    if (e != hipSuccess || p.splits == 1) return e;
    return launch_split_reduce(g, p.splits, ws, s);
}

}  // namespace sbpi
