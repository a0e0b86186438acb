// gemm_bf16_launch.h -- host-side launch of one orientation of the bf16 GEMM.
// Included by one translation unit per orientation so the tile instances of
// the three orientations compile in parallel.
#pragma once

#include "gemm.h"
#include "gemm_bf16_dma.h"
#include "profile.h"

// Pipeline depth per tile (stages); defaults keep LDS within 160 KB.
#ifndef SBP_NS_256x128
#define SBP_NS_256x128 3
#endif
#ifndef SBP_NS_128x128
#define SBP_NS_128x128 4
#endif
#ifndef SBP_NS_128x64
#define SBP_NS_128x64 4
#endif
#ifndef SBP_NS_64x64
#define SBP_NS_64x64 4
#endif

namespace sbpi {

template <bool AK, bool BK_, bool OUTF>
static hipError_t launch_tile(int bm, int bn, int ns, bool dma, const sbpk::GemmArgs &a,
                              int grid, hipStream_t s) {
    char name[160];
    const char *tf[2] = {"false", "true"};
#define SBP_TILE(BM_, BN_)                                                                  \
    if (!dma && bm == BM_ && bn == BN_) {                                                   \
        snprintf(name, sizeof(name), "gemm_bf16_kernel<%d, %d, %s, %s, %s>", BM_, BN_,     \
                 tf[AK], tf[BK_], tf[OUTF]);                                                \
        return launch_kernel(sbpk::gemm_bf16_kernel<BM_, BN_, AK, BK_, OUTF>, name,         \
                             dim3(grid), dim3(sbpk::NT), s, a);                             \
    }
#define SBP_DMA_TILE(BM_, BN_, BKD_, NS_, WGM_, WGN_)                                       \
    if (dma && bm == BM_ && bn == BN_ && (ns == 0 || ns == NS_)) {                          \
        snprintf(name, sizeof(name),                                                        \
                 "gemm_bf16_dma_kernel<%d, %d, %d, %d, %d, %d, %s, %s, %s>", BM_, BN_,      \
                 BKD_, NS_, WGM_, WGN_, tf[AK], tf[BK_], tf[OUTF]);                         \
        return launch_kernel(                                                               \
            sbpk::gemm_bf16_dma_kernel<BM_, BN_, BKD_, NS_, WGM_, WGN_, AK, BK_, OUTF>,     \
            name, dim3(grid), dim3(64 * WGM_ * WGN_), s, a);                                \
    }
    SBP_TILE(256, 128)
    SBP_TILE(128, 256)
    SBP_TILE(128, 128)
    SBP_TILE(128, 64)
    SBP_TILE(64, 128)
    SBP_TILE(64, 64)
    SBP_DMA_TILE(256, 256, 64, 2, 2, 4)
    SBP_DMA_TILE(256, 128, 64, SBP_NS_256x128, 2, 2)
    SBP_DMA_TILE(128, 256, 64, SBP_NS_256x128, 2, 2)
    SBP_DMA_TILE(128, 128, 64, SBP_NS_128x128, 2, 2)
    SBP_DMA_TILE(128, 128, 64, 2, 2, 2)
    SBP_DMA_TILE(128, 64, 64, SBP_NS_128x64, 2, 2)
    SBP_DMA_TILE(64, 128, 64, SBP_NS_128x64, 2, 2)
    SBP_DMA_TILE(64, 64, 64, SBP_NS_64x64, 2, 2)
#undef SBP_TILE
#undef SBP_DMA_TILE
    return hipErrorInvalidValue;
}

// Kernel arguments of product g under plan p (partials, if split, go to ws).
static inline sbpk::GemmArgs make_args(const Gemm &g, const Plan &p, float *ws) {
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
    return a;
}

template <bool AK, bool BK_>
static hipError_t launch_orient(const Gemm &g, const Plan &p, float *ws, hipStream_t s) {
    const sbpk::GemmArgs a = make_args(g, p, ws);
    const int grid = a.tiles_m * a.tiles_n * a.splits;
    // with splits the GEMM writes fp32 partials, whatever the output dtype
    hipError_t e = (g.out_dtype == DT_F32 || p.splits > 1)
                       ? launch_tile<AK, BK_, true>(p.bm, p.bn, p.ns, p.dma, a, grid, s)
                       : launch_tile<AK, BK_, false>(p.bm, p.bn, p.ns, p.dma, a, grid, s);
    if (e != hipSuccess || p.splits == 1) return e;
    return launch_split_reduce(g, p.splits, ws, s);
}

}  // namespace sbpi
