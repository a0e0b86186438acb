// gemm_bf16_launch.h -- host-side launch of one orientation of the bf16 GEMM.
// Included by one translation unit per orientation so the tile instances of
// the three orientations compile in parallel.
#pragma once

#include <algorithm>

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

// Instances of the pipelined kernel: tile, stages, wave layout, reduction
// groups and epilogue. The macro list is shared by the single-product and
// the grouped backward launchers.
#define SBP_DMA_INSTANCES(X)                                    \
    X(256, 256, 64, 2, 2, 4, 1, sbpk::EPI_DIRECT)               \
    X(256, 192, 64, 2, 4, 2, 1, sbpk::EPI_DIRECT)               \
    X(256, 256, 64, 2, 2, 4, 1, sbpk::EPI_ROWQ)                     \
    X(256, 128, 64, SBP_NS_256x128, 2, 2, 1, sbpk::EPI_DIRECT)      \
    X(128, 256, 64, SBP_NS_256x128, 2, 2, 1, sbpk::EPI_DIRECT)      \
    X(128, 128, 64, SBP_NS_128x128, 2, 2, 1, sbpk::EPI_DIRECT)      \
    X(128, 128, 64, 2, 2, 2, 1, sbpk::EPI_DIRECT)                   \
    X(128, 128, 64, 2, 2, 2, 1, sbpk::EPI_ROWQ)                     \
    X(128, 64, 64, SBP_NS_128x64, 2, 2, 1, sbpk::EPI_DIRECT)        \
    X(64, 128, 64, SBP_NS_128x64, 2, 2, 1, sbpk::EPI_DIRECT)        \
    X(64, 64, 64, SBP_NS_64x64, 2, 2, 1, sbpk::EPI_DIRECT)          \
    X(256, 128, 64, SBP_NS_256x128, 2, 2, 2, sbpk::EPI_STAGED)      \
    X(128, 256, 64, SBP_NS_256x128, 2, 2, 2, sbpk::EPI_STAGED)      \
    X(128, 128, 64, SBP_NS_128x128, 2, 2, 2, sbpk::EPI_STAGED)      \
    X(256, 128, 64, SBP_NS_256x128, 2, 2, 2, sbpk::EPI_ROWQ)        \
    X(128, 256, 64, SBP_NS_256x128, 2, 2, 2, sbpk::EPI_ROWQ)        \
    X(128, 128, 64, SBP_NS_128x128, 2, 2, 2, sbpk::EPI_ROWQ) \
    X(256, 256, 32, 5, 2, 4, 1, sbpk::EPI_DIRECT)               \
    X(256, 128, 32, 6, 2, 2, 2, sbpk::EPI_STAGED)               \
    X(128, 256, 32, 6, 2, 2, 2, sbpk::EPI_STAGED)               \
    X(128, 128, 32, 8, 2, 2, 2, sbpk::EPI_STAGED)               \
    X(128, 128, 64, 2, 2, 2, 2, sbpk::EPI_STAGED)               \
    X(128, 64, 64, 2, 2, 2, 1, sbpk::EPI_DIRECT)                \
    X(64, 128, 64, 2, 2, 2, 1, sbpk::EPI_DIRECT)                \
    X(64, 64, 64, 2, 2, 2, 1, sbpk::EPI_DIRECT)                 \
    X(128, 64, 64, 6, 2, 2, 1, sbpk::EPI_DIRECT)                \
    X(64, 128, 64, 6, 2, 2, 1, sbpk::EPI_DIRECT)                \
    X(64, 64, 64, 8, 2, 2, 1, sbpk::EPI_DIRECT)                 \
    X(128, 64, 64, SBP_NS_128x64, 2, 2, 2, sbpk::EPI_STAGED)       \
    X(64, 128, 64, SBP_NS_128x64, 2, 2, 2, sbpk::EPI_STAGED)       \
    X(64, 64, 64, SBP_NS_64x64, 2, 2, 2, sbpk::EPI_STAGED)         \
    X(128, 64, 64, SBP_NS_128x64, 2, 2, 2, sbpk::EPI_ROWQ)         \
    X(64, 128, 64, SBP_NS_128x64, 2, 2, 2, sbpk::EPI_ROWQ)         \
    X(64, 64, 64, SBP_NS_64x64, 2, 2, 2, sbpk::EPI_ROWQ)         \
    X(128, 128, 128, 2, 2, 2, 2, sbpk::EPI_STAGED)                 \
    X(128, 64, 128, 3, 2, 2, 2, sbpk::EPI_STAGED)                  \
    X(64, 128, 128, 3, 2, 2, 2, sbpk::EPI_STAGED)                  \
    X(64, 64, 128, 4, 2, 2, 2, sbpk::EPI_STAGED)                   \
    X(128, 128, 128, 2, 2, 2, 2, sbpk::EPI_ROWQ)                   \
    X(128, 64, 128, 3, 2, 2, 2, sbpk::EPI_ROWQ)                    \
    X(64, 128, 128, 3, 2, 2, 2, sbpk::EPI_ROWQ)                    \
    X(64, 64, 128, 4, 2, 2, 2, sbpk::EPI_ROWQ)

// Instances that also exist in the shifted-index-space form (operands at an
// offset within a 16-byte block, contiguous extents not multiples of 8: see
// GemmArgs); plan.cpp's kShiftInstances lists the same ones.
#define SBP_DMA_SHIFT_INSTANCES(X)                              \
    X(64, 64, 64, SBP_NS_64x64, 2, 2, 1, sbpk::EPI_DIRECT)      \
    X(128, 128, 64, 2, 2, 2, 1, sbpk::EPI_DIRECT)               \
    X(64, 64, 128, 4, 2, 2, 2, sbpk::EPI_STAGED)                \
    X(128, 64, 128, 3, 2, 2, 2, sbpk::EPI_STAGED)               \
    X(64, 128, 128, 3, 2, 2, 2, sbpk::EPI_STAGED)               \
    X(128, 128, 128, 2, 2, 2, 2, sbpk::EPI_STAGED)

// Grid of a launch of `items` work items under plan p: one workgroup per item,
// or (persistent plans) at most occ workgroups per compute unit, a multiple of 8.
static inline int grid_of(const Plan &p, int items) {
    if (p.occ <= 0) return items;
    const int cap = p.occ * device_cus();
    if (items <= cap) return items;
    return std::max(8, cap / 8 * 8);
}

template <bool AK, bool BK_, bool OUTF>
static hipError_t launch_tile(const Plan &p, const sbpk::GemmArgsShift &as, int items,
                              hipStream_t s) {
    const sbpk::GemmArgs a = as;   // the unshifted kernels' arguments
    char name[192];
    const char *tf[2] = {"false", "true"};
    const int grid = grid_of(p, items);
    if (p.dma && p.shift) {
#define SBP_DMA_SHIFT_TILE(BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_)                      \
    if (p.bm == BM_ && p.bn == BN_ && p.bk == BKD_ && (p.ns == 0 || p.ns == NS_) &&          \
        p.kg == KG_ && p.epi == EPI_) {                                                     \
        snprintf(name, sizeof(name),                                                        \
                 "gemm_bf16_dma_kernel<%d, %d, %d, %d, %d, %d, %d, %d, %s, %s, %s, true>",  \
                 BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_, tf[AK], tf[BK_], tf[OUTF]);    \
        return launch_kernel(                                                               \
            sbpk::gemm_bf16_dma_kernel<BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_, AK, BK_, \
                                       OUTF, true>,                                         \
            name, dim3(grid), dim3(64 * WGM_ * WGN_ * KG_), s, as);                         \
    }
        SBP_DMA_SHIFT_INSTANCES(SBP_DMA_SHIFT_TILE)
#undef SBP_DMA_SHIFT_TILE
        return hipErrorInvalidValue;
    }
#define SBP_TILE(BM_, BN_)                                                                  \
    if (!p.dma && p.bm == BM_ && p.bn == BN_) {                                             \
        snprintf(name, sizeof(name), "gemm_bf16_kernel<%d, %d, %s, %s, %s>", BM_, BN_,     \
                 tf[AK], tf[BK_], tf[OUTF]);                                                \
        return launch_kernel(sbpk::gemm_bf16_kernel<BM_, BN_, AK, BK_, OUTF>, name,         \
                             dim3(items), dim3(sbpk::NT), s, a);                            \
    }
#define SBP_DMA_TILE(BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_)                            \
    if (p.dma && p.bm == BM_ && p.bn == BN_ && p.bk == BKD_ &&                               \
        (p.ns == 0 || p.ns == NS_) && p.kg == KG_ && p.epi == EPI_) {                       \
        snprintf(name, sizeof(name),                                                        \
                 "gemm_bf16_dma_kernel<%d, %d, %d, %d, %d, %d, %d, %d, %s, %s, %s>", BM_,   \
                 BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_, tf[AK], tf[BK_], tf[OUTF]);         \
        return launch_kernel(                                                               \
            sbpk::gemm_bf16_dma_kernel<BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_, AK, BK_, \
                                       OUTF>,                                               \
            name, dim3(grid), dim3(64 * WGM_ * WGN_ * KG_), s, a);                          \
    }
    SBP_TILE(256, 128)
    SBP_TILE(128, 256)
    SBP_TILE(128, 128)
    SBP_TILE(128, 64)
    SBP_TILE(64, 128)
    SBP_TILE(64, 64)
    SBP_DMA_INSTANCES(SBP_DMA_TILE)
#undef SBP_TILE
#undef SBP_DMA_TILE
    return hipErrorInvalidValue;
}

// Kernel arguments of product g under plan p (partials, if split, go to ws).
static inline sbpk::GemmArgsShift make_args(const Gemm &g, const Plan &p, float *ws) {
    sbpk::GemmArgsShift a;
    a.A = static_cast<const uint16_t *>(g.A);
    a.B = static_cast<const uint16_t *>(g.B);
    a.sm = a.sn = a.sk = a.kmask = 0;
    if (p.dma && p.shift) {
        // operands at an offset within a 16-byte block: read from the block
        // boundary, shift the kernel's index space (see GemmArgs)
        const int oa = block_offset(g.A), ob = block_offset(g.B);
        const bool ak = g.orient != OR_BWD_WEIGHT, bk = g.orient == OR_BWD_DATA;
        a.A -= oa;
        a.B -= ob;
        a.sm = ak ? 0 : oa;
        a.sn = bk ? 0 : ob;
        a.sk = ak ? oa : 0;
        a.kmask = ak && (a.sk != 0 || g.k % 8 != 0);
    }
    a.C = g.C;
    a.lda = g.lda;
    a.ldb = g.ldb;
    a.ldc = g.ldc;
    a.m = (int32_t)g.m;
    a.n = (int32_t)g.n;
    a.k = (int32_t)g.k;
    a.tiles_m = (int32_t)((g.m + a.sm + p.bm - 1) / p.bm);
    a.tiles_n = (int32_t)((g.n + a.sn + p.bn - 1) / p.bn);
    a.splits = p.splits;
    a.kchunk = p.kblk_per_split * 64;
    a.ws = ws;
    const bool batch_a = g.nbatch() == 1 || (g.sa_b % 8 == 0 && g.sa_h % 8 == 0);
    const bool batch_b = g.nbatch() == 1 || (g.sb_b % 8 == 0 && g.sb_h % 8 == 0);
    a.vec_a = ((reinterpret_cast<uintptr_t>(g.A) & 15) == 0) && (g.lda % 8 == 0) && batch_a;
    a.vec_b = ((reinterpret_cast<uintptr_t>(g.B) & 15) == 0) && (g.ldb % 8 == 0) && batch_b;
    // every batch item's output base must keep the 16-byte alignment
    const int64_t es = g.out_dtype == DT_F32 ? 4 : 2;
    const bool c16 = (reinterpret_cast<uintptr_t>(g.C) & 15) == 0 &&
                     (g.nbatch() == 1 || ((g.sc_b * es) % 16 == 0 && (g.sc_h * es) % 16 == 0));
    // vector stores of whole 4- or 8-column groups: the shifted output
    // columns must keep them aligned
    a.vec_c4 = c16 && (g.ldc % 4 == 0) && a.sn % 4 == 0;
    a.vec_c8 = c16 && (g.ldc % 8 == 0) && a.sn % 8 == 0;
    a.accumulate = g.accumulate;
    a.nbatch = (int32_t)g.nbatch();
    a.heads = (int32_t)g.heads;
    a.sa_b = g.sa_b;
    a.sa_h = g.sa_h;
    a.sb_b = g.sb_b;
    a.sb_h = g.sb_h;
    a.sc_b = g.sc_b;
    a.sc_h = g.sc_h;
    return a;
}

template <bool AK, bool BK_>
static hipError_t launch_orient(const Gemm &g, const Plan &p, float *ws, hipStream_t s) {
    const sbpk::GemmArgsShift a = make_args(g, p, ws);
    const int items = a.tiles_m * a.tiles_n * a.splits * a.nbatch;
    // with splits the GEMM writes fp32 partials, whatever the output dtype
    hipError_t e = (g.out_dtype == DT_F32 || p.splits > 1)
                       ? launch_tile<AK, BK_, true>(p, a, items, s)
                       : launch_tile<AK, BK_, false>(p, a, items, s);
    if (e != hipSuccess || p.splits == 1) return e;
    return launch_split_reduce(g, p.splits, ws, s);
}

}  // namespace sbpi
