// Grouped backward launch: the backward-data and backward-weight products of
// one linear in a single grid (see gemm_bf16_dma_bwd_kernel).
#include "gemm_bf16_launch.h"

namespace sbpi {

namespace {

template <bool OD, bool OW>
hipError_t launch_group_tile(const Plan &p, const sbpk::GemmArgsShift &ds,
                             const sbpk::GemmArgsShift &ws, int data_first, int grid,
                             hipStream_t s) {
    const sbpk::GemmArgs d = ds, w = ws;   // the unshifted kernels' arguments
    char name[192];
    const char *tf[2] = {"false", "true"};
    if (p.shift) {
#define SBP_BWD_SHIFT_TILE(BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_)                         \
    if (p.bm == BM_ && p.bn == BN_ && p.bk == BKD_ && (p.ns == 0 || p.ns == NS_) &&             \
        p.kg == KG_ && p.epi == EPI_) {                                                        \
        snprintf(name, sizeof(name),                                                           \
                 "gemm_bf16_dma_bwd_kernel<%d, %d, %d, %d, %d, %d, %d, %d, %s, %s, true>",    \
                 BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_, tf[OD], tf[OW]);                 \
        return launch_kernel(                                                                  \
            sbpk::gemm_bf16_dma_bwd_kernel<BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_, OD, OW, \
                                           true>,                                              \
            name, dim3(grid), dim3(64 * WGM_ * WGN_ * KG_), s, ds, ws, data_first);            \
    }
        SBP_DMA_SHIFT_INSTANCES(SBP_BWD_SHIFT_TILE)
#undef SBP_BWD_SHIFT_TILE
        return hipErrorInvalidValue;
    }
#define SBP_BWD_TILE(BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_)                           \
    if (p.bm == BM_ && p.bn == BN_ && p.bk == BKD_ && (p.ns == 0 || p.ns == NS_) &&         \
        p.kg == KG_ && p.epi == EPI_) {                                                    \
        snprintf(name, sizeof(name),                                                       \
                 "gemm_bf16_dma_bwd_kernel<%d, %d, %d, %d, %d, %d, %d, %d, %s, %s>", BM_,  \
                 BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_, tf[OD], tf[OW]);                   \
        return launch_kernel(                                                              \
            sbpk::gemm_bf16_dma_bwd_kernel<BM_, BN_, BKD_, NS_, WGM_, WGN_, KG_, EPI_, OD, \
                                           OW>,                                            \
            name, dim3(grid), dim3(64 * WGM_ * WGN_ * KG_), s, d, w, data_first);          \
    }
    SBP_DMA_INSTANCES(SBP_BWD_TILE)
#undef SBP_BWD_TILE
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_bf16_bwd_group(const Gemm &gd, const Plan &pd, const Gemm &gw,
                                 const Plan &pw, float *ws, hipStream_t s) {
    if (pd.bm != pw.bm || pd.bn != pw.bn || pd.bk != pw.bk || pd.ns != pw.ns || pd.kg != pw.kg ||
        pd.epi != pw.epi || pd.shift != pw.shift || !pd.dma || !pw.dma)
        return hipErrorInvalidValue;
    float *const ws_w = ws + plan_ws_floats(gd, pd);
    const sbpk::GemmArgsShift d = make_args(gd, pd, ws);
    const sbpk::GemmArgsShift w = make_args(gw, pw, ws_w);
    const int grid = d.tiles_m * d.tiles_n * d.splits + w.tiles_m * w.tiles_n * w.splits;
    const int data_first = pd.kblk_per_split >= pw.kblk_per_split;
    const bool od = gd.out_dtype == DT_F32 || pd.splits > 1;
    const bool ow = gw.out_dtype == DT_F32 || pw.splits > 1;
    hipError_t e;
    if (od && ow) e = launch_group_tile<true, true>(pd, d, w, data_first, grid, s);
    else if (od) e = launch_group_tile<true, false>(pd, d, w, data_first, grid, s);
    else if (ow) e = launch_group_tile<false, true>(pd, d, w, data_first, grid, s);
    else e = launch_group_tile<false, false>(pd, d, w, data_first, grid, s);
    if (e != hipSuccess) return e;
    if (pd.splits > 1 && pw.splits > 1)
        return launch_split_reduce_pair(gd, pd.splits, ws, gw, pw.splits, ws_w, s);
    if (pd.splits > 1 && (e = launch_split_reduce(gd, pd.splits, ws, s)) != hipSuccess) return e;
    if (pw.splits > 1 && (e = launch_split_reduce(gw, pw.splits, ws_w, s)) != hipSuccess) return e;
    return hipSuccess;
}

}  // namespace sbpi
