// plan.cpp -- choice of output tile and reduction splits for the bf16 GEMM.
//
// A launch fills MI355X's 256 compute units only if it has enough
// workgroups; many local shares of an SBP linear have small outputs and long
// reductions (e.g. a weight gradient of 1024 x 384 over 8192 tokens), so the
// planner trades tile size (MFMA efficiency per workgroup) against the
// number of workgroups and splits of the reduction. It evaluates a small
// analytic time model for every (tile, splits) candidate and keeps the
// fastest. Pure host code.
#include <algorithm>
#include <cmath>
#include <cstdint>

#include "gemm.h"

namespace sbpi {

namespace {

struct TileClass {
    int bm, bn;
    int occ;      // workgroups that fit one compute unit (LDS-limited)
    double eff;   // fraction of the CU's MFMA peak the tile sustains when resident
};

// Generic kernel (register-staged, one step ahead): slower per byte.
const TileClass kGeneric[] = {
    {256, 128, 1, 0.5}, {128, 256, 1, 0.5}, {128, 128, 2, 0.5},
    {128, 64, 2, 0.5},  {64, 128, 2, 0.5},  {64, 64, 4, 0.5},
};
// Pipelined direct-to-LDS kernel.
const TileClass kDma[] = {
    {256, 256, 1, 1.0}, {256, 128, 1, 1.0}, {128, 256, 1, 1.0}, {128, 128, 1, 1.0},
    {128, 64, 1, 1.0},  {64, 128, 1, 1.0},  {64, 64, 2, 1.0},
};

// Time model (measured on MI355X): a workgroup's 64-wide reduction step
// costs the larger of its MFMA time and its operand bytes over the per-CU
// share of L2->LDS bandwidth (about 10 TB/s over 256 CUs when all are busy);
// `eff` scales that rate per kernel. Each wave of workgroups pays a fixed
// latency; split reductions pay their fp32 partials and the reduce kernel.
constexpr double kCUs = 256.0;
constexpr double kCuPeak = 4096.0 * 2.4e9;      // bf16 flop/s per CU
constexpr double kCuL2 = 40.0e9;                // L2 -> LDS bytes/s per CU, chip busy
constexpr double kHbm = 5.0e12;                 // sustained HBM bytes/s (mixed read/write)
constexpr double kRoundLatency = 2.0e-6;        // pipeline fill + epilogue per wave
constexpr double kLaunch = 2.0e-6;              // extra launch (reduce kernel)

thread_local int ov_bm = 0, ov_bn = 0, ov_splits = 1, ov_kernel = 0;

int kblocks(int64_t k) { return (int)((k + 63) / 64); }

// Splits actually launched when asking for s, and blocks per split.
void split_of(int kb_total, int s, int *splits, int *per) {
    if (kb_total <= 0) {
        *splits = 1;
        *per = 1;
        return;
    }
    s = std::max(1, std::min(s, kb_total));
    int p = (kb_total + s - 1) / s;
    *per = p;
    *splits = (kb_total + p - 1) / p;
}

bool fits_ws(const Gemm &g, int splits) {
    if (splits == 1) return true;
    return (double)splits * (double)g.m * (double)g.n <= (double)WS_FLOATS;
}

double model_time(const Gemm &g, const TileClass &t, int splits, int per) {
    const int64_t tiles = ((g.m + t.bm - 1) / t.bm) * ((g.n + t.bn - 1) / t.bn);
    const double wgs = (double)tiles * splits;
    const double rounds = std::ceil(wgs / (kCUs * t.occ));
    const double step_bytes = (t.bm + t.bn) * 128.0;
    const double step = std::max(2.0 * t.bm * t.bn * 64.0 / (kCuPeak * 0.9),
                                 step_bytes * t.occ / (kCuL2 * t.eff));
    const double out_bytes = (splits > 1 || g.out_dtype == DT_F32) ? 4.0 : 2.0;
    const double epi = t.bm * t.bn * out_bytes * t.occ / kCuL2;
    double time = rounds * (per * step + epi + kRoundLatency);
    // the whole product cannot beat HBM for its operands and output
    const double algo_bytes = 2.0 * (g.m * g.k + g.k * g.n) +
                              ((g.out_dtype == DT_F32) ? 4.0 : 2.0) * g.m * g.n;
    time = std::max(time, algo_bytes / kHbm);
    if (splits > 1) {
        const double red = (splits * 4.0 + ((g.out_dtype == DT_F32) ? 4.0 : 2.0)) * g.m * g.n;
        time += red / kHbm + kLaunch;
    }
    return time;
}

}  // namespace

bool tile_supported(int bm, int bn, bool dma) {
    if (dma) {
        for (const TileClass &t : kDma)
            if (t.bm == bm && t.bn == bn) return true;
    } else {
        for (const TileClass &t : kGeneric)
            if (t.bm == bm && t.bn == bn) return true;
    }
    return false;
}

void set_override(int bm, int bn, int splits, int kernel) {
    ov_bm = bm;
    ov_bn = bn;
    ov_splits = std::max(1, splits);
    ov_kernel = kernel;
}

static bool kmajor_a(int orient) { return orient != OR_BWD_WEIGHT; }
static bool kmajor_b(int orient) { return orient == OR_BWD_DATA; }

bool dma_eligible(const Gemm &g) {
    if (g.in_dtype != DT_BF16) return false;
    const auto al = [](const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    if (!al(g.A) || !al(g.B) || g.lda % 8 || g.ldb % 8) return false;
    const int64_t a_contig = kmajor_a(g.orient) ? g.k : g.m;
    const int64_t b_contig = kmajor_b(g.orient) ? g.k : g.n;
    if (a_contig % 8 || b_contig % 8) return false;
    // per-tile buffer offsets stay below 2^31 bytes
    return g.lda <= (int64_t(1) << 21) && g.ldb <= (int64_t(1) << 21);
}

Plan plan_bf16(const Gemm &g) {
    const int kb_total = kblocks(g.k);
    const bool dma = dma_eligible(g);
    Plan best{128, 128, 1, std::max(1, kb_total), dma};
    if (ov_bm != 0) {
        // kernel: 0 either, 1 pipelined (if eligible), 2 generic
        const bool use_dma = dma && ov_kernel != 2;
        Plan p{ov_bm, ov_bn, 1, 1, use_dma};
        if (!tile_supported(p.bm, p.bn, use_dma)) p.bn = 128;   // 256x256 only pipelined
        split_of(kb_total, ov_splits, &p.splits, &p.kblk_per_split);
        while (p.splits > 1 && !fits_ws(g, p.splits))
            split_of(kb_total, p.splits - 1, &p.splits, &p.kblk_per_split);
        return p;
    }
    double best_t = 1e30;
    const TileClass *tiles_tab = dma ? kDma : kGeneric;
    const int ntiles = dma ? (int)(sizeof(kDma) / sizeof(kDma[0]))
                           : (int)(sizeof(kGeneric) / sizeof(kGeneric[0]));
    for (int ti = 0; ti < ntiles; ++ti) {
        const TileClass &t = tiles_tab[ti];
        int last_splits = 0;
        for (int s = 1; s <= 32; ++s) {
            int splits, per;
            split_of(kb_total, s, &splits, &per);
            if (splits == last_splits) continue;
            last_splits = splits;
            if (splits > 1 && per < 2) continue;            // keep >= 128 reduction per split
            if (!fits_ws(g, splits)) continue;
            const double tm = model_time(g, t, splits, per);
            if (tm < best_t * 0.999) {
                best_t = tm;
                best = Plan{t.bm, t.bn, splits, per, dma};
            }
        }
    }
    return best;
}

}  // namespace sbpi
