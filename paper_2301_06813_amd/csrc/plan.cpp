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

#include "gemm.h"

namespace sbpi {

namespace {

struct TileClass {
    int bm, bn;
    int occ;      // workgroups that fit one compute unit (LDS-limited)
    double eff;   // fraction of the CU's MFMA peak the tile sustains when resident
};

// LDS per workgroup is 2 stages x (bm + bn) x 128 B; 160 KB per CU.
const TileClass kTiles[] = {
    {256, 128, 1, 0.70}, {128, 256, 1, 0.70}, {128, 128, 2, 0.60},
    {128, 64, 2, 0.45},  {64, 128, 2, 0.45},  {64, 64, 4, 0.30},
};

constexpr double kCUs = 256.0;
constexpr double kCuPeak = 4096.0 * 2.4e9;      // bf16 flop/s per CU
constexpr double kHbm = 6.0e12;                 // sustainable HBM bytes/s
constexpr double kCuBw = 150.0e9;               // bytes/s one CU streams alone
constexpr double kRoundLatency = 0.6e-6;        // per wave of workgroups

thread_local int ov_bm = 0, ov_bn = 0, ov_splits = 1;

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

bool fits_ws(int64_t tiles, int splits, int bm, int bn) {
    if (splits == 1) return true;
    return tiles <= (int64_t)WS_COUNTERS &&
           (double)tiles * splits * bm * bn <= (double)WS_FLOATS;
}

double model_time(const Gemm &g, const TileClass &t, int splits, int per) {
    const int64_t tiles = ((g.m + t.bm - 1) / t.bm) * ((g.n + t.bn - 1) / t.bn);
    const double wgs = (double)tiles * splits;
    const double slots = kCUs * t.occ;
    const double rounds = std::ceil(wgs / slots);
    const double kc = (double)per * 64.0;
    const double wg_time = t.occ * (2.0 * t.bm * t.bn * kc) / (kCuPeak * t.eff);
    double time = rounds * (wg_time + kRoundLatency);
    const double out_bytes = (g.out_dtype == DT_F32) ? 4.0 : 2.0;
    const double algo_bytes = 2.0 * (g.m * g.k + g.k * g.n) + out_bytes * g.m * g.n;
    time = std::max(time, algo_bytes / kHbm);
    if (splits > 1) {
        time += 2.0 * wgs * t.bm * t.bn * 4.0 / kHbm;              // partials out and back
        time += splits * (double)t.bm * t.bn * 4.0 / kCuBw;         // serial sum in the last WG
    }
    return time;
}

}  // namespace

bool tile_supported(int bm, int bn) {
    for (const TileClass &t : kTiles)
        if (t.bm == bm && t.bn == bn) return true;
    return false;
}

void set_override(int bm, int bn, int splits) {
    ov_bm = bm;
    ov_bn = bn;
    ov_splits = std::max(1, splits);
}

Plan plan_bf16(const Gemm &g) {
    const int kb_total = kblocks(g.k);
    Plan best{128, 128, 1, std::max(1, kb_total)};
    if (ov_bm != 0) {
        Plan p{ov_bm, ov_bn, 1, 1};
        split_of(kb_total, ov_splits, &p.splits, &p.kblk_per_split);
        const int64_t tiles = ((g.m + p.bm - 1) / p.bm) * ((g.n + p.bn - 1) / p.bn);
        while (p.splits > 1 && !fits_ws(tiles, p.splits, p.bm, p.bn))
            split_of(kb_total, p.splits - 1, &p.splits, &p.kblk_per_split);
        return p;
    }
    double best_t = 1e30;
    for (const TileClass &t : kTiles) {
        const int64_t tiles = ((g.m + t.bm - 1) / t.bm) * ((g.n + t.bn - 1) / t.bn);
        int last_splits = 0;
        for (int s = 1; s <= 32; ++s) {
            int splits, per;
            split_of(kb_total, s, &splits, &per);
            if (splits == last_splits) continue;
            last_splits = splits;
            if (splits > 1 && per < 2) continue;            // keep >= 128 reduction per split
            if (!fits_ws(tiles, splits, t.bm, t.bn)) continue;
            const double tm = model_time(g, t, splits, per);
            if (tm < best_t * 0.999) {
                best_t = tm;
                best = Plan{t.bm, t.bn, splits, per};
            }
        }
    }
    return best;
}

}  // namespace sbpi
