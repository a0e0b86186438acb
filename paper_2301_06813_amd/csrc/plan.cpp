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
#include <unordered_map>

#include "gemm.h"

namespace sbpi {

namespace {

struct TileClass {
    int bm, bn;
    int occ;      // workgroups that fit one compute unit (LDS-limited)
    double eff;   // rate factor of the tile's operand stream (see model below)
    int ns;       // pipelined kernel stages (0 = default instance)
    int kg = 1;   // pipelined kernel reduction groups (2: eight waves)
    int epi = 0;  // pipelined kernel epilogue
    int occ_persist = 0;   // persistent workgroups per CU (0: one per item)
    int bk = 64;           // reduction elements per pipeline stage
};

// Generic kernel (register-staged, one step ahead): slower per byte.
const TileClass kGeneric[] = {
    {256, 128, 1, 0.5, 0}, {128, 256, 1, 0.5, 0}, {128, 128, 2, 0.5, 0},
    {128, 64, 2, 0.5, 0},  {64, 128, 2, 0.5, 0},  {64, 64, 4, 0.5, 0},
};
// Pipelined direct-to-LDS kernel.
// The two-stage 128 x 128 instance (64 KB of LDS) runs two workgroups per
// CU: one's output stores overlap the other's loads, which pays off when the
// reduction is short and the output large.
// The 128-wide stages with two reduction groups (one workgroup of eight
// waves per CU) stream their operands about 20 % faster per CU.
const TileClass kDma[] = {
    {256, 256, 1, 1.0, 0}, {256, 192, 1, 1.0, 0},
    {256, 128, 1, 1.0, 0}, {128, 256, 1, 1.0, 0}, {128, 128, 1, 1.0, 0},
    {128, 128, 2, 0.8, 2}, {128, 64, 1, 1.0, 0},  {64, 128, 1, 1.0, 0},  {64, 64, 2, 1.0, 0},
    {128, 128, 1, 1.2, 2, 2, 1, 0, 128}, {128, 64, 1, 1.2, 3, 2, 1, 0, 128},
    {64, 128, 1, 1.2, 3, 2, 1, 0, 128},  {64, 64, 1, 1.2, 4, 2, 1, 0, 128},
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

thread_local int ov_bm = 0, ov_bn = 0, ov_splits = 1, ov_kernel = 0, ov_occ = 0;
thread_local int ov_orients = 7;   // orientations the override applies to (bit per Orient)
thread_local int ov_bwd_mode = 0, ov_bwd_splits_w = 1;   // see set_bwd_override

// Pipelined instances reachable through the plan override, by kernel code
// (see sbp_set_plan_override): code, tile, stages (0 = the tile's default),
// reduction groups, epilogue.
struct Instance {
    int code, bm, bn, ns, kg, epi, bk = 64;
};
constexpr int E_DIRECT = 0, E_STAGED = 1, E_ROWQ = 2;   // = sbpk::EPI_*
const Instance kInstances[] = {
    {1, 256, 256, 0, 1, E_DIRECT}, {1, 256, 192, 0, 1, E_DIRECT},
    {1, 256, 128, 0, 1, E_DIRECT}, {1, 128, 256, 0, 1, E_DIRECT},
    {1, 128, 128, 0, 1, E_DIRECT}, {1, 128, 64, 0, 1, E_DIRECT},  {1, 64, 128, 0, 1, E_DIRECT},
    {1, 64, 64, 0, 1, E_DIRECT},   {4, 128, 128, 2, 1, E_DIRECT}, {5, 256, 128, 0, 2, E_STAGED},
    {5, 128, 256, 0, 2, E_STAGED}, {5, 128, 128, 0, 2, E_STAGED}, {6, 256, 256, 0, 1, E_ROWQ},
    {6, 128, 128, 2, 1, E_ROWQ},   {7, 256, 128, 0, 2, E_ROWQ},   {7, 128, 256, 0, 2, E_ROWQ},
    {7, 128, 128, 0, 2, E_ROWQ},   {8, 256, 256, 5, 1, E_DIRECT, 32},
    {9, 256, 128, 6, 2, E_STAGED, 32}, {9, 128, 256, 6, 2, E_STAGED, 32},
    {9, 128, 128, 8, 2, E_STAGED, 32}, {10, 128, 128, 2, 2, E_STAGED},
    {4, 128, 64, 2, 1, E_DIRECT},      {4, 64, 128, 2, 1, E_DIRECT},
    {4, 64, 64, 2, 1, E_DIRECT},       {11, 128, 64, 6, 1, E_DIRECT},
    {11, 64, 128, 6, 1, E_DIRECT},     {11, 64, 64, 8, 1, E_DIRECT},
    {5, 128, 64, 0, 2, E_STAGED},      {5, 64, 128, 0, 2, E_STAGED},
    {5, 64, 64, 0, 2, E_STAGED},       {7, 128, 64, 0, 2, E_ROWQ},
    {7, 64, 128, 0, 2, E_ROWQ},        {7, 64, 64, 0, 2, E_ROWQ},
    {12, 128, 128, 2, 2, E_STAGED, 128}, {12, 128, 64, 3, 2, E_STAGED, 128},
    {12, 64, 128, 3, 2, E_STAGED, 128},  {12, 64, 64, 4, 2, E_STAGED, 128},
    {13, 128, 128, 2, 2, E_ROWQ, 128},   {13, 128, 64, 3, 2, E_ROWQ, 128},
    {13, 64, 128, 3, 2, E_ROWQ, 128},    {13, 64, 64, 4, 2, E_ROWQ, 128},
};

// Plans measured fastest on MI355X for the local products of the paper's
// workloads (generated by paper_2301_06813_amd/tune.py): orientation, fp32
// output, m, n, k, pipelined-kernel eligibility -> tile, kernel code, splits,
// persistent workgroups per CU. Other products use the model below.
struct Tuned {
    int orient, out_f32;
    int64_t m, n, k;
    int dma, bm, bn, code, splits, occ;
    int64_t nbatch = 1;   // batched products (attention core): batches x heads
};
const Tuned kTuned[] = {
#include "tuned_plans.inc"
    {-1, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0}   // end marker
};

// Backward pairs measured fastest as one grouped launch: backward-data
// product (m, n, k, fp32 output), backward-weight product (same) -> shared
// tile and kernel code, splits of each product. Pairs not listed run as two
// launches (of their tuned or modelled plans).
struct TunedBwd {
    int64_t md, nd, kd;
    int fd;
    int64_t mw, nw, kw;
    int fw, bm, bn, code, sd, sw;
};
const TunedBwd kTunedBwd[] = {
#include "tuned_bwd_plans.inc"
    {-1, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0}   // end marker
};

// Instances with a shifted-index-space form (gemm_bf16_launch.h
// SBP_DMA_SHIFT_INSTANCES): tile, reduction step, stages (0: the tile's
// default), reduction groups, epilogue.
struct ShiftInstance {
    int bm, bn, bk, ns, kg, epi;
};
const ShiftInstance kShiftInstances[] = {
    {64, 64, 64, 0, 1, E_DIRECT},     {128, 128, 64, 2, 1, E_DIRECT},
    {64, 64, 128, 4, 2, E_STAGED},    {128, 64, 128, 3, 2, E_STAGED},
    {64, 128, 128, 3, 2, E_STAGED},   {128, 128, 128, 2, 2, E_STAGED},
};

bool shift_capable(int bm, int bn, int bk, int ns, int kg, int epi) {
    for (const ShiftInstance &i : kShiftInstances)
        if (i.bm == bm && i.bn == bn && i.bk == bk && i.ns == ns && i.kg == kg && i.epi == epi)
            return true;
    return false;
}
bool shift_capable(const Plan &p) { return shift_capable(p.bm, p.bn, p.bk, p.ns, p.kg, p.epi); }

const Instance *find_instance(int code, int bm, int bn) {
    for (const Instance &i : kInstances)
        if (i.code == code && i.bm == bm && i.bn == bn) return &i;
    return nullptr;
}

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

// Workspace floats available to a product: the caller's, capped at the
// preferred size so that plans do not depend on workspaces beyond it.
double ws_budget(const Gemm &g) {
    return (double)std::min(g.ws_floats, WS_FLOATS_PREFERRED);
}

bool fits_ws(const Gemm &g, int splits) {
    if (splits == 1) return true;
    if (g.nbatch() > 1) return false;   // batched launches never split
    return (double)splits * (double)g.m * (double)partial_ld(g.n) <= ws_budget(g);
}

// Work items of one product under (tile, splits): count, time per item, and
// the cost of its split reduction (0 without splits).
struct Est {
    double wgs, wg_time, extra;
};

Est estimate(const Gemm &g, const TileClass &t, int splits, int per) {
    const int64_t tiles = ((g.m + t.bm - 1) / t.bm) * ((g.n + t.bn - 1) / t.bn) * g.nbatch();
    const double step_bytes = (t.bm + t.bn) * 128.0;
    const double step = std::max(2.0 * t.bm * t.bn * 64.0 / (kCuPeak * 0.9),
                                 step_bytes * t.occ / (kCuL2 * t.eff));
    const double out_bytes = (splits > 1 || g.out_dtype == DT_F32) ? 4.0 : 2.0;
    // output stores overlap other workgroups' loads when two share a CU
    const double epi = t.bm * t.bn * out_bytes / kCuL2 / t.occ;
    Est e{(double)tiles * splits, per * step + epi + kRoundLatency / t.occ, 0.0};
    if (splits > 1) {
        const double red = (splits * 4.0 + ((g.out_dtype == DT_F32) ? 4.0 : 2.0)) * g.m * g.n;
        e.extra = red / kHbm + kLaunch;
    }
    return e;
}

double algo_bytes(const Gemm &g) {
    return (2.0 * (g.m * g.k + g.k * g.n) + ((g.out_dtype == DT_F32) ? 4.0 : 2.0) * g.m * g.n) *
           (double)g.nbatch();
}

double model_time(const Gemm &g, const TileClass &t, int splits, int per) {
    const Est e = estimate(g, t, splits, per);
    const double rounds = std::ceil(e.wgs / (kCUs * t.occ));
    return std::max(rounds * e.wg_time, algo_bytes(g) / kHbm) + e.extra;
}

// Two products sharing one grid: the longer items are dispatched first and
// the shorter fill in behind them.
double model_pair(const Gemm &gd, const Gemm &gw, const TileClass &t, int sd, int pd, int sw,
                  int pw) {
    const Est a = estimate(gd, t, sd, pd), b = estimate(gw, t, sw, pw);
    const Est &lo = (a.wg_time >= b.wg_time) ? a : b;
    const Est &sh = (a.wg_time >= b.wg_time) ? b : a;
    const double slots = kCUs * t.occ;
    const double total = lo.wgs * lo.wg_time + sh.wgs * sh.wg_time;
    const double mk = std::max(std::ceil(lo.wgs / slots) * lo.wg_time, total / slots + sh.wg_time);
    return std::max(mk, (algo_bytes(gd) + algo_bytes(gw)) / kHbm) + a.extra + b.extra;
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

bool override_supported(int bm, int bn, int kernel) {
    if (kernel == 0 || kernel == 2) return tile_supported(bm, bn, true);
    return find_instance(kernel, bm, bn) != nullptr;
}

int kernel_code(const Plan &p) {
    if (!p.dma) return 2;
    for (const Instance &i : kInstances)
        if (i.bm == p.bm && i.bn == p.bn && i.kg == p.kg && i.epi == p.epi && i.bk == p.bk &&
            (i.ns == p.ns || (i.ns == 0 && p.ns == 0)))
            return i.code;
    return 1;
}

void set_override_occ(int occ) { ov_occ = occ < 0 ? 0 : occ; }

void set_override_orients(int mask) { ov_orients = mask & 7; }

void set_bwd_override(int mode, int splits_w) {
    ov_bwd_mode = mode;
    ov_bwd_splits_w = splits_w < 1 ? 1 : splits_w;
}

void set_override(int bm, int bn, int splits, int kernel) {
    ov_bm = bm;
    ov_bn = bn;
    ov_splits = std::max(1, splits);
    ov_kernel = kernel;
}

static bool kmajor_a(int orient) { return orient != OR_BWD_WEIGHT; }
static bool kmajor_b(int orient) { return orient == OR_BWD_DATA; }

int block_offset(const void *p) {
    return (int)((reinterpret_cast<uintptr_t>(p) >> 1) & 7);
}

bool dma_eligible(const Gemm &g) {
    if (g.in_dtype != DT_BF16) return false;
    // every row of an operand starts at the same offset within a 16-byte block
    if (g.lda % 8 || g.ldb % 8) return false;
    if ((reinterpret_cast<uintptr_t>(g.A) | reinterpret_cast<uintptr_t>(g.B)) & 1) return false;
    const int oa = block_offset(g.A), ob = block_offset(g.B);
    if (g.nbatch() > 1) {
        // batched: every item's operand bases 16-byte aligned, ends on chunks
        if (oa || ob) return false;
        if (g.sa_b % 8 || g.sa_h % 8 || g.sb_b % 8 || g.sb_h % 8) return false;
        if ((kmajor_a(g.orient) ? g.k : g.m) % 8 || (kmajor_b(g.orient) ? g.k : g.n) % 8)
            return false;
    }
    // An offset along m or n shifts the output index; along the reduction
    // both operands must be k-major with the same offset (a k-major A with
    // an n-major B needs an aligned A).
    if (g.orient == OR_FWD && oa) return false;
    if (g.orient == OR_BWD_DATA && oa != ob) return false;
    // per-tile buffer offsets stay below 2^31 bytes
    return g.lda <= (int64_t(1) << 21) && g.ldb <= (int64_t(1) << 21);
}

int dma_mode(const Gemm &g) {
    if (!dma_eligible(g)) return 0;
    const int64_t a_contig = kmajor_a(g.orient) ? g.k : g.m;
    const int64_t b_contig = kmajor_b(g.orient) ? g.k : g.n;
    const bool aligned = block_offset(g.A) == 0 && block_offset(g.B) == 0 && a_contig % 8 == 0 &&
                         b_contig % 8 == 0;
    return aligned ? 1 : 2;
}

static Plan plan_uncached(const Gemm &g);

// Tuned entry of product g under pipelined-kernel mode `mode` (nullptr if none).
static const Tuned *tuned_for(const Gemm &g, int mode) {
    if (g.in_dtype != DT_BF16) return nullptr;
    const int f32 = g.out_dtype == DT_F32 ? 1 : 0;
    for (const Tuned &t : kTuned) {
        if (t.orient < 0) break;
        if (t.orient == g.orient && t.out_f32 == f32 && t.m == g.m && t.n == g.n && t.k == g.k &&
            t.dma == mode && t.nbatch == g.nbatch())
            return &t;
    }
    return nullptr;
}

int device_cus() {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cached[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

namespace {
struct Key {
    int64_t v[11];
    bool operator==(const Key &o) const {
        for (int i = 0; i < 11; ++i)
            if (v[i] != o.v[i]) return false;
        return true;
    }
};
struct KeyHash {
    size_t operator()(const Key &k) const {
        size_t h = 1469598103934665603ull;
        for (int i = 0; i < 11; ++i) h = (h ^ (size_t)k.v[i]) * 1099511628211ull;
        return h;
    }
};
Key key_of(const Gemm &g, int mode) {
    return Key{{g.orient, g.in_dtype, g.out_dtype, g.m, g.n, g.k, mode,
                ov_bm * 1000 + ov_bn, ((ov_splits * 100 + ov_kernel) * 100 + ov_occ) * 8 + ov_orients,
                g.nbatch(), (int64_t)std::min(g.ws_floats, WS_FLOATS_PREFERRED)}};
}
thread_local std::unordered_map<Key, Plan, KeyHash> plan_cache;
}  // namespace

Plan plan_bf16(const Gemm &g) {
    const Key k = key_of(g, dma_mode(g));
    auto it = plan_cache.find(k);
    if (it != plan_cache.end()) return it->second;
    const Plan p = plan_uncached(g);
    if (plan_cache.size() > 4096) plan_cache.clear();
    plan_cache.emplace(k, p);
    return p;
}

// Grouped plan of both products on instance `in` (tile bm x bn) with the
// given splits; false if it does not fit the workspace.
static bool grouped_plan(const Gemm &gd, const Gemm &gw, const Instance *in, int bm, int bn,
                         int sd, int sw, Plan *pd, Plan *pw) {
    const bool sh = dma_mode(gd) == 2 || dma_mode(gw) == 2;
    if (sh && !shift_capable(bm, bn, in->bk, in->ns, in->kg, in->epi)) return false;
    for (int w = 0; w < 2; ++w) {
        const Gemm &g = w ? gw : gd;
        Plan &p = w ? *pw : *pd;
        p = Plan{bm, bn, 1, 1, true, in->ns, in->kg, in->epi, 0, in->bk};
        p.shift = sh;
        split_of(kblocks(g.k), w ? sw : sd, &p.splits, &p.kblk_per_split);
    }
    return (double)plan_ws_floats(gd, *pd) + (double)plan_ws_floats(gw, *pw) <= ws_budget(gd);
}

size_t plan_ws_floats(const Gemm &g, const Plan &p) {
    return p.splits > 1 ? (size_t)p.splits * (size_t)g.m * (size_t)partial_ld(g.n) : 0;
}

bool plan_bf16_bwd(const Gemm &gd, const Gemm &gw, Plan *pd, Plan *pw) {
    if (gd.nbatch() > 1 || gw.nbatch() > 1) {   // batched products run one by one
        *pd = plan_bf16(gd);
        *pw = plan_bf16(gw);
        return false;
    }
    *pd = plan_bf16(gd);
    *pw = plan_bf16(gw);
    if (ov_bwd_mode == 1) return false;
    if (ov_bm != 0 && ov_kernel == 2) return false;
    if (!dma_eligible(gd) || !dma_eligible(gw)) return false;
    if (ov_bm != 0 && ov_bwd_mode == 2) {
        // tuning: grouped on the override's instance, backward-data splits from
        // the plan override, backward-weight splits from the backward override
        const Instance *in = find_instance(ov_kernel == 0 ? 1 : ov_kernel, ov_bm, ov_bn);
        return in && grouped_plan(gd, gw, in, ov_bm, ov_bn, ov_splits, ov_bwd_splits_w, pd, pw);
    }
    if (ov_bm == 0) {
        const int fd = gd.out_dtype == DT_F32, fw = gw.out_dtype == DT_F32;
        for (const TunedBwd &t : kTunedBwd) {
            if (t.md < 0) break;
            if (t.md == gd.m && t.nd == gd.n && t.kd == gd.k && t.fd == fd && t.mw == gw.m &&
                t.nw == gw.n && t.kw == gw.k && t.fw == fw) {
                const Instance *in = find_instance(t.code, t.bm, t.bn);
                if (in && grouped_plan(gd, gw, in, t.bm, t.bn, t.sd, t.sw, pd, pw)) return true;
                *pd = plan_bf16(gd);
                *pw = plan_bf16(gw);
                break;
            }
        }
        // measured plans of both products: they run as measured, one after the other
        if (tuned_for(gd, dma_mode(gd)) && tuned_for(gw, dma_mode(gw))) return false;
    }
    const bool sh = dma_mode(gd) == 2 || dma_mode(gw) == 2;
    if (ov_bm != 0) {
        // an override fixes the tile (and the splits of both products)
        if (!pd->dma || !pw->dma) return false;
        pw->bm = pd->bm;
        pw->bn = pd->bn;
        pw->ns = pd->ns;
        pw->kg = pd->kg;
        pw->epi = pd->epi;
        pw->bk = pd->bk;
        if (sh && !shift_capable(*pd)) return false;
        pd->shift = pw->shift = sh;
        pd->occ = pw->occ = 0;   // the grouped launch runs one workgroup per item
        return (double)plan_ws_floats(gd, *pd) + (double)plan_ws_floats(gw, *pw) <=
               ws_budget(gd);
    }
    const TileClass *sep_d = nullptr, *sep_w = nullptr;
    for (const TileClass &t : kDma) {
        if (t.bm == pd->bm && t.bn == pd->bn && t.ns == pd->ns && t.kg == pd->kg &&
            t.epi == pd->epi && t.bk == pd->bk)
            sep_d = &t;
        if (t.bm == pw->bm && t.bn == pw->bn && t.ns == pw->ns && t.kg == pw->kg &&
            t.epi == pw->epi && t.bk == pw->bk)
            sep_w = &t;
    }
    if (!sep_d || !sep_w) return false;
    double best = model_time(gd, *sep_d, pd->splits, pd->kblk_per_split) +
                  model_time(gw, *sep_w, pw->splits, pw->kblk_per_split);
    bool grouped = false;
    const int kd = kblocks(gd.k), kw = kblocks(gw.k);
    for (const TileClass &t : kDma) {
        if (sh && !shift_capable(t.bm, t.bn, t.bk, t.ns, t.kg, t.epi)) continue;
        int last_d = 0;
        for (int a = 1; a <= 16; ++a) {
            int sd, perd;
            split_of(kd, a, &sd, &perd);
            if (sd == last_d) continue;
            last_d = sd;
            if (sd > 1 && perd < 2) continue;
            int last_w = 0;
            for (int b = 1; b <= 16; ++b) {
                int sw, perw;
                split_of(kw, b, &sw, &perw);
                if (sw == last_w) continue;
                last_w = sw;
                if (sw > 1 && perw < 2) continue;
                const double wsz = (sd > 1 ? (double)sd * gd.m * gd.n : 0.0) +
                                   (sw > 1 ? (double)sw * gw.m * gw.n : 0.0);
                if (wsz > ws_budget(gd)) continue;
                const double tm = model_pair(gd, gw, t, sd, perd, sw, perw);
                if (tm < best * 0.97) {
                    best = tm;
                    grouped = true;
                    *pd = Plan{t.bm, t.bn, sd, perd, true, t.ns, t.kg, t.epi, 0, t.bk};
                    *pw = Plan{t.bm, t.bn, sw, perw, true, t.ns, t.kg, t.epi, 0, t.bk};
                    pd->shift = pw->shift = sh;
                }
            }
        }
    }
    return grouped;
}

static Plan plan_uncached(const Gemm &g) {
    const int kb_total = kblocks(g.k);
    const int mode = dma_mode(g);
    const bool dma = mode > 0;
    Plan best{128, 128, 1, std::max(1, kb_total), dma};
    if (mode == 2) {
        best.ns = 2;   // the two-stage 128 x 128 instance has a shifted form
        best.shift = true;
    }
    if (ov_bm != 0 && ((ov_orients >> g.orient) & 1)) {
        // kernel: 0 or 1 the tile's default pipelined instance (if eligible),
        // 2 generic, other codes the instance of kInstances (if eligible);
        // a product the pipelined kernel cannot read runs the generic kernel,
        // and so does one that needs the shifted form of an instance without
        // one
        bool use_dma = dma && ov_kernel != 2;
        const Instance *in = nullptr;
        if (use_dma) {
            in = find_instance(ov_kernel == 0 ? 1 : ov_kernel, ov_bm, ov_bn);
            if (!in) in = find_instance(1, ov_bm, ov_bn);
            if (mode == 2 && !shift_capable(ov_bm, ov_bn, in->bk, in->ns, in->kg, in->epi))
                use_dma = false;
        }
        Plan p{ov_bm, ov_bn, 1, 1, use_dma};
        if (use_dma) {
            p.ns = in->ns;
            p.kg = in->kg;
            p.epi = in->epi;
            p.bk = in->bk;
            p.occ = ov_occ;
            p.shift = mode == 2;
        } else if (!tile_supported(p.bm, p.bn, false)) {
            p.bn = 128;   // 256x256 only pipelined
        }
        split_of(kb_total, ov_splits, &p.splits, &p.kblk_per_split);
        while (p.splits > 1 && !fits_ws(g, p.splits))
            split_of(kb_total, p.splits - 1, &p.splits, &p.kblk_per_split);
        return p;
    }
    if (const Tuned *t = tuned_for(g, mode)) {
        Plan p{t->bm, t->bn, 1, 1, dma && t->code != 2};
        const Instance *in = p.dma ? find_instance(t->code, t->bm, t->bn) : nullptr;
        if (in && mode == 2 && !shift_capable(t->bm, t->bn, in->bk, in->ns, in->kg, in->epi))
            in = nullptr;
        if ((!p.dma && tile_supported(t->bm, t->bn, false)) || in) {
            if (in) {
                p.ns = in->ns;
                p.kg = in->kg;
                p.epi = in->epi;
                p.bk = in->bk;
                p.occ = t->occ;
                p.shift = mode == 2;
            }
            split_of(kb_total, t->splits, &p.splits, &p.kblk_per_split);
            if (fits_ws(g, p.splits)) return p;
        }
    }
    double best_t = 1e30;
    const TileClass *tiles_tab = dma ? kDma : kGeneric;
    const int ntiles = dma ? (int)(sizeof(kDma) / sizeof(kDma[0]))
                           : (int)(sizeof(kGeneric) / sizeof(kGeneric[0]));
    for (int ti = 0; ti < ntiles; ++ti) {
        const TileClass &t = tiles_tab[ti];
        if (mode == 2 && !shift_capable(t.bm, t.bn, t.bk, t.ns, t.kg, t.epi)) continue;
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
                best = Plan{t.bm, t.bn, splits, per, dma, t.ns, t.kg, t.epi, t.occ_persist, t.bk};
                best.shift = mode == 2;
            }
        }
    }
    return best;
}

}  // namespace sbpi
