// search.cpp -- the alpha-beta cost model (AutoDDL Sec. 3.1, Table 2) and
// the coordinate-descent strategy search (Sec. 4.4) over per-layer SBP
// signatures of a chain of linear layers. Host logic only.
#include <stdint.h>

#include <cmath>
#include <vector>

#include "../../include/sbp.h"

namespace {

bool valid_state(int32_t kind, int32_t axis) {
    if (kind == SBP_SPLIT) return axis == 0 || axis == 1;
    return (kind == SBP_BROADCAST || kind == SBP_PARTIAL) && axis == -1;
}

// The dual state of a gradient: S(i) -> S(i), B -> P, P -> B.
sbp_layout_t grad_of(sbp_layout_t l) {
    if (l.kind == SBP_BROADCAST) l.kind = SBP_PARTIAL;
    else if (l.kind == SBP_PARTIAL) l.kind = SBP_BROADCAST;
    return l;
}

// States of X and W for each signature id (SBP_SIG_*).
struct XW {
    int32_t xk, xa, wk, wa;
};
const XW kSigInputs[6] = {
    {SBP_SPLIT, 0, SBP_BROADCAST, -1},     // DP
    {SBP_BROADCAST, -1, SBP_SPLIT, 1},     // COL
    {SBP_SPLIT, 1, SBP_SPLIT, 0},          // KS
    {SBP_PARTIAL, -1, SBP_BROADCAST, -1},  // PB
    {SBP_BROADCAST, -1, SBP_PARTIAL, -1},  // BP
    {SBP_BROADCAST, -1, SBP_BROADCAST, -1} // BB
};

// X, Y and dW states of signature s on p devices (rank 0; states do not
// depend on the rank), from the library's own signature rule.
int sig_states(int s, int32_t p, sbp_layout_t *x, sbp_layout_t *y, sbp_layout_t *dw) {
    if (s < 0 || s > 5) return SBP_ERR_SIGNATURE;
    const XW &t = kSigInputs[s];
    *x = sbp_layout_t{t.xk, t.xa, p, 0};
    const sbp_layout_t w{t.wk, t.wa, p, 0};
    return sbp_signature(x, &w, y, nullptr, nullptr, dw);
}

int check_chain(const sbp_chain_t *n) {
    if (!n || !n->M || !n->K || !n->N) return SBP_ERR_NULL;
    if (n->layers < 1) return SBP_ERR_SHAPE;
    if (n->p < 1) return SBP_ERR_LAYOUT;
    if (!(n->alpha >= 0) || !(n->beta >= 0) || !(n->act_bytes >= 0) || !(n->grad_bytes >= 0))
        return SBP_ERR_SHAPE;
    for (int l = 0; l < n->layers; ++l) {
        if (n->M[l] < 0 || n->K[l] < 0 || n->N[l] < 0) return SBP_ERR_SHAPE;
        if (n->M[l] != n->M[0]) return SBP_ERR_SHAPE;
    }
    if (!valid_state(n->in_kind, n->in_axis) || !valid_state(n->out_kind, n->out_axis))
        return SBP_ERR_LAYOUT;
    return SBP_OK;
}

// Forward redistribution from -> to of `bytes`, plus the backward move of
// the gradient from grad(to) to grad(from).
double move_cost(const sbp_layout_t &from, const sbp_layout_t &to, double bytes, double a,
                 double b) {
    double f = 0, g = 0;
    sbp_boxing_cost(&from, &to, bytes, a, b, &f, nullptr);
    const sbp_layout_t gt = grad_of(to), gf = grad_of(from);
    sbp_boxing_cost(&gt, &gf, bytes, a, b, &g, nullptr);
    return f + g;
}

// Chain cost of signatures s (already validated chain).
int chain_cost(const sbp_chain_t *n, const int32_t *s, double *cost) {
    const double a = n->alpha, b = n->beta;
    sbp_layout_t prev{n->in_kind, n->in_axis, n->p, 0};
    double bytes = (double)n->M[0] * (double)n->K[0] * n->act_bytes;
    double total = 0;
    for (int l = 0; l < n->layers; ++l) {
        if (s[l] < 0 || s[l] > 5 || !((n->allowed >> s[l]) & 1u)) return SBP_ERR_SIGNATURE;
        sbp_layout_t x, y, dw;
        int rc = sig_states(s[l], n->p, &x, &y, &dw);
        if (rc) return rc;
        if (x.kind == SBP_PARTIAL) return SBP_ERR_SIGNATURE;   // P inputs end no chain link
        total += move_cost(prev, x, bytes, a, b);
        if (dw.kind == SBP_PARTIAL) {
            double ar = 0;
            sbp_collective_cost(SBP_COLL_ALLREDUCE, n->p,
                                (double)n->K[l] * (double)n->N[l] * n->grad_bytes, a, b, &ar);
            total += ar;
        }
        prev = y;
        bytes = (double)n->M[l] * (double)n->N[l] * n->act_bytes;
    }
    const sbp_layout_t last{n->out_kind, n->out_axis, n->p, 0};
    total += move_cost(prev, last, bytes, a, b);
    *cost = total;
    return SBP_OK;
}

// splitmix64 (S. Vigna): a counter-based 64-bit generator.
uint64_t splitmix64(uint64_t *state) {
    uint64_t z = (*state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

}  // namespace

extern "C" {

int sbp_collective_cost(int32_t coll, int32_t p, double n, double alpha, double beta,
                        double *cost) {
    if (!cost) return SBP_ERR_NULL;
    if (p < 1) return SBP_ERR_LAYOUT;
    if (!(n >= 0) || !(alpha >= 0) || !(beta >= 0)) return SBP_ERR_SHAPE;
    const double q = (double)p;
    switch (coll) {
        case SBP_COLL_ALLREDUCE: *cost = (2 * q - 1) * alpha + 2 * (q - 1) / q * n * beta; break;
        case SBP_COLL_ALLGATHER:
        case SBP_COLL_REDUCESCATTER: *cost = (q - 1) * alpha + (q - 1) / q * n * beta; break;
        case SBP_COLL_ALLTOALL: *cost = (q - 1) * alpha + n * beta; break;
        default: return SBP_ERR_LAYOUT;
    }
    return SBP_OK;
}

int sbp_boxing_cost(const sbp_layout_t *from, const sbp_layout_t *to, double bytes, double alpha,
                    double beta, double *cost, int32_t *coll_out) {
    if (!from || !to || !cost) return SBP_ERR_NULL;
    if (!valid_state(from->kind, from->axis) || !valid_state(to->kind, to->axis) ||
        from->p < 1 || from->p != to->p)
        return SBP_ERR_LAYOUT;
    if (!(bytes >= 0)) return SBP_ERR_SHAPE;
    int32_t coll = -1;
    double n = bytes;
    if (from->kind == SBP_SPLIT && to->kind == SBP_SPLIT && from->axis != to->axis) {
        coll = SBP_COLL_ALLTOALL;
        n = bytes / from->p;   // each device's output
    } else if (from->kind == SBP_SPLIT && to->kind == SBP_BROADCAST) {
        coll = SBP_COLL_ALLGATHER;
    } else if (from->kind == SBP_PARTIAL && to->kind == SBP_SPLIT) {
        coll = SBP_COLL_REDUCESCATTER;
    } else if (from->kind == SBP_PARTIAL && to->kind == SBP_BROADCAST) {
        coll = SBP_COLL_ALLREDUCE;
    }
    if (coll_out) *coll_out = coll;
    if (coll < 0) {
        *cost = 0;
        return SBP_OK;
    }
    return sbp_collective_cost(coll, from->p, n, alpha, beta, cost);
}

int sbp_chain_cost(const sbp_chain_t *net, const int32_t *sigs, double *cost) {
    if (!sigs || !cost) return SBP_ERR_NULL;
    int rc = check_chain(net);
    if (rc) return rc;
    return chain_cost(net, sigs, cost);
}

int sbp_search_strategy(const sbp_chain_t *net, int32_t restarts, uint64_t seed,
                        int32_t *sigs_out, double *cost_out, double *sweep_costs,
                        int32_t max_sweeps, int32_t *sweeps_out) {
    if (!sigs_out || !cost_out) return SBP_ERR_NULL;
    int rc = check_chain(net);
    if (rc) return rc;
    if (restarts < 1) return SBP_ERR_SHAPE;
    // signatures a chain can use: allowed, and not fed a Partial-sum input
    std::vector<int32_t> cand;
    for (int s = 0; s < 6; ++s) {
        if (!((net->allowed >> s) & 1u)) continue;
        sbp_layout_t x, y, dw;
        if (sig_states(s, net->p, &x, &y, &dw) == SBP_OK && x.kind != SBP_PARTIAL)
            cand.push_back(s);
    }
    if (cand.empty()) return SBP_ERR_SIGNATURE;
    const int L = net->layers;
    std::vector<int32_t> cur(L), best(L);
    double best_cost = INFINITY;
    uint64_t st = seed;
    int32_t nsweeps = 0;
    for (int run = 0; run < restarts; ++run) {
        for (int l = 0; l < L; ++l)
            cur[l] = run == 0 ? cand[0] : cand[splitmix64(&st) % cand.size()];
        double c = 0;
        if ((rc = chain_cost(net, cur.data(), &c))) return rc;
        if (sweep_costs && nsweeps < max_sweeps) sweep_costs[nsweeps] = c;   // the run's start
        ++nsweeps;
        for (bool changed = true; changed;) {
            changed = false;
            for (int l = 0; l < L; ++l) {
                const int32_t keep = cur[l];
                int32_t arg = keep;
                double argc = c;
                for (int32_t s : cand) {
                    if (s == keep) continue;
                    cur[l] = s;
                    double t = 0;
                    if ((rc = chain_cost(net, cur.data(), &t))) return rc;
                    if (t < argc) {
                        argc = t;
                        arg = s;
                    }
                }
                cur[l] = arg;
                if (arg != keep) {
                    c = argc;
                    changed = true;
                }
            }
            if (sweep_costs && nsweeps < max_sweeps) sweep_costs[nsweeps] = c;
            ++nsweeps;
        }
        if (c < best_cost) {
            best_cost = c;
            best = cur;
        }
    }
    for (int l = 0; l < L; ++l) sigs_out[l] = best[l];
    *cost_out = best_cost;
    if (sweeps_out) *sweeps_out = nsweeps;
    return SBP_OK;
}

}  // extern "C"
