// attn_api.cpp -- C ABI of the attention core under a head split
// (include/sbp.h, "attention core under a head split").
//
// Multi-head attention reduces to batched matrix products (AutoDDL Sec. 2).
// With the head dimension split over p devices every operand is Split on
// heads, so device r multiplies its own heads: one product per (batch, local
// head), launched as one batched GEMM on the same kernels as the linear
// layer. Validation happens on the host before any HIP call.
#include <stdint.h>

#include <algorithm>
#include <utility>

#include "../../include/sbp.h"
#include "api_internal.h"
#include "gemm.h"

namespace {

int64_t elsz(int32_t dtype) { return dtype == SBP_F32 ? 4 : 2; }

// Heads [h0, h0 + hr) of H on rank r of p (the balanced split rule).
void head_split(int64_t H, int32_t p, int32_t r, int64_t *h0, int64_t *hr) {
    const int64_t base = H / p, rem = H % p;
    *hr = base + (r < rem ? 1 : 0);
    *h0 = (int64_t)r * base + (r < rem ? r : rem);
}

int check_view4(const sbp_view4_t *v) {
    if (!v) return SBP_ERR_NULL;
    if (v->dtype != SBP_BF16 && v->dtype != SBP_F32) return SBP_ERR_DTYPE;
    const int64_t ext[4] = {v->batch, v->heads, v->rows, v->cols};
    for (int64_t e : ext)
        if (e < 0 || e > INT32_MAX) return SBP_ERR_SHAPE;
    if (v->ld < v->cols || v->ld < 1 || v->stride_b < 0 || v->stride_h < 0) return SBP_ERR_SHAPE;
    if (v->ld > (int64_t(1) << 40) || v->stride_b > (int64_t(1) << 40) ||
        v->stride_h > (int64_t(1) << 40))
        return SBP_ERR_SHAPE;
    const bool empty = v->batch == 0 || v->heads == 0 || v->rows == 0 || v->cols == 0;
    if (!empty) {
        if (!v->data) return SBP_ERR_NULL;
        if (reinterpret_cast<uintptr_t>(v->data) % elsz(v->dtype)) return SBP_ERR_ALIGN;
    }
    return SBP_OK;
}

// An input operand: its rank-r base and local head count.
struct In4 {
    const char *ptr;
    int64_t heads;
    const sbp_view4_t *v;
};

// [begin, end) bytes a 4-D view with `heads` heads starting at p touches.
std::pair<uintptr_t, uintptr_t> span4(const void *p, const sbp_view4_t *v, int64_t heads) {
    if (!p || v->batch == 0 || heads == 0 || v->rows == 0 || v->cols == 0) return {0, 0};
    const int64_t last = (v->batch - 1) * v->stride_b + (heads - 1) * v->stride_h +
                         (v->rows - 1) * v->ld + v->cols;
    const uintptr_t b = reinterpret_cast<uintptr_t>(p);
    return {b, b + (uintptr_t)(last * elsz(v->dtype))};
}

bool overlap(std::pair<uintptr_t, uintptr_t> a, std::pair<uintptr_t, uintptr_t> b) {
    if (a.first == a.second || b.first == b.second) return false;
    return a.first < b.second && b.first < a.second;
}

// No two elements of an output view share an address: with the outer
// dimensions sorted by stride, each stride covers the span of the smaller ones.
bool injective(const sbp_view4_t *v) {
    struct D {
        int64_t stride, n;
    } d[3] = {{v->ld, v->rows}, {v->stride_h, v->heads}, {v->stride_b, v->batch}};
    std::sort(d, d + 3, [](const D &a, const D &b) { return a.stride < b.stride; });
    int64_t span = v->cols;   // elements covered by the dimensions below
    for (const D &x : d) {
        if (x.n <= 1) continue;
        if (x.stride < span) return false;
        span = x.stride * (x.n - 1) + span;
    }
    return true;
}

// The call's head split: H (when some input is GLOBAL) and rank r's heads.
int resolve_heads(const sbp_view4_t *const *ins, int nin, int32_t p, int32_t r, int64_t *hr,
                  In4 *out) {
    if (p < 1 || r < 0 || r >= p) return SBP_ERR_LAYOUT;
    int64_t H = -1, local = -1;
    for (int i = 0; i < nin; ++i) {
        const sbp_view4_t *v = ins[i];
        if (v->scope == SBP_GLOBAL) {
            if (H >= 0 && v->heads != H) return SBP_ERR_SHAPE;
            H = v->heads;
        } else if (v->scope == SBP_LOCAL) {
            if (local >= 0 && v->heads != local) return SBP_ERR_SHAPE;
            local = v->heads;
        } else {
            return SBP_ERR_SHAPE;
        }
    }
    int64_t h0 = 0;
    if (H >= 0) {
        head_split(H, p, r, &h0, hr);
        if (local >= 0 && local != *hr) return SBP_ERR_SHAPE;
    } else {
        *hr = local;
    }
    for (int i = 0; i < nin; ++i) {
        const sbp_view4_t *v = ins[i];
        out[i].v = v;
        out[i].heads = *hr;
        out[i].ptr = static_cast<const char *>(v->data);
        if (v->scope == SBP_GLOBAL && *hr > 0 && out[i].ptr)
            out[i].ptr += h0 * v->stride_h * elsz(v->dtype);
    }
    return SBP_OK;
}

// Output checks: shape [batch][hr][rows][cols], dtype, no self-overlap, no
// overlap with the inputs' spans.
int check_out4(const sbp_view4_t *o, int64_t batch, int64_t hr, int64_t rows, int64_t cols,
               const In4 *ins, int nin) {
    int rc = check_view4(o);
    if (rc) return rc;
    if (o->batch != batch || o->heads != hr || o->rows != rows || o->cols != cols)
        return SBP_ERR_SHAPE;
    if (o->scope == SBP_ACCUMULATE && o->dtype != SBP_F32) return SBP_ERR_DTYPE;
    if (!injective(o)) return SBP_ERR_SHAPE;
    const auto os = span4(o->data, o, hr);
    for (int i = 0; i < nin; ++i)
        if (overlap(os, span4(ins[i].ptr, ins[i].v, ins[i].heads))) return SBP_ERR_ALIAS;
    return SBP_OK;
}

// Work items of a batched product must fit a 31-bit index (64 x 64 tiles).
bool items_fit(int64_t m, int64_t n, int64_t nb) {
    const double items = (double)((m + 63) / 64) * (double)((n + 63) / 64) * (double)nb;
    return items < 2147483647.0;
}

// One batched product: per (batch, local head), C = A op B with the given
// orientation; A, B are inputs, o the output view.
sbpi::Gemm batched(int orient, const In4 &a, const In4 &b, const sbp_view4_t *o, int64_t m,
                   int64_t n, int64_t k) {
    sbpi::Gemm g{orient, SBP_BF16, o->dtype, a.ptr, a.v->ld, b.ptr, b.v->ld, o->data, o->ld,
                 m, n, k};
    g.accumulate = o->scope == SBP_ACCUMULATE;
    g.batches = o->batch;
    g.heads = o->heads;
    g.sa_b = a.v->stride_b;
    g.sa_h = a.v->stride_h;
    g.sb_b = b.v->stride_b;
    g.sb_h = b.v->stride_h;
    g.sc_b = o->stride_b;
    g.sc_h = o->stride_h;
    return g;
}

int inputs_ok(const sbp_view4_t *const *ins, int nin) {
    for (int i = 0; i < nin; ++i) {
        int rc = check_view4(ins[i]);
        if (rc) return rc;
        if (ins[i]->dtype != SBP_BF16) return SBP_ERR_DTYPE;
        if (ins[i]->batch != ins[0]->batch) return SBP_ERR_SHAPE;
    }
    return SBP_OK;
}

int launch(const sbpi::Gemm &g, hipStream_t s) {
    if (g.nbatch() == 0) return SBP_OK;
    return sbpa::run_gemm(g, s);
}

}  // namespace

extern "C" {

int sbp_attn_scores(const sbp_view4_t *Q, const sbp_view4_t *K, sbp_view4_t *S, int32_t p,
                    int32_t r, hipStream_t stream) {
    if (!Q || !K || !S) return SBP_ERR_NULL;
    const sbp_view4_t *ins[2] = {Q, K};
    int rc = inputs_ok(ins, 2);
    if (rc) return rc;
    In4 in[2];
    int64_t hr;
    if ((rc = resolve_heads(ins, 2, p, r, &hr, in))) return rc;
    if (Q->cols != K->cols) return SBP_ERR_SHAPE;
    if ((rc = check_out4(S, Q->batch, hr, Q->rows, K->rows, in, 2))) return rc;
    if (!items_fit(Q->rows, K->rows, Q->batch * hr)) return SBP_ERR_SHAPE;
    // S = Q K^T: both operands k-major (the backward-data orientation)
    return launch(batched(sbpi::OR_BWD_DATA, in[0], in[1], S, Q->rows, K->rows, Q->cols), stream);
}

int sbp_attn_context(const sbp_view4_t *P, const sbp_view4_t *V, sbp_view4_t *O, int32_t p,
                     int32_t r, hipStream_t stream) {
    if (!P || !V || !O) return SBP_ERR_NULL;
    const sbp_view4_t *ins[2] = {P, V};
    int rc = inputs_ok(ins, 2);
    if (rc) return rc;
    In4 in[2];
    int64_t hr;
    if ((rc = resolve_heads(ins, 2, p, r, &hr, in))) return rc;
    if (P->cols != V->rows) return SBP_ERR_SHAPE;
    if ((rc = check_out4(O, P->batch, hr, P->rows, V->cols, in, 2))) return rc;
    if (!items_fit(P->rows, V->cols, P->batch * hr)) return SBP_ERR_SHAPE;
    // O = P V: A k-major, B n-major (the forward orientation)
    return launch(batched(sbpi::OR_FWD, in[0], in[1], O, P->rows, V->cols, P->cols), stream);
}

int sbp_attn_scores_bwd(const sbp_view4_t *dS, const sbp_view4_t *Q, const sbp_view4_t *K,
                        sbp_view4_t *dQ, sbp_view4_t *dK, int32_t p, int32_t r,
                        hipStream_t stream) {
    if (!dS || !Q || !K || !dQ || !dK) return SBP_ERR_NULL;
    const sbp_view4_t *ins[3] = {dS, Q, K};
    int rc = inputs_ok(ins, 3);
    if (rc) return rc;
    In4 in[3];
    int64_t hr;
    if ((rc = resolve_heads(ins, 3, p, r, &hr, in))) return rc;
    // dS: [Sq][Sk], Q: [Sq][D], K: [Sk][D]
    if (dS->rows != Q->rows || dS->cols != K->rows || Q->cols != K->cols) return SBP_ERR_SHAPE;
    if ((rc = check_out4(dQ, dS->batch, hr, Q->rows, Q->cols, in, 3))) return rc;
    if ((rc = check_out4(dK, dS->batch, hr, K->rows, K->cols, in, 3))) return rc;
    if (overlap(span4(dQ->data, dQ, hr), span4(dK->data, dK, hr))) return SBP_ERR_ALIAS;
    if (!items_fit(Q->rows, Q->cols, dS->batch * hr) ||
        !items_fit(K->rows, K->cols, dS->batch * hr))
        return SBP_ERR_SHAPE;
    // dQ = dS K (forward orientation); dK = dS^T Q (backward-weight orientation)
    if ((rc = launch(batched(sbpi::OR_FWD, in[0], in[2], dQ, Q->rows, Q->cols, K->rows), stream)))
        return rc;
    return launch(batched(sbpi::OR_BWD_WEIGHT, in[0], in[1], dK, K->rows, K->cols, Q->rows),
                  stream);
}

int sbp_attn_context_bwd(const sbp_view4_t *dO, const sbp_view4_t *P, const sbp_view4_t *V,
                         sbp_view4_t *dP, sbp_view4_t *dV, int32_t p, int32_t r,
                         hipStream_t stream) {
    if (!dO || !P || !V || !dP || !dV) return SBP_ERR_NULL;
    const sbp_view4_t *ins[3] = {dO, P, V};
    int rc = inputs_ok(ins, 3);
    if (rc) return rc;
    In4 in[3];
    int64_t hr;
    if ((rc = resolve_heads(ins, 3, p, r, &hr, in))) return rc;
    // dO: [Sq][D], P: [Sq][Sk], V: [Sk][D]
    if (dO->rows != P->rows || P->cols != V->rows || dO->cols != V->cols) return SBP_ERR_SHAPE;
    if ((rc = check_out4(dP, dO->batch, hr, P->rows, P->cols, in, 3))) return rc;
    if ((rc = check_out4(dV, dO->batch, hr, V->rows, V->cols, in, 3))) return rc;
    if (overlap(span4(dP->data, dP, hr), span4(dV->data, dV, hr))) return SBP_ERR_ALIAS;
    if (!items_fit(P->rows, P->cols, dO->batch * hr) ||
        !items_fit(V->rows, V->cols, dO->batch * hr))
        return SBP_ERR_SHAPE;
    // dP = dO V^T (backward-data orientation); dV = P^T dO (backward-weight)
    if ((rc = launch(batched(sbpi::OR_BWD_DATA, in[0], in[2], dP, P->rows, P->cols, dO->cols),
                     stream)))
        return rc;
    return launch(batched(sbpi::OR_BWD_WEIGHT, in[1], in[0], dV, V->rows, V->cols, P->rows),
                  stream);
}

}  // extern "C"
