// sbp_api.cpp -- the C ABI declared in include/sbp.h.
//
// Host-side SBP logic (AutoDDL Sec. 4.1 states, Sec. 4.2 SBP matmul rule,
// Sec. 4.3 gradient states): layout checks, shard indexing, signature
// resolution, argument validation, then one kernel launch on the caller's
// stream. Every validation happens before the first HIP call. 1-D layouts
// (one state on a mesh of p devices) and nd layouts (one state per mesh
// axis) share the validation and launch code below; an nd signature is one
// 1-D factor per mesh axis.
#include <stdint.h>
#include <string.h>

#include <utility>

#include "../../include/sbp.h"
#include "api_internal.h"
#include "gemm.h"

namespace {

thread_local int g_last_hip = 0;

enum Sig { SIG_DP = 0, SIG_COL = 1, SIG_KS = 2, SIG_PB = 3, SIG_BP = 4, SIG_BB = 5, SIG_NONE = -1 };

bool is_split(const sbp_layout_t *l, int axis) {
    return l->kind == SBP_SPLIT && l->axis == axis;
}
bool is_bcast(const sbp_layout_t *l) { return l->kind == SBP_BROADCAST; }
bool is_partial(const sbp_layout_t *l) { return l->kind == SBP_PARTIAL; }

int check_layout(const sbp_layout_t *l) {
    if (!l) return SBP_ERR_NULL;
    if (l->p < 1 || l->r < 0 || l->r >= l->p) return SBP_ERR_LAYOUT;
    if (l->kind == SBP_SPLIT) {
        if (l->axis != 0 && l->axis != 1) return SBP_ERR_LAYOUT;
    } else if (l->kind == SBP_BROADCAST || l->kind == SBP_PARTIAL) {
        if (l->axis != -1) return SBP_ERR_LAYOUT;
    } else {
        return SBP_ERR_LAYOUT;
    }
    return SBP_OK;
}

int check_pair(const sbp_layout_t *a, const sbp_layout_t *b) {
    int rc = check_layout(a);
    if (rc) return rc;
    rc = check_layout(b);
    if (rc) return rc;
    if (a->p != b->p || a->r != b->r) return SBP_ERR_LAYOUT;
    return SBP_OK;
}

// Forward rule (Sec. 4.2, 1-D factors): (S0,B)->S0, (B,S1)->S1, (S1,S0)->P;
// and, by linearity of the product in each operand, (P,B)->P, (B,P)->P and
// (B,B)->B.
Sig sig_from_xw(const sbp_layout_t *x, const sbp_layout_t *w) {
    if (is_split(x, 0) && is_bcast(w)) return SIG_DP;
    if (is_bcast(x) && is_split(w, 1)) return SIG_COL;
    if (is_split(x, 1) && is_split(w, 0)) return SIG_KS;
    if (is_partial(x) && is_bcast(w)) return SIG_PB;
    if (is_bcast(x) && is_partial(w)) return SIG_BP;
    if (is_bcast(x) && is_bcast(w)) return SIG_BB;
    return SIG_NONE;
}
// Backward-data inputs: dY takes Y's dual state (S stays S, P becomes B, B
// becomes P).
Sig sig_from_dyw(const sbp_layout_t *dy, const sbp_layout_t *w) {
    if (is_split(dy, 0) && is_bcast(w)) return SIG_DP;
    if (is_split(dy, 1) && is_split(w, 1)) return SIG_COL;
    if (is_bcast(dy) && is_split(w, 0)) return SIG_KS;
    if (is_bcast(dy) && is_bcast(w)) return SIG_PB;
    if (is_bcast(dy) && is_partial(w)) return SIG_BP;
    if (is_partial(dy) && is_bcast(w)) return SIG_BB;
    return SIG_NONE;
}
Sig sig_from_xdy(const sbp_layout_t *x, const sbp_layout_t *dy) {
    if (is_split(x, 0) && is_split(dy, 0)) return SIG_DP;
    if (is_bcast(x) && is_split(dy, 1)) return SIG_COL;
    if (is_split(x, 1) && is_bcast(dy)) return SIG_KS;
    if (is_partial(x) && is_bcast(dy)) return SIG_PB;
    if (is_bcast(x) && is_bcast(dy)) return SIG_BP;
    if (is_bcast(x) && is_partial(dy)) return SIG_BB;
    return SIG_NONE;
}

sbp_layout_t mk(int32_t kind, int32_t axis, const sbp_layout_t *like) {
    sbp_layout_t l;
    l.kind = kind;
    l.axis = axis;
    l.p = like->p;
    l.r = like->r;
    return l;
}

// States of Y, dY, dX, dW for a signature (gradient of S(i) is S(i), of B is
// P, of P is B; Sec. 4.3 states the broadcast-weight case).
void states_of(Sig s, const sbp_layout_t *like, sbp_layout_t out[4]) {
    switch (s) {
        case SIG_DP:
            out[0] = mk(SBP_SPLIT, 0, like);
            out[1] = mk(SBP_SPLIT, 0, like);
            out[2] = mk(SBP_SPLIT, 0, like);
            out[3] = mk(SBP_PARTIAL, -1, like);
            break;
        case SIG_COL:
            out[0] = mk(SBP_SPLIT, 1, like);
            out[1] = mk(SBP_SPLIT, 1, like);
            out[2] = mk(SBP_PARTIAL, -1, like);
            out[3] = mk(SBP_SPLIT, 1, like);
            break;
        case SIG_PB:   // X P, W B: Y P, dY B, dX B, dW P
            out[0] = mk(SBP_PARTIAL, -1, like);
            out[1] = mk(SBP_BROADCAST, -1, like);
            out[2] = mk(SBP_BROADCAST, -1, like);
            out[3] = mk(SBP_PARTIAL, -1, like);
            break;
        case SIG_BP:   // X B, W P: Y P, dY B, dX P, dW B
            out[0] = mk(SBP_PARTIAL, -1, like);
            out[1] = mk(SBP_BROADCAST, -1, like);
            out[2] = mk(SBP_PARTIAL, -1, like);
            out[3] = mk(SBP_BROADCAST, -1, like);
            break;
        case SIG_BB:   // X B, W B: Y B, dY P, dX P, dW P
            out[0] = mk(SBP_BROADCAST, -1, like);
            out[1] = mk(SBP_PARTIAL, -1, like);
            out[2] = mk(SBP_PARTIAL, -1, like);
            out[3] = mk(SBP_PARTIAL, -1, like);
            break;
        default:
            out[0] = mk(SBP_PARTIAL, -1, like);
            out[1] = mk(SBP_BROADCAST, -1, like);
            out[2] = mk(SBP_SPLIT, 1, like);
            out[3] = mk(SBP_SPLIT, 0, like);
            break;
    }
}

size_t elsize(int32_t dtype) { return dtype == SBP_F32 ? 4 : 2; }

// A validated local (rank-r) operand.
struct Local {
    const char *ptr;
    int64_t rows, cols, ld;
    int32_t dtype;
    bool global;
    int64_t grows, gcols;   // global extent when the view was global
};

int check_view_common(const sbp_view_t *v) {
    if (!v) return SBP_ERR_NULL;
    if (v->dtype != SBP_BF16 && v->dtype != SBP_F32) return SBP_ERR_DTYPE;
    if (v->rows < 0 || v->cols < 0 || v->rows > INT32_MAX || v->cols > INT32_MAX)
        return SBP_ERR_SHAPE;
    if (v->ld < v->cols || v->ld < 1) return SBP_ERR_SHAPE;
    if (v->rows > 0 && v->cols > 0) {
        if (!v->data) return SBP_ERR_NULL;
        if (reinterpret_cast<uintptr_t>(v->data) % elsize(v->dtype)) return SBP_ERR_ALIGN;
    }
    return SBP_OK;
}

// [begin, end) bytes a view touches (empty when it has no elements).
std::pair<uintptr_t, uintptr_t> extent(const void *p, int64_t rows, int64_t cols, int64_t ld,
                                       int32_t dtype) {
    if (rows <= 0 || cols <= 0 || !p) return {0, 0};
    uintptr_t b = reinterpret_cast<uintptr_t>(p);
    uintptr_t e = b + (uintptr_t)(((rows - 1) * ld + cols) * (int64_t)elsize(dtype));
    return {b, e};
}

bool overlaps(std::pair<uintptr_t, uintptr_t> a, std::pair<uintptr_t, uintptr_t> b) {
    if (a.first == a.second || b.first == b.second) return false;
    return a.first < b.second && b.first < a.second;
}

// Output checks shared by the three entry points.
int check_output(const sbp_view_t *o, int64_t rows, int64_t cols, int32_t in_dtype,
                 int32_t out_kind, const Local &a, const Local &b) {
    int rc = check_view_common(o);
    if (rc) return rc;
    if (o->rows != rows || o->cols != cols) return SBP_ERR_SHAPE;
    if (in_dtype == SBP_F32 && o->dtype != SBP_F32) return SBP_ERR_DTYPE;
    if (out_kind == SBP_PARTIAL && o->dtype != SBP_F32) return SBP_ERR_DTYPE;
    if (o->scope == SBP_ACCUMULATE && o->dtype != SBP_F32) return SBP_ERR_DTYPE;
    auto oe = extent(o->data, o->rows, o->cols, o->ld, o->dtype);
    if (overlaps(oe, extent(a.ptr, a.rows, a.cols, a.ld, a.dtype)) ||
        overlaps(oe, extent(b.ptr, b.rows, b.cols, b.ld, b.dtype)))
        return SBP_ERR_ALIAS;
    return SBP_OK;
}

// ---------------------------------------------------------------- workspace
static_assert(SBP_WORKSPACE_BYTES == (int64_t)(sbpi::WS_FLOATS_PREFERRED * sizeof(float)),
              "preferred workspace size");

// A caller's workspace (NULL: none): the split partials it can hold.
struct Ws {
    float *ptr = nullptr;
    size_t floats = 0;
    std::pair<uintptr_t, uintptr_t> span{0, 0};
};

int check_ws(const sbp_workspace_t *ws, Ws *out) {
    *out = Ws{};
    if (!ws || ws->bytes == 0) return SBP_OK;
    if (ws->bytes < 0) return SBP_ERR_SHAPE;
    if (!ws->data) return SBP_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(ws->data) & 15) return SBP_ERR_ALIGN;
    out->ptr = static_cast<float *>(ws->data);
    out->floats = (size_t)ws->bytes / sizeof(float);
    const uintptr_t b = reinterpret_cast<uintptr_t>(ws->data);
    out->span = {b, b + (uintptr_t)ws->bytes};
    return SBP_OK;
}

// The workspace overlaps none of a product's operands or its output.
bool ws_disjoint(const Ws &w, const sbpi::Gemm &g) {
    if (!w.ptr) return true;
    const bool a_km = g.orient != sbpi::OR_BWD_WEIGHT, b_km = g.orient == sbpi::OR_BWD_DATA;
    const auto a = a_km ? extent(g.A, g.m, g.k, g.lda, g.in_dtype)
                        : extent(g.A, g.k, g.m, g.lda, g.in_dtype);
    const auto b = b_km ? extent(g.B, g.n, g.k, g.ldb, g.in_dtype)
                        : extent(g.B, g.k, g.n, g.ldb, g.in_dtype);
    const auto c = extent(g.C, g.m, g.n, g.ldc, g.out_dtype);
    return !overlaps(w.span, a) && !overlaps(w.span, b) && !overlaps(w.span, c);
}

int run(sbpi::Gemm g, const Ws &w, hipStream_t s) {
    if (g.m == 0 || g.n == 0) return SBP_OK;
    hipError_t e;
    if (g.in_dtype == SBP_F32) {
        e = sbpi::launch_f32(g, s);
    } else {
        g.ws_floats = w.floats;
        const sbpi::Plan p = sbpi::plan_bf16(g);
        if (sbpi::plan_ws_floats(g, p) > w.floats) return SBP_ERR_WORKSPACE;
        e = sbpi::launch_bf16(g, p, w.ptr, s);
    }
    if (e != hipSuccess) {
        g_last_hip = (int)e;
        return SBP_ERR_HIP;
    }
    return SBP_OK;
}

// ------------------------------------------------------------ nd layouts
// The 1-D layout (kind, axis, p, r) of mesh axis a of an nd layout.
sbp_layout_t axis_layout(const sbp_nd_layout_t *l, int a) {
    sbp_layout_t o;
    o.kind = l->kind[a];
    o.axis = l->axis[a];
    o.p = l->p[a];
    o.r = l->c[a];
    return o;
}

int check_nd(const sbp_nd_layout_t *l) {
    if (!l) return SBP_ERR_NULL;
    if (l->ndim < 1 || l->ndim > SBP_MAX_MESH_DIMS) return SBP_ERR_LAYOUT;
    for (int a = 0; a < l->ndim; ++a) {
        const sbp_layout_t o = axis_layout(l, a);
        int rc = check_layout(&o);
        if (rc) return rc;
    }
    return SBP_OK;
}

int check_pair(const sbp_nd_layout_t *a, const sbp_nd_layout_t *b) {
    int rc = check_nd(a);
    if (rc) return rc;
    if ((rc = check_nd(b))) return rc;
    if (a->ndim != b->ndim) return SBP_ERR_LAYOUT;
    for (int i = 0; i < a->ndim; ++i)
        if (a->p[i] != b->p[i] || a->c[i] != b->c[i]) return SBP_ERR_LAYOUT;
    return SBP_OK;
}


void nd_set(sbp_nd_layout_t *l, int a, const sbp_layout_t &o) {
    l->kind[a] = o.kind;
    l->axis[a] = o.axis;
}

// Which pair of operands a product's signature is read from.
enum Pair { PAIR_XW = 0, PAIR_DYW = 1, PAIR_XDY = 2 };

// Per-axis factor of an nd signature: the 1-D signature of that axis's states.
int factor_of(Pair pr, const sbp_layout_t &a, const sbp_layout_t &b) {
    Sig s = pr == PAIR_XW ? sig_from_xw(&a, &b)
                          : (pr == PAIR_DYW ? sig_from_dyw(&a, &b) : sig_from_xdy(&a, &b));
    return s == SIG_NONE ? -1 : s;
}

// Signature of a product from its two input layouts: st[0..3] get the
// states of Y, dY, dX, dW. 1-D form: the table at the top of sbp.h.
int resolve(Pair pr, const sbp_layout_t *a, const sbp_layout_t *b, sbp_layout_t st[4]) {
    int rc = check_pair(a, b);
    if (rc) return rc;
    Sig s = pr == PAIR_XW ? sig_from_xw(a, b)
                          : (pr == PAIR_DYW ? sig_from_dyw(a, b) : sig_from_xdy(a, b));
    if (s == SIG_NONE) return SBP_ERR_SIGNATURE;
    states_of(s, a, st);
    return SBP_OK;
}

// nd form: one factor per mesh axis (Sec. 4.2, the 3-D rule factors).
int resolve(Pair pr, const sbp_nd_layout_t *a, const sbp_nd_layout_t *b, sbp_nd_layout_t st[4],
            int *factors = nullptr) {
    int rc = check_pair(a, b);
    if (rc) return rc;
    for (int t = 0; t < 4; ++t) st[t] = *a;
    for (int i = 0; i < a->ndim; ++i) {
        const sbp_layout_t la = axis_layout(a, i), lb = axis_layout(b, i);
        const int f = factor_of(pr, la, lb);
        if (f < 0) return SBP_ERR_SIGNATURE;
        if (factors) factors[i] = f;
        sbp_layout_t o[4];
        states_of((Sig)f, &la, o);
        for (int t = 0; t < 4; ++t) nd_set(&st[t], i, o[t]);
    }
    return SBP_OK;
}

bool is_partial(const sbp_layout_t &l) { return l.kind == SBP_PARTIAL; }
bool is_partial(const sbp_nd_layout_t &l) {
    for (int a = 0; a < l.ndim; ++a)
        if (l.kind[a] == SBP_PARTIAL) return true;
    return false;
}

int shard_of(const sbp_layout_t *l, int64_t rows, int64_t cols, sbp_shard_t *s) {
    return sbp_shard_index(l, rows, cols, s);
}
int shard_of(const sbp_nd_layout_t *l, int64_t rows, int64_t cols, sbp_shard_t *s) {
    return sbp_nd_shard_index(l, rows, cols, s);
}

template <class L>
int local_input(const sbp_view_t *v, const L *l, Local *out) {
    int rc = check_view_common(v);
    if (rc) return rc;
    if (v->scope != SBP_GLOBAL && v->scope != SBP_LOCAL) return SBP_ERR_SHAPE;
    out->dtype = v->dtype;
    out->ld = v->ld;
    out->grows = v->rows;
    out->gcols = v->cols;
    out->global = (v->scope == SBP_GLOBAL);
    if (out->global) {
        sbp_shard_t s;
        rc = shard_of(l, v->rows, v->cols, &s);
        if (rc) return rc;
        out->rows = s.rows;
        out->cols = s.cols;
        out->ptr = static_cast<const char *>(v->data);
        if (s.rows > 0 && s.cols > 0)
            out->ptr += (s.row_off * v->ld + s.col_off) * (int64_t)elsize(v->dtype);
    } else {
        out->rows = v->rows;
        out->cols = v->cols;
        out->ptr = static_cast<const char *>(v->data);
    }
    return SBP_OK;
}

// Validation and operand mapping of the three products (no HIP calls), for
// 1-D (L = sbp_layout_t) and nd (L = sbp_nd_layout_t) layouts.
template <class L>
int prep_fwd(const sbp_view_t *X, const L *lx, const sbp_view_t *W, const L *lw,
             const sbp_view_t *Y, sbpi::Gemm *g, L *st_out) {
    if (!X || !W || !Y || !lx || !lw) return SBP_ERR_NULL;
    L st[4];
    int rc = resolve(PAIR_XW, lx, lw, st);
    if (rc) return rc;
    Local x, w;
    if ((rc = local_input(X, lx, &x))) return rc;
    if ((rc = local_input(W, lw, &w))) return rc;
    if (x.dtype != w.dtype) return SBP_ERR_DTYPE;
    if (x.global && w.global && x.gcols != w.grows) return SBP_ERR_SHAPE;
    if (x.cols != w.rows) return SBP_ERR_SHAPE;
    const int kind = is_partial(st[0]) ? SBP_PARTIAL : SBP_SPLIT;
    if ((rc = check_output(Y, x.rows, w.cols, x.dtype, kind, x, w))) return rc;
    *g = sbpi::Gemm{sbpi::OR_FWD, x.dtype, Y->dtype, x.ptr, x.ld, w.ptr, w.ld,
                    Y->data, Y->ld, x.rows, w.cols, x.cols};
    g->accumulate = Y->scope == SBP_ACCUMULATE;
    *st_out = st[0];
    return SBP_OK;
}

template <class L>
int prep_bwd_data(const sbp_view_t *dY, const L *ldy, const sbp_view_t *W, const L *lw,
                  const sbp_view_t *dX, sbpi::Gemm *g, L *st_out) {
    if (!dY || !W || !dX || !ldy || !lw) return SBP_ERR_NULL;
    L st[4];
    int rc = resolve(PAIR_DYW, ldy, lw, st);
    if (rc) return rc;
    Local d, w;
    if ((rc = local_input(dY, ldy, &d))) return rc;
    if ((rc = local_input(W, lw, &w))) return rc;
    if (d.dtype != w.dtype) return SBP_ERR_DTYPE;
    if (d.global && w.global && d.gcols != w.gcols) return SBP_ERR_SHAPE;
    if (d.cols != w.cols) return SBP_ERR_SHAPE;
    const int kind = is_partial(st[2]) ? SBP_PARTIAL : SBP_SPLIT;
    if ((rc = check_output(dX, d.rows, w.rows, d.dtype, kind, d, w))) return rc;
    *g = sbpi::Gemm{sbpi::OR_BWD_DATA, d.dtype, dX->dtype, d.ptr, d.ld, w.ptr, w.ld,
                    dX->data, dX->ld, d.rows, w.rows, d.cols};
    g->accumulate = dX->scope == SBP_ACCUMULATE;
    *st_out = st[2];
    return SBP_OK;
}

template <class L>
int prep_bwd_weight(const sbp_view_t *X, const L *lx, const sbp_view_t *dY, const L *ldy,
                    const sbp_view_t *dW, sbpi::Gemm *g, L *st_out) {
    if (!X || !dY || !dW || !lx || !ldy) return SBP_ERR_NULL;
    L st[4];
    int rc = resolve(PAIR_XDY, lx, ldy, st);
    if (rc) return rc;
    Local x, d;
    if ((rc = local_input(X, lx, &x))) return rc;
    if ((rc = local_input(dY, ldy, &d))) return rc;
    if (x.dtype != d.dtype) return SBP_ERR_DTYPE;
    if (x.global && d.global && x.grows != d.grows) return SBP_ERR_SHAPE;
    if (x.rows != d.rows) return SBP_ERR_SHAPE;
    const int kind = is_partial(st[3]) ? SBP_PARTIAL : SBP_SPLIT;
    if ((rc = check_output(dW, x.cols, d.cols, x.dtype, kind, x, d))) return rc;
    *g = sbpi::Gemm{sbpi::OR_BWD_WEIGHT, x.dtype, dW->dtype, x.ptr, x.ld, d.ptr, d.ld,
                    dW->data, dW->ld, x.cols, d.cols, x.rows};
    g->accumulate = dW->scope == SBP_ACCUMULATE;
    *st_out = st[3];
    return SBP_OK;
}

// Both backward products: one grouped launch when the planner finds it
// faster, else two launches. An empty product is skipped.
int hip_fail(hipError_t e) {
    g_last_hip = (int)e;
    return SBP_ERR_HIP;
}

int run_pair(sbpi::Gemm gd, sbpi::Gemm gw, const Ws &w, hipStream_t s) {
    const bool ed = gd.m == 0 || gd.n == 0, ew = gw.m == 0 || gw.n == 0;
    if (gd.in_dtype == SBP_BF16 && !ed && !ew) {
        gd.ws_floats = gw.ws_floats = w.floats;
        sbpi::Plan pd, pw;
        if (sbpi::plan_bf16_bwd(gd, gw, &pd, &pw)) {
            if (sbpi::plan_ws_floats(gd, pd) + sbpi::plan_ws_floats(gw, pw) > w.floats)
                return SBP_ERR_WORKSPACE;
            hipError_t e = sbpi::launch_bf16_bwd_group(gd, pd, gw, pw, w.ptr, s);
            if (e != hipSuccess) return hip_fail(e);
            return SBP_OK;
        }
    }
    // two launches in stream order: each may use the whole workspace
    int rc = run(gd, w, s);
    if (rc) return rc;
    return run(gw, w, s);
}

// The three input states of a backward call describe one signature: the
// factor read from (X, W) equals those read from (dY, W) and (X, dY).
bool one_signature(const sbp_layout_t *lx, const sbp_layout_t *lw, const sbp_layout_t *ldy) {
    const Sig s = sig_from_xw(lx, lw);
    return s != SIG_NONE && sig_from_dyw(ldy, lw) == s && sig_from_xdy(lx, ldy) == s;
}
bool one_signature(const sbp_nd_layout_t *lx, const sbp_nd_layout_t *lw,
                   const sbp_nd_layout_t *ldy) {
    for (int a = 0; a < lx->ndim; ++a) {
        const sbp_layout_t x = axis_layout(lx, a), w = axis_layout(lw, a),
                           d = axis_layout(ldy, a);
        const int f = factor_of(PAIR_XW, x, w);
        if (f < 0 || factor_of(PAIR_DYW, d, w) != f || factor_of(PAIR_XDY, x, d) != f)
            return false;
    }
    return true;
}

template <class L>
int linear_fwd(const sbp_view_t *X, const L *lx, const sbp_view_t *W, const L *lw,
               sbp_view_t *Y, L *ly_out, const sbp_workspace_t *ws, hipStream_t stream) {
    sbpi::Gemm g;
    L st;
    int rc = prep_fwd(X, lx, W, lw, Y, &g, &st);
    if (rc) return rc;
    Ws w;
    if ((rc = check_ws(ws, &w))) return rc;
    if (!ws_disjoint(w, g)) return SBP_ERR_ALIAS;
    if ((rc = run(g, w, stream))) return rc;
    if (ly_out) *ly_out = st;
    return SBP_OK;
}

template <class L>
int linear_bwd_data(const sbp_view_t *dY, const L *ldy, const sbp_view_t *W, const L *lw,
                    sbp_view_t *dX, L *ldx_out, const sbp_workspace_t *ws, hipStream_t stream) {
    sbpi::Gemm g;
    L st;
    int rc = prep_bwd_data(dY, ldy, W, lw, dX, &g, &st);
    if (rc) return rc;
    Ws w;
    if ((rc = check_ws(ws, &w))) return rc;
    if (!ws_disjoint(w, g)) return SBP_ERR_ALIAS;
    if ((rc = run(g, w, stream))) return rc;
    if (ldx_out) *ldx_out = st;
    return SBP_OK;
}

template <class L>
int linear_bwd_weight(const sbp_view_t *X, const L *lx, const sbp_view_t *dY, const L *ldy,
                      sbp_view_t *dW, L *ldw_out, const sbp_workspace_t *ws,
                      hipStream_t stream) {
    sbpi::Gemm g;
    L st;
    int rc = prep_bwd_weight(X, lx, dY, ldy, dW, &g, &st);
    if (rc) return rc;
    Ws w;
    if ((rc = check_ws(ws, &w))) return rc;
    if (!ws_disjoint(w, g)) return SBP_ERR_ALIAS;
    if ((rc = run(g, w, stream))) return rc;
    if (ldw_out) *ldw_out = st;
    return SBP_OK;
}

// Validation and operand mapping of both backward products (no HIP calls).
template <class L>
int prep_bwd_pair(const sbp_view_t *dY, const L *ldy, const sbp_view_t *X, const L *lx,
                  const sbp_view_t *W, const L *lw, sbp_view_t *dX, sbp_view_t *dW,
                  sbpi::Gemm *gd, L *sd, sbpi::Gemm *gw, L *sw) {
    if (!dY || !X || !W || !dX || !dW || !ldy || !lx || !lw) return SBP_ERR_NULL;
    int rc = check_pair(lx, lw);
    if (rc) return rc;
    if ((rc = check_pair(ldy, lw))) return rc;
    // the three input states must describe one signature
    if (!one_signature(lx, lw, ldy)) return SBP_ERR_SIGNATURE;
    if ((rc = prep_bwd_data(dY, ldy, W, lw, dX, gd, sd))) return rc;
    if ((rc = prep_bwd_weight(X, lx, dY, ldy, dW, gw, sw))) return rc;
    // no output may overlap the other output or the input it is not checked
    // against above (dX vs X, dW vs W)
    const auto ex = extent(dX->data, dX->rows, dX->cols, dX->ld, dX->dtype);
    const auto ew = extent(dW->data, dW->rows, dW->cols, dW->ld, dW->dtype);
    const auto xr = extent(gw->A, gw->k, gw->m, gw->lda, gw->in_dtype);   // X_r: k x m view
    const auto wr = extent(gd->B, gd->n, gd->k, gd->ldb, gd->in_dtype);   // W_r: n x k view
    if (overlaps(ex, ew) || overlaps(ex, xr) || overlaps(ew, wr)) return SBP_ERR_ALIAS;
    return SBP_OK;
}

template <class L>
int linear_bwd(const sbp_view_t *dY, const L *ldy, const sbp_view_t *X, const L *lx,
               const sbp_view_t *W, const L *lw, sbp_view_t *dX, L *ldx_out, sbp_view_t *dW,
               L *ldw_out, const sbp_workspace_t *ws, hipStream_t stream) {
    sbpi::Gemm gd, gw;
    L sd, sw;
    int rc = prep_bwd_pair(dY, ldy, X, lx, W, lw, dX, dW, &gd, &sd, &gw, &sw);
    if (rc) return rc;
    Ws w;
    if ((rc = check_ws(ws, &w))) return rc;
    if (!ws_disjoint(w, gd) || !ws_disjoint(w, gw)) return SBP_ERR_ALIAS;
    if ((rc = run_pair(gd, gw, w, stream))) return rc;
    if (ldx_out) *ldx_out = sd;
    if (ldw_out) *ldw_out = sw;
    return SBP_OK;
}

}  // namespace

namespace sbpa {
int run_gemm(const sbpi::Gemm &g, hipStream_t s) { return run(g, Ws{}, s); }
}  // namespace sbpa

extern "C" {

int sbp_shard_index(const sbp_layout_t *l, int64_t rows, int64_t cols, sbp_shard_t *out) {
    if (!l || !out) return SBP_ERR_NULL;
    int rc = check_layout(l);
    if (rc) return rc;
    if (rows < 0 || cols < 0) return SBP_ERR_SHAPE;
    sbp_shard_t s{0, 0, rows, cols};
    if (l->kind == SBP_SPLIT) {
        const int64_t D = (l->axis == 0) ? rows : cols;
        const int64_t base = D / l->p, rem = D % l->p;
        const int64_t len = base + (l->r < rem ? 1 : 0);
        const int64_t off = (int64_t)l->r * base + (l->r < rem ? l->r : rem);
        if (l->axis == 0) {
            s.row_off = off;
            s.rows = len;
        } else {
            s.col_off = off;
            s.cols = len;
        }
    }
    *out = s;
    return SBP_OK;
}

int sbp_signature(const sbp_layout_t *x, const sbp_layout_t *w, sbp_layout_t *y,
                  sbp_layout_t *dy, sbp_layout_t *dx, sbp_layout_t *dw) {
    if (!x || !w) return SBP_ERR_NULL;
    int rc = check_pair(x, w);
    if (rc) return rc;
    Sig s = sig_from_xw(x, w);
    if (s == SIG_NONE) return SBP_ERR_SIGNATURE;
    sbp_layout_t st[4];
    states_of(s, x, st);
    if (y) *y = st[0];
    if (dy) *dy = st[1];
    if (dx) *dx = st[2];
    if (dw) *dw = st[3];
    return SBP_OK;
}

int sbp_linear_fwd(const sbp_view_t *X, const sbp_layout_t *lx, const sbp_view_t *W,
                   const sbp_layout_t *lw, sbp_view_t *Y, sbp_layout_t *ly_out,
                   const sbp_workspace_t *ws, hipStream_t stream) {
    return linear_fwd(X, lx, W, lw, Y, ly_out, ws, stream);
}

int sbp_linear_bwd_data(const sbp_view_t *dY, const sbp_layout_t *ldy, const sbp_view_t *W,
                        const sbp_layout_t *lw, sbp_view_t *dX, sbp_layout_t *ldx_out,
                        const sbp_workspace_t *ws, hipStream_t stream) {
    return linear_bwd_data(dY, ldy, W, lw, dX, ldx_out, ws, stream);
}

int sbp_linear_bwd_weight(const sbp_view_t *X, const sbp_layout_t *lx, const sbp_view_t *dY,
                          const sbp_layout_t *ldy, sbp_view_t *dW, sbp_layout_t *ldw_out,
                          const sbp_workspace_t *ws, hipStream_t stream) {
    return linear_bwd_weight(X, lx, dY, ldy, dW, ldw_out, ws, stream);
}

int sbp_linear_bwd(const sbp_view_t *dY, const sbp_layout_t *ldy, const sbp_view_t *X,
                   const sbp_layout_t *lx, const sbp_view_t *W, const sbp_layout_t *lw,
                   sbp_view_t *dX, sbp_layout_t *ldx_out, sbp_view_t *dW,
                   sbp_layout_t *ldw_out, const sbp_workspace_t *ws, hipStream_t stream) {
    return linear_bwd(dY, ldy, X, lx, W, lw, dX, ldx_out, dW, ldw_out, ws, stream);
}

int sbp_linear_bwd_noalloc(const sbp_view_t *dY, const sbp_layout_t *ldy, const sbp_view_t *X,
                           const sbp_layout_t *lx, const sbp_view_t *W, const sbp_layout_t *lw,
                           sbp_view_t *dX, sbp_layout_t *ldx_out, sbp_view_t *dW,
                           sbp_layout_t *ldw_out, hipStream_t stream) {
    sbpi::Gemm gd, gw;
    sbp_layout_t sd, sw;
    int rc = prep_bwd_pair(dY, ldy, X, lx, W, lw, dX, dW, &gd, &sd, &gw, &sw);
    if (rc) return rc;
    Ws w;
    hipError_t e = sbpi::static_scratch(&w.ptr, &w.floats);
    if (e != hipSuccess) return hip_fail(e);
    const uintptr_t b = reinterpret_cast<uintptr_t>(w.ptr);
    w.span = {b, b + w.floats * sizeof(float)};
    if (!ws_disjoint(w, gd) || !ws_disjoint(w, gw)) return SBP_ERR_ALIAS;
    // the plan is limited to partials that fit the scratch; run_pair refuses
    // (SBP_ERR_WORKSPACE) any plan that would need more
    if ((rc = run_pair(gd, gw, w, stream))) return rc;
    if (ldx_out) *ldx_out = sd;
    if (ldw_out) *ldw_out = sw;
    return SBP_OK;
}

int sbp_mesh_coords(int32_t ndim, const int32_t *nodes, const int32_t *gpus, int64_t node,
                    int64_t gpu, int32_t *c) {
    if (!nodes || !c) return SBP_ERR_NULL;
    if (ndim < 1 || ndim > SBP_MAX_MESH_DIMS) return SBP_ERR_LAYOUT;
    int64_t n_total = 1, g_total = 1;
    for (int a = 0; a < ndim; ++a) {
        const int64_t g = gpus ? gpus[a] : 1;
        if (nodes[a] < 1 || g < 1) return SBP_ERR_LAYOUT;
        n_total *= nodes[a];
        g_total *= g;
        if (n_total * g_total > INT32_MAX) return SBP_ERR_LAYOUT;   // devices fit int32
    }
    if (node < 0 || node >= n_total || gpu < 0 || gpu >= g_total) return SBP_ERR_LAYOUT;
    // mixed-radix digits, mesh axis 0 fastest, at both levels
    for (int a = 0; a < ndim; ++a) {
        const int64_t g = gpus ? gpus[a] : 1;
        const int64_t nd = node % nodes[a], gd = gpu % g;
        node /= nodes[a];
        gpu /= g;
        c[a] = (int32_t)(nd * g + gd);
    }
    return SBP_OK;
}

int sbp_nd_shard_index(const sbp_nd_layout_t *l, int64_t rows, int64_t cols, sbp_shard_t *out) {
    if (!l || !out) return SBP_ERR_NULL;
    int rc = check_nd(l);
    if (rc) return rc;
    if (rows < 0 || cols < 0) return SBP_ERR_SHAPE;
    sbp_shard_t s{0, 0, rows, cols};
    // nested splits in mesh-axis order: each split axis cuts the current
    // block of its tensor axis (the 1-D balanced rule on the block's extent)
    for (int a = 0; a < l->ndim; ++a) {
        if (l->kind[a] != SBP_SPLIT) continue;
        const sbp_layout_t o = axis_layout(l, a);
        const bool r0 = (l->axis[a] == 0);
        sbp_shard_t sub;
        if ((rc = sbp_shard_index(&o, r0 ? s.rows : 1, r0 ? 1 : s.cols, &sub))) return rc;
        if (r0) {
            s.row_off += sub.row_off;
            s.rows = sub.rows;
        } else {
            s.col_off += sub.col_off;
            s.cols = sub.cols;
        }
    }
    *out = s;
    return SBP_OK;
}

int sbp_nd_signature(const sbp_nd_layout_t *x, const sbp_nd_layout_t *w, sbp_nd_layout_t *y,
                     sbp_nd_layout_t *dy, sbp_nd_layout_t *dx, sbp_nd_layout_t *dw) {
    if (!x || !w) return SBP_ERR_NULL;
    sbp_nd_layout_t st[4];
    int rc = resolve(PAIR_XW, x, w, st);
    if (rc) return rc;
    if (y) *y = st[0];
    if (dy) *dy = st[1];
    if (dx) *dx = st[2];
    if (dw) *dw = st[3];
    return SBP_OK;
}

int sbp_nd_linear_fwd(const sbp_view_t *X, const sbp_nd_layout_t *lx, const sbp_view_t *W,
                      const sbp_nd_layout_t *lw, sbp_view_t *Y, sbp_nd_layout_t *ly_out,
                      const sbp_workspace_t *ws, hipStream_t stream) {
    return linear_fwd(X, lx, W, lw, Y, ly_out, ws, stream);
}

int sbp_nd_linear_bwd_data(const sbp_view_t *dY, const sbp_nd_layout_t *ldy,
                           const sbp_view_t *W, const sbp_nd_layout_t *lw, sbp_view_t *dX,
                           sbp_nd_layout_t *ldx_out, const sbp_workspace_t *ws,
                           hipStream_t stream) {
    return linear_bwd_data(dY, ldy, W, lw, dX, ldx_out, ws, stream);
}

int sbp_nd_linear_bwd_weight(const sbp_view_t *X, const sbp_nd_layout_t *lx,
                             const sbp_view_t *dY, const sbp_nd_layout_t *ldy, sbp_view_t *dW,
                             sbp_nd_layout_t *ldw_out, const sbp_workspace_t *ws,
                             hipStream_t stream) {
    return linear_bwd_weight(X, lx, dY, ldy, dW, ldw_out, ws, stream);
}

int sbp_nd_linear_bwd(const sbp_view_t *dY, const sbp_nd_layout_t *ldy, const sbp_view_t *X,
                      const sbp_nd_layout_t *lx, const sbp_view_t *W, const sbp_nd_layout_t *lw,
                      sbp_view_t *dX, sbp_nd_layout_t *ldx_out, sbp_view_t *dW,
                      sbp_nd_layout_t *ldw_out, const sbp_workspace_t *ws, hipStream_t stream) {
    return linear_bwd(dY, ldy, X, lx, W, lw, dX, ldx_out, dW, ldw_out, ws, stream);
}

const char *sbp_strerror(int code) {
    switch (code) {
        case SBP_OK: return "success";
        case SBP_ERR_NULL: return "a required pointer is NULL";
        case SBP_ERR_LAYOUT: return "invalid SBP layout (p, r, kind or axis), or layouts disagree on p or r";
        case SBP_ERR_SIGNATURE: return "the input SBP states form no supported signature";
        case SBP_ERR_SHAPE: return "shape mismatch, ld < cols, or output view is not the local output shape";
        case SBP_ERR_DTYPE: return "unsupported or inconsistent dtype (partial-sum outputs must be fp32)";
        case SBP_ERR_ALIAS: return "the output overlaps an input";
        case SBP_ERR_ALIGN: return "a data pointer is not aligned to its element size";
        case SBP_ERR_HIP: return "a HIP runtime call failed";
        case SBP_ERR_WORKSPACE: return "the split partials of the call's plan do not fit its workspace";
    }
    return "unknown error code";
}

int sbp_last_hip_error(void) { return g_last_hip; }

int sbp_plan(int op, int64_t m, int64_t n, int64_t k, int32_t in_dtype, int32_t out_dtype,
             int32_t *tile_m, int32_t *tile_n, int32_t *splits, int32_t *kernel) {
    if (!tile_m || !tile_n || !splits || !kernel) return SBP_ERR_NULL;
    if (m < 0 || n < 0 || k < 0 || m > INT32_MAX || n > INT32_MAX || k > INT32_MAX ||
        op < 0 || op > 2)
        return SBP_ERR_SHAPE;
    if ((in_dtype != SBP_BF16 && in_dtype != SBP_F32) ||
        (out_dtype != SBP_BF16 && out_dtype != SBP_F32))
        return SBP_ERR_DTYPE;
    if (in_dtype == SBP_F32) {
        *tile_m = 64;
        *tile_n = 64;
        *splits = 1;
        *kernel = 3;
        return SBP_OK;
    }
    // Plan for 16-byte aligned operands with tight leading dimensions.
    static const char aligned[16] __attribute__((aligned(16))) = {0};
    const int64_t lda = (op == 2) ? m : k, ldb = (op == 1) ? k : n;
    sbpi::Gemm g{op, in_dtype, out_dtype, aligned, lda, aligned, ldb, nullptr, 0, m, n, k};
    g.ws_floats = sbpi::WS_FLOATS_PREFERRED;
    sbpi::Plan p = sbpi::plan_bf16(g);
    *tile_m = p.bm;
    *tile_n = p.bn;
    *splits = p.splits;
    *kernel = sbpi::kernel_code(p);
    return SBP_OK;
}

int sbp_plan_bwd(int64_t md, int64_t nd, int64_t kd, int32_t out_d, int64_t mw, int64_t nw,
                 int64_t kw, int32_t out_w, int32_t *grouped, int32_t *tile_m, int32_t *tile_n,
                 int32_t *splits_d, int32_t *splits_w) {
    if (!grouped || !tile_m || !tile_n || !splits_d || !splits_w) return SBP_ERR_NULL;
    const int64_t dims[6] = {md, nd, kd, mw, nw, kw};
    for (int64_t d : dims)
        if (d < 0 || d > INT32_MAX) return SBP_ERR_SHAPE;
    if ((out_d != SBP_BF16 && out_d != SBP_F32) || (out_w != SBP_BF16 && out_w != SBP_F32))
        return SBP_ERR_DTYPE;
    static const char aligned[16] __attribute__((aligned(16))) = {0};
    sbpi::Gemm gd{sbpi::OR_BWD_DATA, SBP_BF16, out_d, aligned, kd, aligned, kd, nullptr, 0,
                  md, nd, kd};
    sbpi::Gemm gw{sbpi::OR_BWD_WEIGHT, SBP_BF16, out_w, aligned, mw, aligned, nw, nullptr, 0,
                  mw, nw, kw};
    gd.ws_floats = gw.ws_floats = sbpi::WS_FLOATS_PREFERRED;
    sbpi::Plan pd, pw;
    *grouped = sbpi::plan_bf16_bwd(gd, gw, &pd, &pw) ? 1 : 0;
    *tile_m = pd.bm;
    *tile_n = pd.bn;
    *splits_d = pd.splits;
    *splits_w = pw.splits;
    return SBP_OK;
}

int sbp_set_plan_override(int32_t tile_m, int32_t tile_n, int32_t splits, int32_t kernel,
                          int32_t wgs_per_cu) {
    if (tile_m == 0) {
        sbpi::set_override(0, 0, 1, 0);
        sbpi::set_override_occ(0);
        sbpi::set_bwd_override(0, 1);
        sbpi::set_override_orients(7);
        return SBP_OK;
    }
    if (splits < 1 || wgs_per_cu < 0 || wgs_per_cu > 8) return SBP_ERR_SHAPE;
    if (!sbpi::override_supported(tile_m, tile_n, kernel)) return SBP_ERR_SHAPE;
    sbpi::set_override(tile_m, tile_n, splits, kernel);
    sbpi::set_override_occ(wgs_per_cu);
    return SBP_OK;
}

int sbp_set_override_orients(int32_t mask) {
    if (mask < 1 || mask > 7) return SBP_ERR_SHAPE;
    sbpi::set_override_orients(mask);
    return SBP_OK;
}

int sbp_set_bwd_override(int32_t mode, int32_t splits_w) {
    if (mode < 0 || mode > 2 || splits_w < 1) return SBP_ERR_SHAPE;
    sbpi::set_bwd_override(mode, splits_w);
    return SBP_OK;
}

}  // extern "C"
