/*
 * oracle.c -- plain CPU oracle for the local-shard SBP linear layer.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may call, link or
 * load this file: only the tests, the smoke check and the benchmark's CPU
 * baseline use it. It shares no code, header, table or helper with the HIP
 * library; it has its own split formula, its own signature table and its own
 * bf16 decoding and rounding.
 *
 * What it computes (AutoDDL, Sec. 4.2 "Distributed Matrix Multiplication
 * based on SBP", and Sec. 4.3 "Sources of Communication"):
 *
 *   A 2-D tensor in SBP state Split(i) is cut into p contiguous blocks along
 *   axis i, one per device; Broadcast means every device holds all of it;
 *   Partial-sum means every device holds a tensor of the full shape and the
 *   true tensor is the element-wise sum over devices (Sec. 4.1, Fig. 5 and
 *   its caption; Sec. 1 defines the partial-sum state).
 *
 *   For I W = O on a 1-D mesh of p devices, the three per-axis factors of
 *   the 3-D rule of Sec. 4.2 are
 *       data parallel   (S(0), B)    -> S(0)      [p1 = p2 = 1 case]
 *       column          (B,    S(1)) -> S(1)      [p0 = p2 = 1 case]
 *       K-split         (S(1), S(0)) -> P         [p0 = p1 = 1 case]
 *   and each device multiplies its local shares ("local matmul").
 *
 *   Backward: dX = dY W^T and dW = X^T dY on the same local shares. A
 *   broadcast operand's gradient is a partial sum (Sec. 4.3: a replicated
 *   weight receives gradients in the partial-sum state); a split operand's
 *   gradient is split the same way.
 *
 * Arithmetic: inputs are decoded exactly (bf16 bits u16 -> fp32 by a 16-bit
 * shift, fp32 as is) and every product and sum is taken in fp64, in
 * increasing reduction index, with no blocking or reordering. Products of two
 * fp32 values are exact in fp64, so the result is the exact product rounded
 * only by the fp64 running sum.
 *
 * Parity status: pinned (reassembly invariant against brute-force global
 * products, exact integer cases, closed forms, p = 1 textbook case, bf16
 * rounding against a library conversion); see tests/test_oracle_*.py.
 */
#include <stdint.h>
#include <string.h>
#include <math.h>

/* ----------------------------------------------------------------- ids --- */
/* signatures */
enum { ORC_DP = 0, ORC_COL = 1, ORC_KS = 2 };
/* operations */
enum { ORC_FWD = 0, ORC_BWD_DATA = 1, ORC_BWD_WEIGHT = 2 };
/* tensor state kinds */
enum { ORC_SPLIT = 0, ORC_BCAST = 1, ORC_PARTIAL = 2 };
/* input encodings */
enum { ORC_IN_BF16 = 0, ORC_IN_F32 = 1 };

/* ------------------------------------------------------------ the split --- */
/*
 * Balanced contiguous split of an extent D over p devices, rank r.
 * The paper does not say how an extent that p does not divide is cut; the
 * reading taken is contiguous blocks in rank order where the first D mod p
 * ranks get one extra element.
 */
void orc_split(int64_t D, int64_t p, int64_t r, int64_t *off, int64_t *len)
{
    int64_t base = D / p;
    int64_t rem = D % p;
    *len = base + (r < rem ? 1 : 0);
    *off = r * base + (r < rem ? r : rem);
}

/* --------------------------------------------------- signature table ---- */
/*
 * For signature sig, writes the (kind, axis) state of the six tensors in the
 * order X, W, Y, dY, dX, dW. Axis is -1 for Broadcast and Partial-sum.
 * Returns 0, or -1 for an unknown signature.
 */
int orc_tags(int sig, int32_t kinds[6], int32_t axes[6])
{
    /*                 X          W          Y            dY         dX           dW        */
    static const int32_t K[3][6] = {
        {ORC_SPLIT, ORC_BCAST, ORC_SPLIT,   ORC_SPLIT, ORC_SPLIT,   ORC_PARTIAL}, /* DP  */
        {ORC_BCAST, ORC_SPLIT, ORC_SPLIT,   ORC_SPLIT, ORC_PARTIAL, ORC_SPLIT  }, /* COL */
        {ORC_SPLIT, ORC_SPLIT, ORC_PARTIAL, ORC_BCAST, ORC_SPLIT,   ORC_SPLIT  }, /* KS  */
    };
    static const int32_t A[3][6] = {
        { 0, -1,  0,  0,  0, -1},
        {-1,  1,  1,  1, -1,  1},
        { 1,  0, -1, -1,  1,  0},
    };
    if (sig < 0 || sig > 2) return -1;
    for (int t = 0; t < 6; ++t) { kinds[t] = K[sig][t]; axes[t] = A[sig][t]; }
    return 0;
}

/* A local share of a row-major global matrix: rows [r0, r0+nr), cols [c0, c0+nc). */
typedef struct { int64_t r0, nr, c0, nc; } orc_share;

/* Rank r's share of a rows x cols tensor in state (kind, axis). */
static orc_share share_of(int32_t kind, int32_t axis, int64_t rows, int64_t cols,
                          int64_t p, int64_t r)
{
    orc_share s = {0, rows, 0, cols};
    if (kind == ORC_SPLIT && axis == 0) orc_split(rows, p, r, &s.r0, &s.nr);
    if (kind == ORC_SPLIT && axis == 1) orc_split(cols, p, r, &s.c0, &s.nc);
    return s;
}

/* --------------------------------------------------- input decoding ------ */
static double decode(const void *base, int enc, int64_t idx)
{
    if (enc == ORC_IN_BF16) {
        uint16_t h = ((const uint16_t *)base)[idx];
        uint32_t u = (uint32_t)h << 16;
        float f;
        memcpy(&f, &u, sizeof f);
        return (double)f;
    }
    return (double)((const float *)base)[idx];
}

/* ------------------------------------------------- local output shape --- */
/*
 * Shapes of rank r's operand shares and output for one operation.
 * X is M x K, W is K x N, dY is M x N (global, row-major).
 */
typedef struct { orc_share x, w, dy; int64_t out_rows, out_cols; } orc_plan;

static int make_plan(int sig, int op, int64_t M, int64_t K, int64_t N,
                     int64_t p, int64_t r, orc_plan *pl)
{
    int32_t kd[6], ax[6];
    if (orc_tags(sig, kd, ax) != 0) return -1;
    if (op < 0 || op > 2 || p < 1 || r < 0 || r >= p) return -1;
    pl->x = share_of(kd[0], ax[0], M, K, p, r);
    pl->w = share_of(kd[1], ax[1], K, N, p, r);
    pl->dy = share_of(kd[3], ax[3], M, N, p, r);
    if (op == ORC_FWD) {          /* Y_r = X_r W_r            : (x.nr) x (w.nc) */
        pl->out_rows = pl->x.nr;
        pl->out_cols = pl->w.nc;
    } else if (op == ORC_BWD_DATA) { /* dX_r = dY_r W_r^T     : (dy.nr) x (w.nr) */
        pl->out_rows = pl->dy.nr;
        pl->out_cols = pl->w.nr;
    } else {                      /* dW_r = X_r^T dY_r        : (x.nc) x (dy.nc) */
        pl->out_rows = pl->x.nc;
        pl->out_cols = pl->dy.nc;
    }
    return 0;
}

/* Output shape and state of operation op under signature sig for rank r. */
int orc_out_shape(int sig, int op, int64_t M, int64_t K, int64_t N, int64_t p,
                  int64_t r, int64_t *rows, int64_t *cols, int32_t *kind,
                  int32_t *axis)
{
    orc_plan pl;
    int32_t kd[6], ax[6];
    if (make_plan(sig, op, M, K, N, p, r, &pl) != 0) return -1;
    orc_tags(sig, kd, ax);
    int t = (op == ORC_FWD) ? 2 : (op == ORC_BWD_DATA ? 4 : 5);
    *rows = pl.out_rows;
    *cols = pl.out_cols;
    *kind = kd[t];
    *axis = ax[t];
    return 0;
}

/* One element (i, j) of rank r's output: a plain dot product in fp64. */
static double element(const orc_plan *pl, int op, int enc, int64_t K, int64_t N,
                      const void *X, const void *W, const void *dY, int64_t i,
                      int64_t j)
{
    double acc = 0.0;
    if (op == ORC_FWD) {
        /* Y[i][j] = sum_k X_r[i][k] W_r[k][j] */
        for (int64_t k = 0; k < pl->x.nc; ++k)
            acc += decode(X, enc, (pl->x.r0 + i) * K + (pl->x.c0 + k)) *
                   decode(W, enc, (pl->w.r0 + k) * N + (pl->w.c0 + j));
    } else if (op == ORC_BWD_DATA) {
        /* dX[i][j] = sum_t dY_r[i][t] W_r[j][t] */
        for (int64_t t = 0; t < pl->dy.nc; ++t)
            acc += decode(dY, enc, (pl->dy.r0 + i) * N + (pl->dy.c0 + t)) *
                   decode(W, enc, (pl->w.r0 + j) * N + (pl->w.c0 + t));
    } else {
        /* dW[i][j] = sum_t X_r[t][i] dY_r[t][j] */
        for (int64_t t = 0; t < pl->x.nr; ++t)
            acc += decode(X, enc, (pl->x.r0 + t) * K + (pl->x.c0 + i)) *
                   decode(dY, enc, (pl->dy.r0 + t) * N + (pl->dy.c0 + j));
    }
    return acc;
}

/*
 * Block [i0, i1) x [j0, j1) of rank r's output of operation op, as fp64,
 * written row-major into out ((i1-i0) x (j1-j0)). Inputs are the global,
 * contiguous row-major X (M x K), W (K x N) and dY (M x N); only the tensors
 * the operation reads need to be non-null. Returns 0, or -1 on a bad
 * argument (unknown signature/op, rank out of range, block outside the
 * output).
 */
int orc_linear_block(int sig, int op, int enc, int64_t M, int64_t K, int64_t N,
                     int64_t p, int64_t r, const void *X, const void *W,
                     const void *dY, int64_t i0, int64_t i1, int64_t j0,
                     int64_t j1, double *out)
{
    orc_plan pl;
    if (make_plan(sig, op, M, K, N, p, r, &pl) != 0) return -1;
    if (enc != ORC_IN_BF16 && enc != ORC_IN_F32) return -1;
    if (i0 < 0 || j0 < 0 || i1 < i0 || j1 < j0 || i1 > pl.out_rows ||
        j1 > pl.out_cols)
        return -1;
    int64_t w = j1 - j0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = i0; i < i1; ++i)
        for (int64_t j = j0; j < j1; ++j)
            out[(i - i0) * w + (j - j0)] =
                element(&pl, op, enc, K, N, X, W, dY, i, j);
    return 0;
}

/* n single elements (ii[s], jj[s]) of rank r's output, as fp64. */
int orc_linear_samples(int sig, int op, int enc, int64_t M, int64_t K,
                       int64_t N, int64_t p, int64_t r, const void *X,
                       const void *W, const void *dY, int64_t n,
                       const int64_t *ii, const int64_t *jj, double *out)
{
    orc_plan pl;
    if (make_plan(sig, op, M, K, N, p, r, &pl) != 0) return -1;
    if (enc != ORC_IN_BF16 && enc != ORC_IN_F32) return -1;
    for (int64_t s = 0; s < n; ++s)
        if (ii[s] < 0 || ii[s] >= pl.out_rows || jj[s] < 0 || jj[s] >= pl.out_cols)
            return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t s = 0; s < n; ++s)
        out[s] = element(&pl, op, enc, K, N, X, W, dY, ii[s], jj[s]);
    return 0;
}

/*
 * Round fp64 values to bfloat16 (8 significant bits, round to nearest, ties
 * to even) and return the 16-bit patterns. Used where a bf16 output of the
 * library is compared bit for bit with an exactly known value. Values beyond
 * the bf16 range become infinities; zero keeps its sign.
 */
void orc_round_bf16(const double *in, uint16_t *out, int64_t n)
{
    for (int64_t s = 0; s < n; ++s) {
        double x = in[s];
        double y;
        if (x == 0.0 || isnan(x) || isinf(x)) {
            y = x;
        } else {
            int e;
            double m = frexp(x, &e);           /* x = m 2^e, 0.5 <= |m| < 1 */
            double q = nearbyint(m * 256.0);   /* 8 significant bits, ties even */
            y = ldexp(q, e - 8);
            if (fabs(y) > 3.3895313892515355e38) y = copysign(INFINITY, x);
        }
        float f = (float)y;                    /* exact: y has 8 significant bits */
        uint32_t u;
        memcpy(&u, &f, sizeof u);
        out[s] = (uint16_t)(u >> 16);
    }
}
