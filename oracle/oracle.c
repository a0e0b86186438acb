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
 *   By linearity three more signatures need no split at all:
 *       partial input   (P, B) -> P    and    (B, P) -> P
 *       replicated      (B, B) -> B
 *   (a product is linear in each operand, so partial sums of one operand
 *   give partial sums of the product; two replicated operands give a
 *   replicated product).
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
 * only by the fp64 running sum. orc_linear_block_f32 is the same loop with
 * an fp32 accumulator (each step c = fl32(c + fl32(a b)), built with
 * -ffp-contract=off): the plain fp32 triple loop, for the fp32-path parity
 * check and the timed CPU baseline.
 *
 * The nd-SBP section below extends this to device meshes (one state per
 * mesh axis).
 *
 * Parity status: pinned (reassembly invariant against brute-force global
 * products, exact integer cases, closed forms, p = 1 textbook case, bf16
 * rounding against a library conversion; for meshes, Listing 1's blocks,
 * the heterogeneous GPU mapping example and the mesh reassembly invariant);
 * see tests/test_oracle_*.py.
 */
#include <stdint.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ----------------------------------------------------------------- ids --- */
/* signatures */
enum { ORC_DP = 0, ORC_COL = 1, ORC_KS = 2, ORC_PB = 3, ORC_BP = 4, ORC_BB = 5 };
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
 * The gradient of a Split(i) tensor is Split(i), of a Broadcast tensor a
 * Partial-sum (Sec. 4.3), of a Partial-sum tensor a Broadcast.
 * Returns 0, or -1 for an unknown signature.
 */
int orc_tags(int sig, int32_t kinds[6], int32_t axes[6])
{
    /*                 X            W            Y            dY           dX           dW        */
    static const int32_t K[6][6] = {
        {ORC_SPLIT,   ORC_BCAST,   ORC_SPLIT,   ORC_SPLIT,   ORC_SPLIT,   ORC_PARTIAL}, /* DP  */
        {ORC_BCAST,   ORC_SPLIT,   ORC_SPLIT,   ORC_SPLIT,   ORC_PARTIAL, ORC_SPLIT  }, /* COL */
        {ORC_SPLIT,   ORC_SPLIT,   ORC_PARTIAL, ORC_BCAST,   ORC_SPLIT,   ORC_SPLIT  }, /* KS  */
        {ORC_PARTIAL, ORC_BCAST,   ORC_PARTIAL, ORC_BCAST,   ORC_BCAST,   ORC_PARTIAL}, /* PB  */
        {ORC_BCAST,   ORC_PARTIAL, ORC_PARTIAL, ORC_BCAST,   ORC_PARTIAL, ORC_BCAST  }, /* BP  */
        {ORC_BCAST,   ORC_BCAST,   ORC_BCAST,   ORC_PARTIAL, ORC_PARTIAL, ORC_PARTIAL}, /* BB  */
    };
    static const int32_t A[6][6] = {
        { 0, -1,  0,  0,  0, -1},
        {-1,  1,  1,  1, -1,  1},
        { 1,  0, -1, -1,  1,  0},
        {-1, -1, -1, -1, -1, -1},
        {-1, -1, -1, -1, -1, -1},
        {-1, -1, -1, -1, -1, -1},
    };
    if (sig < 0 || sig > 5) return -1;
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

/* Output shape of op from the operand shares already in pl. */
static void set_out_shape(int op, orc_plan *pl)
{
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
}

static int make_plan(int sig, int op, int64_t M, int64_t K, int64_t N,
                     int64_t p, int64_t r, orc_plan *pl)
{
    int32_t kd[6], ax[6];
    if (orc_tags(sig, kd, ax) != 0) return -1;
    if (op < 0 || op > 2 || p < 1 || r < 0 || r >= p) return -1;
    pl->x = share_of(kd[0], ax[0], M, K, p, r);
    pl->w = share_of(kd[1], ax[1], K, N, p, r);
    pl->dy = share_of(kd[3], ax[3], M, N, p, r);
    set_out_shape(op, pl);
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

/* The same dot product with an fp32 accumulator: c = fl32(c + fl32(a b)) at
 * every step, in increasing reduction index. */
static float element_f32(const orc_plan *pl, int op, int enc, int64_t K, int64_t N,
                         const void *X, const void *W, const void *dY, int64_t i,
                         int64_t j)
{
    float acc = 0.0f;
    if (op == ORC_FWD) {
        for (int64_t t = 0; t < pl->x.nc; ++t) {
            const float a = (float)decode(X, enc, (pl->x.r0 + i) * K + (pl->x.c0 + t));
            const float b = (float)decode(W, enc, (pl->w.r0 + t) * N + (pl->w.c0 + j));
            const float ab = a * b;
            acc = acc + ab;
        }
    } else if (op == ORC_BWD_DATA) {
        for (int64_t t = 0; t < pl->dy.nc; ++t) {
            const float a = (float)decode(dY, enc, (pl->dy.r0 + i) * N + (pl->dy.c0 + t));
            const float b = (float)decode(W, enc, (pl->w.r0 + j) * N + (pl->w.c0 + t));
            const float ab = a * b;
            acc = acc + ab;
        }
    } else {
        for (int64_t t = 0; t < pl->x.nr; ++t) {
            const float a = (float)decode(X, enc, (pl->x.r0 + t) * K + (pl->x.c0 + i));
            const float b = (float)decode(dY, enc, (pl->dy.r0 + t) * N + (pl->dy.c0 + j));
            const float ab = a * b;
            acc = acc + ab;
        }
    }
    return acc;
}

/* Fills block [i0, i1) x [j0, j1) of the output described by pl. */
static int run_block(const orc_plan *pl, int op, int enc, int64_t K, int64_t N,
                     const void *X, const void *W, const void *dY, int64_t i0,
                     int64_t i1, int64_t j0, int64_t j1, double *out)
{
    if (enc != ORC_IN_BF16 && enc != ORC_IN_F32) return -1;
    if (i0 < 0 || j0 < 0 || i1 < i0 || j1 < j0 || i1 > pl->out_rows ||
        j1 > pl->out_cols)
        return -1;
    int64_t w = j1 - j0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = i0; i < i1; ++i)
        for (int64_t j = j0; j < j1; ++j)
            out[(i - i0) * w + (j - j0)] =
                element(pl, op, enc, K, N, X, W, dY, i, j);
    return 0;
}

/* Fills out[s] with element (ii[s], jj[s]) of the output described by pl. */
static int run_samples(const orc_plan *pl, int op, int enc, int64_t K, int64_t N,
                       const void *X, const void *W, const void *dY, int64_t n,
                       const int64_t *ii, const int64_t *jj, double *out)
{
    if (enc != ORC_IN_BF16 && enc != ORC_IN_F32) return -1;
    for (int64_t s = 0; s < n; ++s)
        if (ii[s] < 0 || ii[s] >= pl->out_rows || jj[s] < 0 || jj[s] >= pl->out_cols)
            return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t s = 0; s < n; ++s)
        out[s] = element(pl, op, enc, K, N, X, W, dY, ii[s], jj[s]);
    return 0;
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
    return run_block(&pl, op, enc, K, N, X, W, dY, i0, i1, j0, j1, out);
}

/* As orc_linear_block, accumulating in fp32 (element_f32); out is fp32. */
int orc_linear_block_f32(int sig, int op, int enc, int64_t M, int64_t K, int64_t N,
                         int64_t p, int64_t r, const void *X, const void *W,
                         const void *dY, int64_t i0, int64_t i1, int64_t j0,
                         int64_t j1, float *out)
{
    orc_plan pl;
    if (make_plan(sig, op, M, K, N, p, r, &pl) != 0) return -1;
    if (enc != ORC_IN_BF16 && enc != ORC_IN_F32) return -1;
    if (i0 < 0 || j0 < 0 || i1 < i0 || j1 < j0 || i1 > pl.out_rows || j1 > pl.out_cols)
        return -1;
    int64_t w = j1 - j0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = i0; i < i1; ++i)
        for (int64_t j = j0; j < j1; ++j)
            out[(i - i0) * w + (j - j0)] = element_f32(&pl, op, enc, K, N, X, W, dY, i, j);
    return 0;
}

/* Threads the oracle's parallel loops use (omp_get_max_threads), and a way
 * to change it (for single-thread timings); 1 without OpenMP. */
int orc_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void orc_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* n single elements (ii[s], jj[s]) of rank r's output, as fp64. */
int orc_linear_samples(int sig, int op, int enc, int64_t M, int64_t K,
                       int64_t N, int64_t p, int64_t r, const void *X,
                       const void *W, const void *dY, int64_t n,
                       const int64_t *ii, const int64_t *jj, double *out)
{
    orc_plan pl;
    if (make_plan(sig, op, M, K, N, p, r, &pl) != 0) return -1;
    return run_samples(&pl, op, enc, K, N, X, W, dY, n, ii, jj, out);
}

/* -------------------------------------- nd-SBP on device meshes ------- */
/*
 * On a d-dimensional device mesh (Sec. 4.1, Listing 1: one SBP state per
 * level of the placement hierarchy) a tensor has one state per mesh axis,
 * and a device is named by its mesh coordinate c[0..d-1].
 *
 * Share. The splits nest in mesh-axis order: mesh axis 0 cuts the tensor
 * axis it splits into p[0] balanced blocks and keeps block c[0]; every later
 * mesh axis that splits the same tensor axis cuts the block kept so far
 * with the same balanced rule. Broadcast and Partial-sum axes keep the
 * block. (Reading: the paper gives the composition through shapes only --
 * Listing 1's 2 x 2 blocks -- and writes merged splits as one split over
 * p1*p2; the nesting order makes (S1:p1, S1:p2) the split over p1*p2 with
 * block c1*p2 + c2 whenever p1*p2 divides the extent.)
 *
 * Signature. Each mesh axis carries one 1-D signature of the table above
 * (the 3-D rule of Sec. 4.2 is DP on mesh axis 0, COL on axis 1, KS on
 * axis 2); an axis with X and W both Broadcast replicates the product.
 *
 * Mesh coordinate of a device (Sec. 4.2, heterogeneous networks). Mesh axis
 * a spans nodes[a] nodes x gpus[a] GPUs per node. The node index and the
 * GPU index are each read as mixed-radix numbers with mesh axis 0 as the
 * lowest digit, and c[a] = (node digit a) * gpus[a] + (GPU digit a). The
 * paper's example (S0:(1,2), B:(2,2)) -- split 0 of the data on GPUs
 * (0,0), (0,2), (1,0), (1,2) -- fixes the GPU-level digit order; putting
 * the node digit above the GPU digit within one mesh axis is a reading.
 */
#define ORC_MAXD 4

int orc_mesh_coord(int d, const int32_t *nodes, const int32_t *gpus,
                   int64_t node, int64_t gpu, int32_t *c)
{
    if (d < 1 || d > ORC_MAXD) return -1;
    int64_t node_stride = 1, gpu_stride = 1;
    for (int a = 0; a < d; ++a) {
        if (nodes[a] < 1 || gpus[a] < 1) return -1;
        int64_t n_digit = (node / node_stride) % nodes[a];
        int64_t g_digit = (gpu / gpu_stride) % gpus[a];
        c[a] = (int32_t)(n_digit * gpus[a] + g_digit);
        node_stride *= nodes[a];
        gpu_stride *= gpus[a];
    }
    if (node < 0 || node >= node_stride || gpu < 0 || gpu >= gpu_stride) return -1;
    return 0;
}

/* Factor of one mesh axis from the (kind, axis) states of X and W on it. */
static int axis_factor(int32_t xk, int32_t xa, int32_t wk, int32_t wa)
{
    int32_t kd[6], ax[6];
    for (int sig = 0; sig < 6; ++sig) {
        orc_tags(sig, kd, ax);
        if (kd[0] == xk && ax[0] == xa && kd[1] == wk && ax[1] == wa) return sig;
    }
    return -1;
}

/*
 * Per mesh axis, the (kind, axis) states of X, W, Y, dY, dX, dW for the
 * given states of X and W (d entries each). kinds and axes receive 6*d
 * entries, tensor-major: tensor t on mesh axis a at [t*d + a]. Returns 0, or
 * -1 when some mesh axis carries no factor.
 */
int orc_nd_tags(int d, const int32_t *xk, const int32_t *xa, const int32_t *wk,
                const int32_t *wa, int32_t *kinds, int32_t *axes)
{
    if (d < 1 || d > ORC_MAXD) return -1;
    for (int a = 0; a < d; ++a) {
        int f = axis_factor(xk[a], xa[a], wk[a], wa[a]);
        int32_t kd[6], ax[6];
        if (f < 0) return -1;
        orc_tags(f, kd, ax);
        for (int t = 0; t < 6; ++t) {
            kinds[t * d + a] = kd[t];
            axes[t * d + a] = ax[t];
        }
    }
    return 0;
}

static int valid_mesh(int d, const int32_t *p, const int32_t *c)
{
    if (d < 1 || d > ORC_MAXD) return 0;
    for (int a = 0; a < d; ++a)
        if (p[a] < 1 || c[a] < 0 || c[a] >= p[a]) return 0;
    return 1;
}

/* The device's share of a rows x cols tensor with states (k[a], ax[a]). */
static orc_share nd_share_of(int d, const int32_t *k, const int32_t *ax,
                             const int32_t *p, const int32_t *c, int64_t rows,
                             int64_t cols)
{
    orc_share s = {0, rows, 0, cols};
    for (int a = 0; a < d; ++a) {
        int64_t off, len;
        if (k[a] != ORC_SPLIT) continue;
        if (ax[a] == 0) {
            orc_split(s.nr, p[a], c[a], &off, &len);
            s.r0 += off;
            s.nr = len;
        } else {
            orc_split(s.nc, p[a], c[a], &off, &len);
            s.c0 += off;
            s.nc = len;
        }
    }
    return s;
}

/*
 * Share (row offset, col offset, rows, cols) of a rows x cols tensor in
 * per-axis states (k, ax) for the device at c on mesh p. Returns 0, or -1
 * for a bad mesh, coordinate or state.
 */
int orc_nd_share(int d, const int32_t *k, const int32_t *ax, const int32_t *p,
                 const int32_t *c, int64_t rows, int64_t cols, int64_t out[4])
{
    if (!valid_mesh(d, p, c) || rows < 0 || cols < 0) return -1;
    for (int a = 0; a < d; ++a) {
        if (k[a] == ORC_SPLIT && (ax[a] == 0 || ax[a] == 1)) continue;
        if ((k[a] == ORC_BCAST || k[a] == ORC_PARTIAL) && ax[a] == -1) continue;
        return -1;
    }
    orc_share s = nd_share_of(d, k, ax, p, c, rows, cols);
    out[0] = s.r0;
    out[1] = s.c0;
    out[2] = s.nr;
    out[3] = s.nc;
    return 0;
}

/* Operand shares and output shape of op for the device at c. */
static int make_nd_plan(int op, int64_t M, int64_t K, int64_t N, int d,
                        const int32_t *p, const int32_t *c, const int32_t *xk,
                        const int32_t *xa, const int32_t *wk, const int32_t *wa,
                        orc_plan *pl, int32_t *kinds, int32_t *axes)
{
    if (op < 0 || op > 2 || !valid_mesh(d, p, c)) return -1;
    if (orc_nd_tags(d, xk, xa, wk, wa, kinds, axes) != 0) return -1;
    pl->x = nd_share_of(d, kinds + 0 * d, axes + 0 * d, p, c, M, K);
    pl->w = nd_share_of(d, kinds + 1 * d, axes + 1 * d, p, c, K, N);
    pl->dy = nd_share_of(d, kinds + 3 * d, axes + 3 * d, p, c, M, N);
    set_out_shape(op, pl);
    return 0;
}

/* Output shape of op and its per-axis states (d entries each). */
int orc_nd_out_shape(int op, int64_t M, int64_t K, int64_t N, int d,
                     const int32_t *p, const int32_t *c, const int32_t *xk,
                     const int32_t *xa, const int32_t *wk, const int32_t *wa,
                     int64_t *rows, int64_t *cols, int32_t *kind, int32_t *axis)
{
    orc_plan pl;
    int32_t kinds[6 * ORC_MAXD], axes[6 * ORC_MAXD];
    if (make_nd_plan(op, M, K, N, d, p, c, xk, xa, wk, wa, &pl, kinds, axes) != 0)
        return -1;
    int t = (op == ORC_FWD) ? 2 : (op == ORC_BWD_DATA ? 4 : 5);
    *rows = pl.out_rows;
    *cols = pl.out_cols;
    for (int a = 0; a < d; ++a) {
        kind[a] = kinds[t * d + a];
        axis[a] = axes[t * d + a];
    }
    return 0;
}

/* nd forms of orc_linear_block and orc_linear_samples. */
int orc_nd_linear_block(int op, int enc, int64_t M, int64_t K, int64_t N, int d,
                        const int32_t *p, const int32_t *c, const int32_t *xk,
                        const int32_t *xa, const int32_t *wk, const int32_t *wa,
                        const void *X, const void *W, const void *dY, int64_t i0,
                        int64_t i1, int64_t j0, int64_t j1, double *out)
{
    orc_plan pl;
    int32_t kinds[6 * ORC_MAXD], axes[6 * ORC_MAXD];
    if (make_nd_plan(op, M, K, N, d, p, c, xk, xa, wk, wa, &pl, kinds, axes) != 0)
        return -1;
    return run_block(&pl, op, enc, K, N, X, W, dY, i0, i1, j0, j1, out);
}

int orc_nd_linear_samples(int op, int enc, int64_t M, int64_t K, int64_t N, int d,
                          const int32_t *p, const int32_t *c, const int32_t *xk,
                          const int32_t *xa, const int32_t *wk, const int32_t *wa,
                          const void *X, const void *W, const void *dY, int64_t n,
                          const int64_t *ii, const int64_t *jj, double *out)
{
    orc_plan pl;
    int32_t kinds[6 * ORC_MAXD], axes[6 * ORC_MAXD];
    if (make_nd_plan(op, M, K, N, d, p, c, xk, xa, wk, wa, &pl, kinds, axes) != 0)
        return -1;
    return run_samples(&pl, op, enc, K, N, X, W, dY, n, ii, jj, out);
}

/* ------------------------------ attention core under a head split ----- */
/*
 * Multi-head attention reduces to batched matrix products (Sec. 2). Tensors
 * are contiguous [batch][heads][rows][cols]; with the head dimension split
 * over p devices (the balanced split above) device r holds heads
 * [h0, h0 + hr) of every operand and computes, per batch b and local head
 * h (global head h0 + h), the products below. Outputs are [batch][hr][.][.].
 *
 *   ORC_ATT_S   S[i][j]  = sum_d Q[i][d]  K[j][d]     (scores)
 *   ORC_ATT_O   O[i][d]  = sum_j P[i][j]  V[j][d]     (context)
 *   ORC_ATT_DQ  dQ[i][d] = sum_j dS[i][j] K[j][d]
 *   ORC_ATT_DK  dK[j][d] = sum_i dS[i][j] Q[i][d]
 *   ORC_ATT_DP  dP[i][j] = sum_d dO[i][d] V[j][d]
 *   ORC_ATT_DV  dV[j][d] = sum_i P[i][j]  dO[i][d]
 *
 * Arguments: the two operands in the order written (e.g. dS then K), with
 * sq, sk and d the query length, key length and head dimension.
 */
enum { ORC_ATT_S = 0, ORC_ATT_O = 1, ORC_ATT_DQ = 2, ORC_ATT_DK = 3, ORC_ATT_DP = 4,
       ORC_ATT_DV = 5 };

/* Rows and columns of one output matrix, and the shapes of the operands. */
static int att_shapes(int which, int64_t sq, int64_t sk, int64_t d, int64_t *orow,
                      int64_t *ocol, int64_t *r1, int64_t *c1, int64_t *r2, int64_t *c2)
{
    switch (which) {
    case ORC_ATT_S:  *orow = sq; *ocol = sk; *r1 = sq; *c1 = d;  *r2 = sk; *c2 = d;  return 0;
    case ORC_ATT_O:  *orow = sq; *ocol = d;  *r1 = sq; *c1 = sk; *r2 = sk; *c2 = d;  return 0;
    case ORC_ATT_DQ: *orow = sq; *ocol = d;  *r1 = sq; *c1 = sk; *r2 = sk; *c2 = d;  return 0;
    case ORC_ATT_DK: *orow = sk; *ocol = d;  *r1 = sq; *c1 = sk; *r2 = sq; *c2 = d;  return 0;
    case ORC_ATT_DP: *orow = sq; *ocol = sk; *r1 = sq; *c1 = d;  *r2 = sk; *c2 = d;  return 0;
    case ORC_ATT_DV: *orow = sk; *ocol = d;  *r1 = sq; *c1 = sk; *r2 = sq; *c2 = d;  return 0;
    }
    return -1;
}

int orc_attn(int which, int enc, int64_t nb, int64_t nh, int64_t sq, int64_t sk,
             int64_t d, int64_t p, int64_t r, const void *T1, const void *T2,
             double *out)
{
    int64_t orow, ocol, r1, c1, r2, c2, h0, hr;
    if (att_shapes(which, sq, sk, d, &orow, &ocol, &r1, &c1, &r2, &c2) != 0) return -1;
    if (enc != ORC_IN_BF16 && enc != ORC_IN_F32) return -1;
    if (p < 1 || r < 0 || r >= p || nb < 0 || nh < 0) return -1;
    orc_split(nh, p, r, &h0, &hr);
    const int64_t s1 = r1 * c1, s2 = r2 * c2;   /* elements per (batch, head) matrix */
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t b = 0; b < nb; ++b)
        for (int64_t h = 0; h < hr; ++h) {
            const int64_t m1 = (b * nh + h0 + h) * s1, m2 = (b * nh + h0 + h) * s2;
            double *o = out + (b * hr + h) * orow * ocol;
            for (int64_t i = 0; i < orow; ++i)
                for (int64_t j = 0; j < ocol; ++j) {
                    double acc = 0.0;
                    switch (which) {
                    case ORC_ATT_S:   /* Q[i][t] K[j][t] */
                        for (int64_t t = 0; t < d; ++t)
                            acc += decode(T1, enc, m1 + i * c1 + t) * decode(T2, enc, m2 + j * c2 + t);
                        break;
                    case ORC_ATT_O:   /* P[i][t] V[t][j] */
                    case ORC_ATT_DQ:  /* dS[i][t] K[t][j] */
                        for (int64_t t = 0; t < sk; ++t)
                            acc += decode(T1, enc, m1 + i * c1 + t) * decode(T2, enc, m2 + t * c2 + j);
                        break;
                    case ORC_ATT_DK:  /* dS[t][i] Q[t][j] */
                    case ORC_ATT_DV:  /* P[t][i] dO[t][j] */
                        for (int64_t t = 0; t < sq; ++t)
                            acc += decode(T1, enc, m1 + t * c1 + i) * decode(T2, enc, m2 + t * c2 + j);
                        break;
                    case ORC_ATT_DP:  /* dO[i][t] V[j][t] */
                        for (int64_t t = 0; t < d; ++t)
                            acc += decode(T1, enc, m1 + i * c1 + t) * decode(T2, enc, m2 + j * c2 + t);
                        break;
                    }
                    o[i * ocol + j] = acc;
                }
        }
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
