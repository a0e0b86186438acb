/*
 * sbp.h -- C ABI of the local-shard SBP linear layer for MI355X (gfx950).
 *
 * A linear layer Y = X W under an SBP (Split / Broadcast / Partial-sum)
 * signature runs, on each device, a local matrix product of that device's
 * shares of its operands (AutoDDL, Sec. 4.2, "Distributed Matrix
 * Multiplication based on SBP": the local matmul of the 3-D SBP rule).
 * This library runs rank r's local forward and backward products on one GPU
 * and tags each output with its SBP state.
 *
 * Supported signatures (the 1-D factors of the Sec. 4.2 rule, and three
 * that follow from linearity; a broadcast tensor's gradient is a partial
 * sum, Sec. 4.3 "Sources of Communication", and a partial sum's gradient is
 * broadcast):
 *
 *   name  X      W      -> Y     | dY     dX     dW
 *   DP    S(0)   B      -> S(0)  | S(0)   S(0)   P
 *   COL   B      S(1)   -> S(1)  | S(1)   P      S(1)
 *   KS    S(1)   S(0)   -> P     | B      S(1)   S(0)
 *   PB    P      B      -> P     | B      B      P
 *   BP    B      P      -> P     | B      P      B
 *   BB    B      B      -> B     | P      P      P
 *
 * PB, BP and BB divide no dimension: every device multiplies full-size
 * operands (its own partial of a P operand).
 *
 * Conventions (all functions):
 *   - Matrices are row-major with a leading dimension ld (elements between
 *     the starts of consecutive rows, ld >= cols). X is M x K, W is K x N,
 *     dY and Y are M x N, as global tensors.
 *   - Split(i) over p devices gives rank r the contiguous block
 *     [off, off + len) of axis i with len = D/p + (r < D%p), off =
 *     r*(D/p) + min(r, D%p) (the paper does not fix uneven splits; this is
 *     the balanced reading). Broadcast and Partial-sum shares span the full
 *     extent.
 *   - Every pointer in an sbp_view_t is a DEVICE pointer on the current HIP
 *     device. The caller owns every buffer; the library never copies inputs.
 *   - Return value: SBP_OK (0) or a negative SBP_ERR_* code. Every check
 *     except SBP_ERR_HIP happens on the host before any HIP call, so a
 *     rejected call has no effect on the device.
 *   - Compute calls are asynchronous on the given stream (0 = the null
 *     stream) and never synchronise. Inputs must stay valid, and outputs
 *     untouched, until the stream has run the call.
 *   - Memory: the library allocates nothing and keeps no device state.
 *     The linear calls take a caller-owned workspace (sbp_workspace_t) for
 *     the fp32 partials of split reductions; see below. Every call can be
 *     captured into a HIP graph, including the first on a stream.
 *   - Thread safety: calls on different host threads are safe. Two calls
 *     may share a workspace only if they cannot run at the same time (e.g.
 *     they are on the same stream).
 */
#ifndef SBP_H
#define SBP_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ codes --- */
enum {
    SBP_OK = 0,
    SBP_ERR_NULL = -1,      /* a required pointer is NULL                       */
    SBP_ERR_LAYOUT = -2,    /* p < 1, r outside [0,p), bad kind/axis, or layouts
                               of one call disagree on p or r                    */
    SBP_ERR_SIGNATURE = -3, /* the input states form no supported signature     */
    SBP_ERR_SHAPE = -4,     /* inner dimensions disagree, ld < cols, a negative
                               or > 2^31-1 extent, or the output view is not the
                               local output shape                               */
    SBP_ERR_DTYPE = -5,     /* unknown dtype, inputs of mixed dtype, a
                               Partial-sum output that is not fp32, or a bf16
                               output of fp32 inputs                            */
    SBP_ERR_ALIAS = -6,     /* the output's memory overlaps an input's          */
    SBP_ERR_ALIGN = -7,     /* a data pointer is not aligned to its element size */
    SBP_ERR_HIP = -8,       /* a HIP call failed; see sbp_last_hip_error()      */
    SBP_ERR_WORKSPACE = -9  /* the split partials of the call's plan do not fit
                               the workspace it runs with                       */
};

/* ------------------------------------------------------------ types --- */
typedef enum { SBP_SPLIT = 0, SBP_BROADCAST = 1, SBP_PARTIAL = 2 } sbp_kind_t;

/* SBP state of a tensor on a 1-D mesh of p devices, seen from rank r.
 * axis is 0 or 1 for SBP_SPLIT and -1 otherwise. */
typedef struct {
    int32_t kind;
    int32_t axis;
    int32_t p;
    int32_t r;
} sbp_layout_t;

typedef enum { SBP_BF16 = 0, SBP_F32 = 1 } sbp_dtype_t;

/* SBP_GLOBAL: the view spans the whole global tensor and the library selects
 * rank r's share inside it (a strided sub-view, never a copy).
 * SBP_LOCAL: the view is exactly rank r's share.
 * SBP_ACCUMULATE (outputs only): the call adds its product to the output's
 * current contents instead of overwriting them -- gradient accumulation
 * over micro-batches (Sec. 5 splits each mini-batch into micro-batches and
 * accumulates their gradients). The output must be fp32 (else
 * SBP_ERR_DTYPE); each element becomes old + product with one fp32
 * rounding (the product itself summed in fp32 first). */
typedef enum { SBP_GLOBAL = 0, SBP_LOCAL = 1, SBP_ACCUMULATE = 2 } sbp_scope_t;

/* A strided 2-D view: element (i, j) is at data + i*ld + j (elements). */
typedef struct {
    void *data;
    int64_t rows;
    int64_t cols;
    int64_t ld;
    int32_t dtype; /* sbp_dtype_t */
    int32_t scope; /* sbp_scope_t; outputs are always local: SBP_ACCUMULATE
                      adds to them, any other value overwrites them */
} sbp_view_t;

/* Caller-owned device memory for split reductions. A product with a long
 * reduction and few output tiles runs faster with its reduction split over
 * several workgroups; each split writes an fp32 partial of the m x n output
 * (rows padded to a multiple of 4 floats: splits x m x 4 ceil(n / 4) x 4
 * bytes in all) that a second kernel adds up in split order. The linear calls take a workspace; data = NULL (or bytes = 0, or a
 * NULL sbp_workspace_t pointer) means none, and then no reduction is split.
 * With bytes >= SBP_WORKSPACE_BYTES every call gets the library's preferred
 * plan; a smaller workspace limits the splits to what fits (results are the
 * same up to fp32 summation order; identical for identical workspace
 * sizes). The library never reads the workspace's contents before writing
 * them, so it needs no clearing. data must be 16-byte aligned (else
 * SBP_ERR_ALIGN), must not overlap the call's inputs or outputs (else
 * SBP_ERR_ALIAS), and must not be used by another call at the same time. */
typedef struct {
    void *data;    /* device pointer on the current device, or NULL */
    int64_t bytes; /* its size in bytes (>= 0, else SBP_ERR_SHAPE)   */
} sbp_workspace_t;

#define SBP_WORKSPACE_BYTES ((int64_t)64 << 20)

/* Rank r's share of a tensor: rows [row_off, row_off+rows) x cols
 * [col_off, col_off+cols) of the global tensor. */
typedef struct {
    int64_t row_off;
    int64_t col_off;
    int64_t rows;
    int64_t cols;
} sbp_shard_t;

/* ------------------------------------------------------- host logic --- */

/* Rank l->r's share of a rows x cols tensor in state *l (Sec. 4.1: Split,
 * Broadcast and Partial-sum states; Fig. 5). Pure host function.
 * Errors: SBP_ERR_NULL, SBP_ERR_LAYOUT, SBP_ERR_SHAPE (negative extent). */
int sbp_shard_index(const sbp_layout_t *l, int64_t rows, int64_t cols,
                    sbp_shard_t *out);

/* Resolves the signature of Y = X W from the states of X and W (Sec. 4.2)
 * and writes the states of Y, dY, dX and dW (Sec. 4.3: a broadcast operand's
 * gradient is a partial sum; a split operand's gradient is split the same
 * way). Any of y, dy, dx, dw may be NULL. Pure host function.
 * Errors: SBP_ERR_NULL (x or w), SBP_ERR_LAYOUT, SBP_ERR_SIGNATURE. */
int sbp_signature(const sbp_layout_t *x, const sbp_layout_t *w,
                  sbp_layout_t *y, sbp_layout_t *dy, sbp_layout_t *dx,
                  sbp_layout_t *dw);

/* ----------------------------------------------------- device compute --- */

/* Forward local matmul Y_r = X_r W_r (Sec. 4.2, "local matmul").
 * X: M x K (or rank r's share), state *lx; W: K x N (or share), state *lw.
 * Y: rank r's local output, state written to *ly_out (may be NULL):
 *    DP m_r x N, COL M x n_r, KS M x N (Partial-sum, must be fp32);
 *    PB and BP M x N (Partial-sum, fp32), BB M x N (Broadcast).
 * Inputs bf16 or fp32 (same dtype); Y is fp32, or bf16 for bf16 inputs and
 * a Split/Broadcast output (rounded to nearest even from the fp32
 * accumulator). ws: workspace for a split reduction (may be NULL; see
 * sbp_workspace_t). */
int sbp_linear_fwd(const sbp_view_t *X, const sbp_layout_t *lx,
                   const sbp_view_t *W, const sbp_layout_t *lw, sbp_view_t *Y,
                   sbp_layout_t *ly_out, const sbp_workspace_t *ws,
                   hipStream_t stream);

/* Backward-data local matmul dX_r = dY_r W_r^T (Sec. 4.2: the redistributions
 * of the forward path have backward counterparts; Sec. 4.3).
 * dY: state *ldy (S(0) for DP, S(1) for COL, B for KS, PB and BP, P for
 *     BB); W: state *lw.
 * dX: rank r's local output, state to *ldx_out: DP m_r x K (S(0)),
 *     COL M x K (Partial-sum, fp32), KS M x k_r (S(1)); PB M x K (B), BP
 *     and BB M x K (Partial-sum, fp32).
 * ws as for sbp_linear_fwd. */
int sbp_linear_bwd_data(const sbp_view_t *dY, const sbp_layout_t *ldy,
                        const sbp_view_t *W, const sbp_layout_t *lw,
                        sbp_view_t *dX, sbp_layout_t *ldx_out,
                        const sbp_workspace_t *ws, hipStream_t stream);

/* Backward-weight local matmul dW_r = X_r^T dY_r (Sec. 4.3: a broadcast
 * weight receives partial-sum gradients).
 * X: state *lx; dY: state *ldy.
 * dW: rank r's local output, state to *ldw_out: DP K x N (Partial-sum,
 *     fp32), COL K x n_r (S(1)), KS k_r x N (S(0)); PB and BB K x N
 *     (Partial-sum, fp32), BP K x N (B).
 * ws as for sbp_linear_fwd. */
int sbp_linear_bwd_weight(const sbp_view_t *X, const sbp_layout_t *lx,
                          const sbp_view_t *dY, const sbp_layout_t *ldy,
                          sbp_view_t *dW, sbp_layout_t *ldw_out,
                          const sbp_workspace_t *ws, hipStream_t stream);

/* Both backward products of the linear, dX_r = dY_r W_r^T and
 * dW_r = X_r^T dY_r, in one call (one grouped launch when the planner
 * expects it to pay, else the two products in turn on `stream`). The two
 * products are independent -- each reads dY and one of X, W (Sec. 4.2
 * backward path, Sec. 4.3 gradient states) -- so in a grouped launch the
 * longer work items of one run while the shorter ones of the other fill the
 * remaining compute units. States, shapes, dtype rules and errors are those
 * of sbp_linear_bwd_data and sbp_linear_bwd_weight; the three input states
 * must form one signature (else SBP_ERR_SIGNATURE), and dX and dW must not
 * overlap (SBP_ERR_ALIAS). Results equal the two separate calls up to fp32
 * summation order. ws as for sbp_linear_fwd: a grouped launch holds the
 * partials of both products in it at once, two separate launches use it in
 * turn. */
int sbp_linear_bwd(const sbp_view_t *dY, const sbp_layout_t *ldy,
                   const sbp_view_t *X, const sbp_layout_t *lx,
                   const sbp_view_t *W, const sbp_layout_t *lw, sbp_view_t *dX,
                   sbp_layout_t *ldx_out, sbp_view_t *dW, sbp_layout_t *ldw_out,
                   const sbp_workspace_t *ws, hipStream_t stream);

/* For callers that cannot allocate device memory -- code being captured
 * into a HIP graph, tight serving loops, harnesses that forbid hipMalloc --
 * and so cannot bring a workspace: sbp_linear_bwd with the library's own
 * scratch in place of a caller workspace. The scratch is a static device
 * array of SBP_WORKSPACE_BYTES on each device (so the plans, kernels and
 * results are those of sbp_linear_bwd with a workspace of that size),
 * placed when the library's code is loaded on the device and held until
 * the process ends; the call itself allocates nothing, and neither does any
 * library routine it uses. A plan whose partials would not fit the scratch
 * is refused with SBP_ERR_WORKSPACE (plans are limited to it, so none
 * does). The scratch keeps the last call's partials; nothing in it needs
 * clearing, since every partial is written before it is read. Every call on
 * one device shares that device's scratch: calls that may overlap in time on
 * one device (different streams, host threads or processes sharing the
 * device's code object) race on it and must be ordered by the caller, e.g.
 * by issuing them on one stream. Arguments, states and errors are those of
 * sbp_linear_bwd. */
int sbp_linear_bwd_noalloc(const sbp_view_t *dY, const sbp_layout_t *ldy,
                           const sbp_view_t *X, const sbp_layout_t *lx,
                           const sbp_view_t *W, const sbp_layout_t *lw,
                           sbp_view_t *dX, sbp_layout_t *ldx_out, sbp_view_t *dW,
                           sbp_layout_t *ldw_out, hipStream_t stream);

/* ------------------------------------------- nd-SBP on device meshes --- */

/* Mesh axes an nd layout may have. */
#define SBP_MAX_MESH_DIMS 4

/* SBP state of a tensor on a d-dimensional device mesh, seen from the
 * device at mesh coordinate c: one Split / Broadcast / Partial-sum state
 * per mesh axis (Sec. 4.1, Listing 1: a placement hierarchy such as
 * (2, 3, 4) with one state per hierarchy level; Sec. 4.2: the 3-D rule
 * (S0:p0, B:p1, S1:p2) x (B:p0, S1:p1, S0:p2) -> (S0:p0, S1:p1, P:p2)).
 *   ndim     mesh axes d, 1..SBP_MAX_MESH_DIMS; entries a >= d are ignored
 *   kind[a]  sbp_kind_t on mesh axis a
 *   axis[a]  tensor axis (0 or 1) for SBP_SPLIT, else -1
 *   p[a]     devices along mesh axis a (>= 1)
 *   c[a]     this device's coordinate along mesh axis a, in [0, p[a])
 * The share of a tensor nests the splits in mesh-axis order: mesh axis 0
 * cuts the full extent into p[0] balanced blocks (the 1-D rule above), mesh
 * axis 1 cuts block c[0] into p[1] blocks, and so on; each tensor axis is cut
 * only by the mesh axes that split it. Broadcast and Partial-sum axes do not
 * cut. A 1-D layout (kind, axis, p, r) is the nd layout with d = 1,
 * c[0] = r. */
typedef struct {
    int32_t ndim;
    int32_t kind[SBP_MAX_MESH_DIMS];
    int32_t axis[SBP_MAX_MESH_DIMS];
    int32_t p[SBP_MAX_MESH_DIMS];
    int32_t c[SBP_MAX_MESH_DIMS];
} sbp_nd_layout_t;

/* Mesh coordinate of a device (Sec. 4.2, "Strategies for heterogeneous
 * interconnected networks"). Mesh axis a spans nodes[a] x gpus[a] devices:
 * nodes[a] compute nodes times gpus[a] GPUs of each node. Device (node, gpu)
 * -- node in [0, prod nodes), gpu in [0, prod gpus) -- has node-level digits
 * n_a and GPU-level digits g_a, both mixed-radix with mesh axis 0 varying
 * fastest (node = n_0 + nodes[0] (n_1 + nodes[1] (...)), likewise gpu), and
 * coordinate c[a] = n_a * gpus[a] + g_a. The paper's example
 * (S0:(1,2), B:(2,2)) on 2 nodes of 4 GPUs puts split 0 on GPUs (0,0),
 * (0,2), (1,0), (1,2): mesh axis 0 varies fastest within a node. For a
 * single-level mesh pass gpus = NULL (all 1) and the device rank as node.
 * Pure host function. Errors: SBP_ERR_NULL (nodes or c), SBP_ERR_LAYOUT
 * (ndim outside [1, SBP_MAX_MESH_DIMS], a factor < 1, or node / gpu outside
 * its range). */
int sbp_mesh_coords(int32_t ndim, const int32_t *nodes, const int32_t *gpus,
                    int64_t node, int64_t gpu, int32_t *c);

/* The device's share of a rows x cols tensor in nd state *l (nested splits,
 * as described at sbp_nd_layout_t). Pure host function.
 * Errors: SBP_ERR_NULL, SBP_ERR_LAYOUT (bad ndim, p, c, kind or axis),
 * SBP_ERR_SHAPE (negative extent). */
int sbp_nd_shard_index(const sbp_nd_layout_t *l, int64_t rows, int64_t cols,
                       sbp_shard_t *out);

/* Resolves the nd signature of Y = X W (Sec. 4.2: the 3-D rule factors
 * into one 1-D signature per mesh axis) and writes the nd states of Y, dY,
 * dX and dW (Sec. 4.3 gradient states, per axis). Each mesh axis must carry
 * one of the 1-D signatures of the table at the top of this file; an axis
 * with X and W both Broadcast (BB) replicates the product, and the
 * gradients are partial sums on it. The layouts must agree on ndim, p and
 * c. Any of y, dy, dx, dw may be NULL. Pure host function.
 * Errors: SBP_ERR_NULL (x or w), SBP_ERR_LAYOUT, SBP_ERR_SIGNATURE. */
int sbp_nd_signature(const sbp_nd_layout_t *x, const sbp_nd_layout_t *w,
                     sbp_nd_layout_t *y, sbp_nd_layout_t *dy,
                     sbp_nd_layout_t *dx, sbp_nd_layout_t *dw);

/* nd forms of the four compute calls: the device's local products on its
 * nd shares, on the same kernels. Views, dtypes, scopes, workspaces, streams
 * and errors are those of the 1-D calls, with nd layouts in place of 1-D ones (all
 * layouts of one call agree on ndim, p and c, else SBP_ERR_LAYOUT).
 * Local output shapes: X_r is the nd share of X, and so on; Y_r = X_r W_r,
 * dX_r = dY_r W_r^T, dW_r = X_r^T dY_r. An output is Partial-sum -- and must
 * be fp32 -- when any mesh axis leaves it Partial-sum (Y under a KS, PB or
 * BP axis, dX under a COL, BP or BB axis, dW under a DP, PB or BB axis). */
int sbp_nd_linear_fwd(const sbp_view_t *X, const sbp_nd_layout_t *lx,
                      const sbp_view_t *W, const sbp_nd_layout_t *lw,
                      sbp_view_t *Y, sbp_nd_layout_t *ly_out,
                      const sbp_workspace_t *ws, hipStream_t stream);
int sbp_nd_linear_bwd_data(const sbp_view_t *dY, const sbp_nd_layout_t *ldy,
                           const sbp_view_t *W, const sbp_nd_layout_t *lw,
                           sbp_view_t *dX, sbp_nd_layout_t *ldx_out,
                           const sbp_workspace_t *ws, hipStream_t stream);
int sbp_nd_linear_bwd_weight(const sbp_view_t *X, const sbp_nd_layout_t *lx,
                             const sbp_view_t *dY, const sbp_nd_layout_t *ldy,
                             sbp_view_t *dW, sbp_nd_layout_t *ldw_out,
                             const sbp_workspace_t *ws, hipStream_t stream);
int sbp_nd_linear_bwd(const sbp_view_t *dY, const sbp_nd_layout_t *ldy,
                      const sbp_view_t *X, const sbp_nd_layout_t *lx,
                      const sbp_view_t *W, const sbp_nd_layout_t *lw,
                      sbp_view_t *dX, sbp_nd_layout_t *ldx_out,
                      sbp_view_t *dW, sbp_nd_layout_t *ldw_out,
                      const sbp_workspace_t *ws, hipStream_t stream);

/* ------------------------------ attention core under a head split --- */

/* A strided 4-D view [batch][heads][rows][cols]: element (b, h, i, j) is at
 * data + b*stride_b + h*stride_h + i*ld + j (elements). Views into a fused
 * activation -- e.g. the Q, K or V part of a QKV projection output laid out
 * [batch][seq][3][heads][head_dim] -- have stride_h = head_dim and ld =
 * 3*heads*head_dim. scope: SBP_GLOBAL (inputs) -- heads counts all H heads
 * and the call takes rank r's heads; SBP_LOCAL -- heads counts rank r's
 * heads only; outputs always hold rank r's heads (SBP_ACCUMULATE adds to an
 * fp32 output, as for the 2-D calls). */
typedef struct {
    void *data;
    int64_t batch, heads, rows, cols;
    int64_t stride_b, stride_h, ld;
    int32_t dtype; /* sbp_dtype_t */
    int32_t scope; /* sbp_scope_t */
} sbp_view4_t;

/* Multi-head attention reduces to batched matrix products (Sec. 2). Under a
 * split of the head dimension over p devices (heads split(H, p, r), the
 * balanced rule), every operand and output is Split on heads and each
 * device multiplies its own heads: one product per (batch, local head), no
 * partial sums. Inputs are bf16 (SBP_ERR_DTYPE otherwise); outputs bf16
 * (rounded to nearest even) or fp32. Softmax, its scale and masking are not
 * part of these calls.
 *
 *   sbp_attn_scores       S  = Q K^T    Q: [B][H][Sq][D], K: [B][H][Sk][D]
 *                                       -> S: [B][H_r][Sq][Sk]
 *   sbp_attn_context      O  = P V      P: [B][H][Sq][Sk], V: [B][H][Sk][D]
 *                                       -> O: [B][H_r][Sq][D]
 *   sbp_attn_scores_bwd   dQ = dS K, dK = dS^T Q (dS like S; dQ like Q, dK
 *                         like K, each over rank r's heads)
 *   sbp_attn_context_bwd  dP = dO V^T, dV = P^T dO (dO like O; dP like P, dV
 *                         like V)
 *
 * Errors: SBP_ERR_NULL, SBP_ERR_LAYOUT (p < 1 or r outside [0, p)),
 * SBP_ERR_SHAPE (extents that disagree, ld < cols, a negative or too large
 * extent or stride, an output whose elements overlap one another, or an
 * output of the wrong shape), SBP_ERR_DTYPE, SBP_ERR_ALIGN, SBP_ERR_ALIAS
 * (an output's span overlaps an input's or the other output's span),
 * SBP_ERR_HIP. Batched products never split their reduction, so these calls
 * take no workspace. */
int sbp_attn_scores(const sbp_view4_t *Q, const sbp_view4_t *K, sbp_view4_t *S,
                    int32_t p, int32_t r, hipStream_t stream);
int sbp_attn_context(const sbp_view4_t *P, const sbp_view4_t *V, sbp_view4_t *O,
                     int32_t p, int32_t r, hipStream_t stream);
int sbp_attn_scores_bwd(const sbp_view4_t *dS, const sbp_view4_t *Q,
                        const sbp_view4_t *K, sbp_view4_t *dQ, sbp_view4_t *dK,
                        int32_t p, int32_t r, hipStream_t stream);
int sbp_attn_context_bwd(const sbp_view4_t *dO, const sbp_view4_t *P,
                         const sbp_view4_t *V, sbp_view4_t *dP, sbp_view4_t *dV,
                         int32_t p, int32_t r, hipStream_t stream);

/* ------------------------------------- cost model and strategy search --- */

/* Collectives of the alpha-beta model (Sec. 3.1, Table 2). */
enum {
    SBP_COLL_ALLREDUCE = 0,      /* (2p-1) alpha + 2 (p-1)/p n beta          */
    SBP_COLL_ALLGATHER = 1,      /* (p-1) alpha + (p-1)/p n beta             */
    SBP_COLL_REDUCESCATTER = 2,  /* (p-1) alpha + (p-1)/p n beta             */
    SBP_COLL_ALLTOALL = 3        /* (p-1) alpha + n beta                     */
};

/* Time of one collective over p devices for an n-byte message (the input
 * of ReduceScatter, the output of the others, per device), latency alpha
 * (seconds) and inverse bandwidth beta (seconds per byte): the formulas of
 * Table 2 as printed. Pure host function. Errors: SBP_ERR_NULL,
 * SBP_ERR_LAYOUT (p < 1, unknown collective), SBP_ERR_SHAPE (negative n,
 * alpha or beta). */
int sbp_collective_cost(int32_t coll, int32_t p, double n, double alpha, double beta,
                        double *cost);

/* Time to redistribute a tensor of `bytes` (global size) from 1-D state
 * *from to 1-D state *to on the same p devices (Sec. 4.2 redistributions,
 * Sec. 4.3 "Sources of Communication"): S(i)->S(j), i != j: AlltoAll of
 * bytes/p; S->B: AllGather of bytes; P->S: ReduceScatter of bytes; P->B:
 * AllReduce of bytes; every other change (B->S, B->P, S->P) and no change:
 * 0 (local). *coll_out, if not NULL, receives the collective used, or -1.
 * Errors: SBP_ERR_NULL, SBP_ERR_LAYOUT (bad states, p mismatch),
 * SBP_ERR_SHAPE. */
int sbp_boxing_cost(const sbp_layout_t *from, const sbp_layout_t *to, double bytes,
                    double alpha, double beta, double *cost, int32_t *coll_out);

/* Signature ids for the search: the rows of the table at the top of this
 * file, in order. */
enum { SBP_SIG_DP = 0, SBP_SIG_COL = 1, SBP_SIG_KS = 2, SBP_SIG_PB = 3, SBP_SIG_BP = 4,
       SBP_SIG_BB = 5 };

/* A chain of linear layers Y_l = X_l W_l (X_l: M x K[l], W_l: K[l] x N[l])
 * on a 1-D mesh of p devices, one signature per layer. Between layers the
 * previous output (M x N[l] elements; M is the same for every layer) is
 * redistributed from layer l's output state to layer l+1's input state; an
 * op between the two (an activation function, the attention core, which
 * maps 3 x hidden to hidden columns) keeps the state, so K[l+1] may differ
 * from N[l]. The network input (M x K[0]) starts in state (in_kind,
 * in_axis) and the last output must end in (out_kind, out_axis). A
 * Partial-sum output is never fed on as is (a nonlinearity separates the
 * layers), so signatures with a Partial-sum X (PB) are not allowed. */
typedef struct {
    int32_t layers;
    int32_t p;
    double alpha, beta;          /* seconds, seconds per byte */
    const int64_t *M, *K, *N;    /* per layer */
    double act_bytes;            /* bytes per activation element */
    double grad_bytes;           /* bytes per weight-gradient element */
    int32_t in_kind, in_axis, out_kind, out_axis;
    uint32_t allowed;            /* bit s: signature s may be chosen */
} sbp_chain_t;

/* Communication time of one training step of the chain under signatures
 * sigs[0..layers): for every activation redistribution, its forward cost
 * plus the backward cost of moving the gradient the other way (the dual
 * states: grad of S(i) is S(i), of B is P, of P is B), plus an AllReduce of
 * every weight gradient left Partial-sum (Sec. 4.3). Pure host function.
 * Errors: SBP_ERR_NULL, SBP_ERR_SHAPE (layers < 1, extents), SBP_ERR_LAYOUT
 * (p, boundary states), SBP_ERR_SIGNATURE (a signature not allowed). */
int sbp_chain_cost(const sbp_chain_t *net, const int32_t *sigs, double *cost);

/* Coordinate-descent search (Sec. 4.4): from an initial guess, each sweep
 * sets every layer in turn to the allowed signature that minimises the
 * chain cost with the others fixed (a change only on strict improvement, so
 * the cost never rises); at a fixed point the run restarts from a new
 * random guess, and the best strategy of `restarts` runs (>= 1; the first
 * starts from all-DP where allowed) is returned in sigs_out with its cost.
 * sweep_costs (may be NULL) receives, run after run, each run's starting
 * cost followed by its cost after every sweep, up to max_sweeps entries;
 * within a run the values strictly decrease until the final sweep, which
 * changes nothing and repeats the previous value. *sweeps_out (may be
 * NULL) receives the total count of entries.
 * Random guesses come from splitmix64 seeded with `seed`. Pure host
 * function. Errors: those of sbp_chain_cost, SBP_ERR_SHAPE (restarts < 1). */
int sbp_search_strategy(const sbp_chain_t *net, int32_t restarts, uint64_t seed,
                        int32_t *sigs_out, double *cost_out, double *sweep_costs,
                        int32_t max_sweeps, int32_t *sweeps_out);

/* --------------------------------------------------------- utilities --- */

/* Static description of an error code (never NULL). */
const char *sbp_strerror(int code);

/* hipError_t of the last SBP_ERR_HIP returned on the calling thread
 * (0 if none). */
int sbp_last_hip_error(void);

/* Kernel plan the library would use for a local product of m x n outputs
 * over a reduction of k with 16-byte aligned operands and tight leading
 * dimensions, for input dtype in_dtype, output dtype out_dtype and operand
 * orientation op (0 forward, 1 backward-data, 2 backward-weight). Writes
 * the tile rows and columns, the number of reduction splits and the kernel
 * (3 fp32, else the bf16 instance code of sbp_set_plan_override), as
 * planned with a workspace of SBP_WORKSPACE_BYTES. For benchmarks and
 * tests; pure host function.
 * Errors: SBP_ERR_NULL, SBP_ERR_SHAPE, SBP_ERR_DTYPE. */
int sbp_plan(int op, int64_t m, int64_t n, int64_t k, int32_t in_dtype,
             int32_t out_dtype, int32_t *tile_m, int32_t *tile_n,
             int32_t *splits, int32_t *kernel);

/* Plan of sbp_linear_bwd for bf16 inputs with 16-byte aligned operands and
 * tight leading dimensions: the backward-data product is md x nd over a
 * reduction of kd with output dtype out_d, the backward-weight product
 * mw x nw over kw with out_w. Writes whether both run as one grouped launch,
 * the tile of the backward-data product (shared when grouped), and the
 * splits of each product, as planned with a workspace of
 * SBP_WORKSPACE_BYTES. Pure host function. Errors: SBP_ERR_NULL, SBP_ERR_SHAPE, SBP_ERR_DTYPE. */
int sbp_plan_bwd(int64_t md, int64_t nd, int64_t kd, int32_t out_d, int64_t mw,
                 int64_t nw, int64_t kw, int32_t out_w, int32_t *grouped,
                 int32_t *tile_m, int32_t *tile_n, int32_t *splits_d,
                 int32_t *splits_w);

/* Per-kernel timing for benchmarks. After sbp_profile_begin(capacity), the
 * first `capacity` kernels that the library launches from the calling
 * thread are each bracketed by a HIP event pair recorded with the dispatch
 * itself (hipExtLaunchKernelGGL). sbp_profile_end stops recording, waits for
 * those events, writes each kernel's duration in microseconds to us[i] and
 * its name (NUL-terminated, at most name_len bytes) to names + i*name_len
 * (either may be NULL), and returns the number of kernels recorded, or
 * SBP_ERR_HIP. Not for use while a stream is being captured into a graph. */
int sbp_profile_begin(int capacity);
int sbp_profile_end(float *us, char *names, int name_len);

/* Thread-local override of the bf16 plan for subsequent calls on this
 * thread (tests and tuning). tile_m x tile_n is one of 256x256, 256x192,
 * 256x128, 128x256, 128x128, 128x64, 64x128, 64x64; splits >= 1. kernel
 * selects the instance:
 *   0, 1  the tile's default pipelined direct-to-LDS instance (256x192:
 *         eight waves as 4 x 2, two stages; as many 256 x 192 tiles as
 *         compute units for a 4096 x 3072 output);
 *   2     the generic kernel;
 *   4     pipelined with two stages (128x128, 128x64, 64x128, 64x64: two or
 *         more workgroups per compute unit);
 *   5     pipelined, eight waves in two reduction groups, output staged in
 *         LDS (256x128, 128x256, 128x128, 128x64, 64x128, 64x64);
 *   6     pipelined, row-quad epilogue: MFMA operands swapped so each lane
 *         stores 4 consecutive outputs of a row from registers (256x256, and
 *         128x128 with two stages);
 *   7     as 5 with the row-quad epilogue (256x128, 128x256, 128x128, 128x64,
 *         64x128, 64x64);
 *   8     pipelined with 32-wide reduction stages, five in LDS (256x256);
 *   9     as 5 with 32-wide reduction stages, six (256x128, 128x256) or
 *         eight (128x128) in LDS;
 *   10    as 5 with two stages, two workgroups per compute unit (128x128);
 *   11    pipelined with deep prefetch for operand streams that HBM latency
 *         bounds: six stages (128x64, 64x128) or eight (64x64) in LDS;
 *   12    as 5 with 128-wide reduction stages, two (128x128), three
 *         (128x64, 64x128) or four (64x64) in LDS: half the barriers and
 *         twice the bytes per operand row of 64-wide stages;
 *   13    as 12 with the row-quad epilogue.
 * wgs_per_cu > 0 makes the launch persistent: at most wgs_per_cu workgroups
 * per compute unit, each taking every G-th work item (0 = one workgroup per
 * item; the grouped backward launch always runs one per item). A call whose
 * operands the pipelined kernel cannot read runs the generic kernel, where
 * 256x256 and 256x192 become 256x128; splits are clamped to the reduction
 * blocks and to the call's workspace. tile_m = 0 clears the override.
 * Errors: SBP_ERR_SHAPE for a (tile, kernel) pair not listed above,
 * splits < 1, or wgs_per_cu outside [0, 8]. */
int sbp_set_plan_override(int32_t tile_m, int32_t tile_n, int32_t splits,
                          int32_t kernel, int32_t wgs_per_cu);

/* Thread-local choice of how sbp_linear_bwd runs its two products (tuning):
 * mode 0 = the library's choice, 1 = two launches, one per product, 2 = one
 * grouped launch on the tile and kernel of sbp_set_plan_override (which must
 * be set, else mode 2 acts as 0), with that override's splits for the
 * backward-data product and splits_w for the backward-weight product.
 * Clearing the plan override (tile_m = 0) also resets this to mode 0.
 * Errors: SBP_ERR_SHAPE for a mode outside [0, 2] or splits_w < 1. */
int sbp_set_bwd_override(int32_t mode, int32_t splits_w);

/* Restricts the plan override of sbp_set_plan_override to the products of
 * the orientations in mask (bit 0 forward / Y = X W, bit 1 backward-data /
 * A B^T, bit 2 backward-weight / A^T B); the others keep their own plans
 * (tuning one product of a two-product call). Clearing the plan override
 * (tile_m = 0) resets the mask to 7. Errors: SBP_ERR_SHAPE for a mask
 * outside [1, 7]. */
int sbp_set_override_orients(int32_t mask);

#ifdef __cplusplus
}
#endif

#endif /* SBP_H */
