"""Rank-r local products of one SBP linear, from torch tensors.

Convenience over the binding: picks the input states of a named signature,
asks the library for the output states (``sbp_signature``) and local output
shape (``sbp_shard_index``), allocates the output and calls the entry point.
All computation happens in libsbp.so.

Signatures are the 1-D factors of AutoDDL's SBP matmul (Sec. 4.2):
DP (S(0),B)->S(0), COL (B,S(1))->S(1), KS (S(1),S(0))->P, and by linearity
PB (P,B)->P, BP (B,P)->P, BB (B,B)->B. On a device mesh an nd signature is
one of them per mesh axis (the 3-D rule of Sec. 4.2 is ("DP", "COL", "KS"));
the ``*_nd`` functions take (factors, mesh, coord).
"""
from __future__ import annotations

import torch

from . import sbp

OPS = ("fwd", "bwd_data", "bwd_weight")


def input_layouts(sig: str, p: int, r: int):
    """States of X and W under signature sig."""
    if sig == "DP":
        return sbp.split(0, p, r), sbp.broadcast(p, r)
    if sig == "COL":
        return sbp.broadcast(p, r), sbp.split(1, p, r)
    if sig == "KS":
        return sbp.split(1, p, r), sbp.split(0, p, r)
    if sig == "PB":
        return sbp.partial(p, r), sbp.broadcast(p, r)
    if sig == "BP":
        return sbp.broadcast(p, r), sbp.partial(p, r)
    if sig == "BB":
        return sbp.broadcast(p, r), sbp.broadcast(p, r)
    raise ValueError("unknown signature %r" % sig)


def layouts(sig: str, p: int, r: int) -> dict:
    x, w = input_layouts(sig, p, r)
    y, dy, dx, dw = sbp.sbp_signature(x, w)
    return {"x": x, "w": w, "y": y, "dy": dy, "dx": dx, "dw": dw}


def layouts_for(lin, wl, r) -> dict:
    """States of one linear of a workload on rank r (for a mesh workload, r
    is the device's mesh coordinate)."""
    if wl.mesh:
        return nd_layouts(lin.factors, wl.mesh, r)
    return layouts(lin.sig, wl.p, r)


# states of X and W on one mesh axis, per factor
FACTOR_STATES = {"DP": ("S0", "B"), "COL": ("B", "S1"), "KS": ("S1", "S0"), "PB": ("P", "B"),
                 "BP": ("B", "P"), "BB": ("B", "B")}


def nd_input_layouts(factors, mesh, coord):
    """nd states of X and W: factor f on mesh axis a puts X and W in the
    states FACTOR_STATES[f] on that axis."""
    xs = [FACTOR_STATES[f][0] for f in factors]
    ws = [FACTOR_STATES[f][1] for f in factors]
    return sbp.nd_layout(xs, mesh, coord), sbp.nd_layout(ws, mesh, coord)


def nd_layouts(factors, mesh, coord) -> dict:
    x, w = nd_input_layouts(factors, mesh, coord)
    y, dy, dx, dw = sbp.sbp_nd_signature(x, w)
    return {"x": x, "w": w, "y": y, "dy": dy, "dx": dx, "dw": dw}


def shard(l, rows: int, cols: int):
    """The library's share of a rows x cols tensor in 1-D or nd state l."""
    if isinstance(l, sbp.sbp_nd_layout_t):
        return sbp.sbp_nd_shard_index(l, rows, cols)
    return sbp.sbp_shard_index(l, rows, cols)


def is_partial(l) -> bool:
    if isinstance(l, sbp.sbp_nd_layout_t):
        return any(l.kind[a] == sbp.SBP_PARTIAL for a in range(l.ndim))
    return l.kind == sbp.SBP_PARTIAL


def out_shape(op: str, L: dict, M: int, K: int, N: int):
    """Local output shape of op for the device's share of global X (MxK), W (KxN)."""
    if op == "fwd":
        return shard(L["x"], M, K).rows, shard(L["w"], K, N).cols
    if op == "bwd_data":
        return shard(L["dy"], M, N).rows, shard(L["w"], K, N).rows
    if op == "bwd_weight":
        return shard(L["x"], M, K).cols, shard(L["dy"], M, N).cols
    raise ValueError(op)


def out_state(op: str, L: dict):
    return L[{"fwd": "y", "bwd_data": "dx", "bwd_weight": "dw"}[op]]


def out_dtype(op: str, L: dict, in_dtype):
    """fp32 for Partial-sum outputs and fp32 inputs, else the input dtype."""
    if is_partial(out_state(op, L)) or in_dtype == torch.float32:
        return torch.float32
    return in_dtype


def alloc_out(op: str, sig: str, p: int, r: int, M: int, K: int, N: int, in_dtype, device):
    return alloc_out_L(op, layouts(sig, p, r), M, K, N, in_dtype, device)


def alloc_out_L(op: str, L: dict, M: int, K: int, N: int, in_dtype, device):
    rows, cols = out_shape(op, L, M, K, N)
    return torch.empty((rows, cols), dtype=out_dtype(op, L, in_dtype), device=device)


def run(op: str, sig: str, p: int, r: int, X, W, dY, out, stream=None):
    """Launch rank r's local product op of signature sig on global X, W, dY
    (torch tensors; a tensor the op does not read may be None) into `out`;
    returns the output state."""
    return run_L(op, layouts(sig, p, r), X, W, dY, out, stream)


def run_L(op: str, L: dict, X, W, dY, out, stream=None, accumulate=False, ws=None):
    """As run, for the states in L (1-D or nd). accumulate: add the product
    to out's fp32 contents (gradient accumulation); ws: the workspace
    argument of the binding (None: its default workspace)."""
    nd = isinstance(L["x"], sbp.sbp_nd_layout_t)
    fns = {"fwd": sbp.sbp_nd_linear_fwd if nd else sbp.sbp_linear_fwd,
           "bwd_data": sbp.sbp_nd_linear_bwd_data if nd else sbp.sbp_linear_bwd_data,
           "bwd_weight": sbp.sbp_nd_linear_bwd_weight if nd else sbp.sbp_linear_bwd_weight}
    o = sbp.view(out, sbp.SBP_ACCUMULATE if accumulate else sbp.SBP_LOCAL)
    if op == "fwd":
        return fns[op](sbp.view(X), L["x"], sbp.view(W), L["w"], o, stream, ws)
    if op == "bwd_data":
        return fns[op](sbp.view(dY), L["dy"], sbp.view(W), L["w"], o, stream, ws)
    if op == "bwd_weight":
        return fns[op](sbp.view(X), L["x"], sbp.view(dY), L["dy"], o, stream, ws)
    raise ValueError(op)


def run_bwd(sig: str, p: int, r: int, X, W, dY, dX, dW, stream=None):
    """Both backward products of rank r in one call (sbp_linear_bwd); returns
    the (dX, dW) states."""
    return run_bwd_L(layouts(sig, p, r), X, W, dY, dX, dW, stream)


def run_bwd_L(L: dict, X, W, dY, dX, dW, stream=None, accumulate_dw=False, ws=None):
    """Both backward products in one call; accumulate_dw adds dW to its fp32
    contents (gradient accumulation over micro-batches)."""
    fn = sbp.sbp_nd_linear_bwd if isinstance(L["x"], sbp.sbp_nd_layout_t) else sbp.sbp_linear_bwd
    return fn(sbp.view(dY), L["dy"], sbp.view(X), L["x"], sbp.view(W), L["w"],
              sbp.view(dX, sbp.SBP_LOCAL),
              sbp.view(dW, sbp.SBP_ACCUMULATE if accumulate_dw else sbp.SBP_LOCAL), stream, ws)


def call_bwd(sig: str, p: int, r: int, X, W, dY, stream=None):
    """Allocate dX and dW and run both backward products; returns (dX, dW, states)."""
    M, K = X.shape
    N = W.shape[1]
    dX = alloc_out("bwd_data", sig, p, r, M, K, N, X.dtype, X.device)
    dW = alloc_out("bwd_weight", sig, p, r, M, K, N, X.dtype, X.device)
    st = run_bwd(sig, p, r, X, W, dY, dX, dW, stream)
    return dX, dW, st


def call(op: str, sig: str, p: int, r: int, X, W, dY, stream=None):
    """Allocate the output and run; returns (out, state)."""
    ref = X if X is not None else dY
    M = (X if X is not None else dY).shape[0]
    K = X.shape[1] if X is not None else W.shape[0]
    N = W.shape[1] if W is not None else dY.shape[1]
    out = alloc_out(op, sig, p, r, M, K, N, ref.dtype, ref.device)
    st = run(op, sig, p, r, X, W, dY, out, stream)
    return out, st


def call_nd(op: str, factors, mesh, coord, X, W, dY, stream=None):
    """nd form of call: the device at mesh coordinate coord under the per-axis
    factors; returns (out, nd state)."""
    L = nd_layouts(factors, mesh, coord)
    ref = X if X is not None else dY
    M = ref.shape[0]
    K = X.shape[1] if X is not None else W.shape[0]
    N = W.shape[1] if W is not None else dY.shape[1]
    out = alloc_out_L(op, L, M, K, N, ref.dtype, ref.device)
    st = run_L(op, L, X, W, dY, out, stream)
    return out, st


def call_bwd_nd(factors, mesh, coord, X, W, dY, stream=None):
    """nd form of call_bwd; returns (dX, dW, states)."""
    L = nd_layouts(factors, mesh, coord)
    M, K = X.shape
    N = W.shape[1]
    dX = alloc_out_L("bwd_data", L, M, K, N, X.dtype, X.device)
    dW = alloc_out_L("bwd_weight", L, M, K, N, X.dtype, X.device)
    st = run_bwd_L(L, X, W, dY, dX, dW, stream)
    return dX, dW, st
