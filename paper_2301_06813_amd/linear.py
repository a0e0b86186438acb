"""Rank-r local products of one SBP linear, from torch tensors.

Convenience over the binding: picks the input states of a named signature,
asks the library for the output states (``sbp_signature``) and local output
shape (``sbp_shard_index``), allocates the output and calls the entry point.
All computation happens in libsbp.so.

Signatures are the 1-D factors of AutoDDL's SBP matmul (Sec. 4.2):
DP (S(0),B)->S(0), COL (B,S(1))->S(1), KS (S(1),S(0))->P.
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
    raise ValueError("unknown signature %r" % sig)


def layouts(sig: str, p: int, r: int) -> dict:
    x, w = input_layouts(sig, p, r)
    y, dy, dx, dw = sbp.sbp_signature(x, w)
    return {"x": x, "w": w, "y": y, "dy": dy, "dx": dx, "dw": dw}


def out_shape(op: str, L: dict, M: int, K: int, N: int):
    """Local output shape of op for rank r's share of global X (MxK), W (KxN)."""
    if op == "fwd":
        return sbp.sbp_shard_index(L["x"], M, K).rows, sbp.sbp_shard_index(L["w"], K, N).cols
    if op == "bwd_data":
        return sbp.sbp_shard_index(L["dy"], M, N).rows, sbp.sbp_shard_index(L["w"], K, N).rows
    if op == "bwd_weight":
        return sbp.sbp_shard_index(L["x"], M, K).cols, sbp.sbp_shard_index(L["dy"], M, N).cols
    raise ValueError(op)


def out_state(op: str, L: dict):
    return L[{"fwd": "y", "bwd_data": "dx", "bwd_weight": "dw"}[op]]


def out_dtype(op: str, L: dict, in_dtype):
    """fp32 for Partial-sum outputs and fp32 inputs, else the input dtype."""
    if out_state(op, L).kind == sbp.SBP_PARTIAL or in_dtype == torch.float32:
        return torch.float32
    return in_dtype


def alloc_out(op: str, sig: str, p: int, r: int, M: int, K: int, N: int, in_dtype, device):
    L = layouts(sig, p, r)
    rows, cols = out_shape(op, L, M, K, N)
    return torch.empty((rows, cols), dtype=out_dtype(op, L, in_dtype), device=device)


def run(op: str, sig: str, p: int, r: int, X, W, dY, out, stream=None):
    """Launch rank r's local product op of signature sig on global X, W, dY
    (torch tensors; a tensor the op does not read may be None) into `out`;
    returns the output state."""
    L = layouts(sig, p, r)
    if op == "fwd":
        return sbp.sbp_linear_fwd(sbp.view(X), L["x"], sbp.view(W), L["w"],
                                  sbp.view(out, sbp.SBP_LOCAL), stream)
    if op == "bwd_data":
        return sbp.sbp_linear_bwd_data(sbp.view(dY), L["dy"], sbp.view(W), L["w"],
                                       sbp.view(out, sbp.SBP_LOCAL), stream)
    if op == "bwd_weight":
        return sbp.sbp_linear_bwd_weight(sbp.view(X), L["x"], sbp.view(dY), L["dy"],
                                         sbp.view(out, sbp.SBP_LOCAL), stream)
    raise ValueError(op)


def run_bwd(sig: str, p: int, r: int, X, W, dY, dX, dW, stream=None):
    """Both backward products of rank r in one call (sbp_linear_bwd); returns
    the (dX, dW) states."""
    L = layouts(sig, p, r)
    return sbp.sbp_linear_bwd(sbp.view(dY), L["dy"], sbp.view(X), L["x"], sbp.view(W), L["w"],
                              sbp.view(dX, sbp.SBP_LOCAL), sbp.view(dW, sbp.SBP_LOCAL), stream)


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
