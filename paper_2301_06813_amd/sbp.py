"""ctypes binding of libsbp.so, the C ABI declared in include/sbp.h.

Argument marshalling only: every computation runs in the library's kernels.
The functions carry the C names; a nonzero return code raises SbpError.
Loading fails loudly when the library has not been built
(``python -m paper_2301_06813_amd.build``); there is no fallback.

``view(tensor, scope)`` turns a 2-D torch tensor with unit column stride into
an ``sbp_view_t`` (pointer, rows, cols, ld, dtype, scope); torch is used only
for device memory and streams.

The linear calls take a caller-owned workspace for split reductions
(``sbp_workspace_t``). Their ``ws`` argument: None (default) uses a
workspace of SBP_WORKSPACE_BYTES that this module allocates with torch once
per (device, stream) and keeps; NO_WORKSPACE runs without one (no split
reductions); a torch tensor or an ``sbp_workspace_t`` is used as given.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsbp.so")

# ---------------------------------------------------------------- constants
SBP_OK = 0
SBP_ERR_NULL = -1
SBP_ERR_LAYOUT = -2
SBP_ERR_SIGNATURE = -3
SBP_ERR_SHAPE = -4
SBP_ERR_DTYPE = -5
SBP_ERR_ALIAS = -6
SBP_ERR_ALIGN = -7
SBP_ERR_HIP = -8
SBP_ERR_WORKSPACE = -9
SBP_WORKSPACE_BYTES = 64 << 20

SBP_SPLIT, SBP_BROADCAST, SBP_PARTIAL = 0, 1, 2
SBP_BF16, SBP_F32 = 0, 1
SBP_GLOBAL, SBP_LOCAL, SBP_ACCUMULATE = 0, 1, 2

EXPORTS = ("sbp_shard_index", "sbp_signature", "sbp_linear_fwd", "sbp_linear_bwd_data",
           "sbp_linear_bwd_weight", "sbp_linear_bwd", "sbp_strerror", "sbp_last_hip_error", "sbp_plan",
           "sbp_plan_bwd", "sbp_set_plan_override", "sbp_set_bwd_override", "sbp_profile_begin",
           "sbp_profile_end", "sbp_mesh_coords", "sbp_nd_shard_index", "sbp_nd_signature",
           "sbp_nd_linear_fwd", "sbp_nd_linear_bwd_data", "sbp_nd_linear_bwd_weight",
           "sbp_nd_linear_bwd", "sbp_attn_scores", "sbp_attn_context", "sbp_attn_scores_bwd",
           "sbp_attn_context_bwd", "sbp_set_override_orients", "sbp_collective_cost",
           "sbp_boxing_cost", "sbp_chain_cost", "sbp_search_strategy", "sbp_linear_bwd_noalloc")

SBP_COLL_ALLREDUCE, SBP_COLL_ALLGATHER, SBP_COLL_REDUCESCATTER, SBP_COLL_ALLTOALL = 0, 1, 2, 3
SBP_SIG_DP, SBP_SIG_COL, SBP_SIG_KS, SBP_SIG_PB, SBP_SIG_BP, SBP_SIG_BB = 0, 1, 2, 3, 4, 5
SIG_IDS = {"DP": 0, "COL": 1, "KS": 2, "PB": 3, "BP": 4, "BB": 5}

SBP_MAX_MESH_DIMS = 4


class sbp_layout_t(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("axis", ctypes.c_int32),
                ("p", ctypes.c_int32), ("r", ctypes.c_int32)]

    def __repr__(self):
        name = {SBP_SPLIT: "S(%d)" % self.axis, SBP_BROADCAST: "B", SBP_PARTIAL: "P"}.get(
            self.kind, "?%d" % self.kind)
        return "%s[p=%d,r=%d]" % (name, self.p, self.r)

    def key(self):
        return (self.kind, self.axis, self.p, self.r)


class sbp_nd_layout_t(ctypes.Structure):
    _fields_ = [("ndim", ctypes.c_int32), ("kind", ctypes.c_int32 * 4),
                ("axis", ctypes.c_int32 * 4), ("p", ctypes.c_int32 * 4),
                ("c", ctypes.c_int32 * 4)]

    def __repr__(self):
        parts = []
        for a in range(self.ndim):
            k = self.kind[a]
            name = {SBP_SPLIT: "S(%d)" % self.axis[a], SBP_BROADCAST: "B",
                    SBP_PARTIAL: "P"}.get(k, "?%d" % k)
            parts.append("%s:%d@%d" % (name, self.p[a], self.c[a]))
        return "(" + ", ".join(parts) + ")"

    def key(self):
        n = self.ndim
        return (n, tuple(self.kind[:n]), tuple(self.axis[:n]), tuple(self.p[:n]),
                tuple(self.c[:n]))

    def states(self):
        """Per mesh axis (kind, axis)."""
        return [(self.kind[a], self.axis[a]) for a in range(self.ndim)]


class sbp_view_t(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("ld", ctypes.c_int64), ("dtype", ctypes.c_int32), ("scope", ctypes.c_int32)]


class sbp_view4_t(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("batch", ctypes.c_int64), ("heads", ctypes.c_int64),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("stride_b", ctypes.c_int64), ("stride_h", ctypes.c_int64),
                ("ld", ctypes.c_int64), ("dtype", ctypes.c_int32), ("scope", ctypes.c_int32)]


class sbp_chain_t(ctypes.Structure):
    _fields_ = [("layers", ctypes.c_int32), ("p", ctypes.c_int32), ("alpha", ctypes.c_double),
                ("beta", ctypes.c_double), ("M", ctypes.POINTER(ctypes.c_int64)),
                ("K", ctypes.POINTER(ctypes.c_int64)), ("N", ctypes.POINTER(ctypes.c_int64)),
                ("act_bytes", ctypes.c_double), ("grad_bytes", ctypes.c_double),
                ("in_kind", ctypes.c_int32), ("in_axis", ctypes.c_int32),
                ("out_kind", ctypes.c_int32), ("out_axis", ctypes.c_int32),
                ("allowed", ctypes.c_uint32)]


class sbp_workspace_t(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("bytes", ctypes.c_int64)]


NO_WORKSPACE = sbp_workspace_t(None, 0)


class sbp_shard_t(ctypes.Structure):
    _fields_ = [("row_off", ctypes.c_int64), ("col_off", ctypes.c_int64),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64)]


class SbpError(RuntimeError):
    def __init__(self, code, hip_error=0):
        self.code = code
        self.hip_error = hip_error
        msg = "%s (%d)" % (sbp_strerror(code), code)
        if code == SBP_ERR_HIP:
            msg += ", hipError %d" % hip_error
        super().__init__(msg)


def split(axis: int, p: int, r: int) -> sbp_layout_t:
    return sbp_layout_t(SBP_SPLIT, axis, p, r)


def broadcast(p: int, r: int) -> sbp_layout_t:
    return sbp_layout_t(SBP_BROADCAST, -1, p, r)


def partial(p: int, r: int) -> sbp_layout_t:
    return sbp_layout_t(SBP_PARTIAL, -1, p, r)


def nd_layout(states, mesh, coord) -> sbp_nd_layout_t:
    """sbp_nd_layout_t from per-mesh-axis states ("S0", "S1", "B", "P" or
    (kind, axis) pairs), mesh extents and this device's mesh coordinate."""
    n = len(mesh)
    if not (1 <= n <= SBP_MAX_MESH_DIMS) or len(states) != n or len(coord) != n:
        raise ValueError("states, mesh and coord need one entry per mesh axis (1..4)")
    names = {"S0": (SBP_SPLIT, 0), "S1": (SBP_SPLIT, 1), "B": (SBP_BROADCAST, -1),
             "P": (SBP_PARTIAL, -1)}
    l = sbp_nd_layout_t()
    l.ndim = n
    for a, st in enumerate(states):
        k, ax = names[st] if isinstance(st, str) else st
        l.kind[a], l.axis[a], l.p[a], l.c[a] = k, ax, mesh[a], coord[a]
    return l


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libsbp.so is not built (%s); run `python -m "
                              "paper_2301_06813_amd.build`" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.sbp_shard_index.argtypes = [P(sbp_layout_t), ctypes.c_int64, ctypes.c_int64,
                                      P(sbp_shard_t)]
        L.sbp_signature.argtypes = [P(sbp_layout_t)] * 6
        WS = P(sbp_workspace_t)
        for fn in ("sbp_linear_fwd", "sbp_linear_bwd_data", "sbp_linear_bwd_weight"):
            getattr(L, fn).argtypes = [P(sbp_view_t), P(sbp_layout_t), P(sbp_view_t),
                                       P(sbp_layout_t), P(sbp_view_t), P(sbp_layout_t),
                                       WS, ctypes.c_void_p]
        L.sbp_linear_bwd.argtypes = [P(sbp_view_t), P(sbp_layout_t), P(sbp_view_t),
                                     P(sbp_layout_t), P(sbp_view_t), P(sbp_layout_t),
                                     P(sbp_view_t), P(sbp_layout_t), P(sbp_view_t),
                                     P(sbp_layout_t), WS, ctypes.c_void_p]
        L.sbp_linear_bwd_noalloc.argtypes = [P(sbp_view_t), P(sbp_layout_t), P(sbp_view_t),
                                             P(sbp_layout_t), P(sbp_view_t), P(sbp_layout_t),
                                             P(sbp_view_t), P(sbp_layout_t), P(sbp_view_t),
                                             P(sbp_layout_t), ctypes.c_void_p]
        L.sbp_strerror.argtypes = [ctypes.c_int]
        L.sbp_strerror.restype = ctypes.c_char_p
        L.sbp_last_hip_error.argtypes = []
        L.sbp_plan.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                               ctypes.c_int32, ctypes.c_int32, P(ctypes.c_int32),
                               P(ctypes.c_int32), P(ctypes.c_int32), P(ctypes.c_int32)]
        L.sbp_set_plan_override.argtypes = [ctypes.c_int32] * 5
        L.sbp_set_bwd_override.argtypes = [ctypes.c_int32] * 2
        L.sbp_set_override_orients.argtypes = [ctypes.c_int32]
        L.sbp_profile_begin.argtypes = [ctypes.c_int]
        L.sbp_profile_end.argtypes = [ctypes.c_void_p, ctypes.c_char_p, ctypes.c_int]
        L.sbp_plan_bwd.argtypes = ([ctypes.c_int64] * 3 + [ctypes.c_int32] + [ctypes.c_int64] * 3 +
                                   [ctypes.c_int32] + [P(ctypes.c_int32)] * 5)
        ND = P(sbp_nd_layout_t)
        L.sbp_mesh_coords.argtypes = [ctypes.c_int32, P(ctypes.c_int32), P(ctypes.c_int32),
                                      ctypes.c_int64, ctypes.c_int64, P(ctypes.c_int32)]
        L.sbp_nd_shard_index.argtypes = [ND, ctypes.c_int64, ctypes.c_int64, P(sbp_shard_t)]
        L.sbp_nd_signature.argtypes = [ND] * 6
        for fn in ("sbp_nd_linear_fwd", "sbp_nd_linear_bwd_data", "sbp_nd_linear_bwd_weight"):
            getattr(L, fn).argtypes = [P(sbp_view_t), ND, P(sbp_view_t), ND, P(sbp_view_t), ND,
                                       WS, ctypes.c_void_p]
        L.sbp_nd_linear_bwd.argtypes = [P(sbp_view_t), ND, P(sbp_view_t), ND, P(sbp_view_t), ND,
                                        P(sbp_view_t), ND, P(sbp_view_t), ND, WS,
                                        ctypes.c_void_p]
        V4 = P(sbp_view4_t)
        for fn in ("sbp_attn_scores", "sbp_attn_context"):
            getattr(L, fn).argtypes = [V4, V4, V4, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
        for fn in ("sbp_attn_scores_bwd", "sbp_attn_context_bwd"):
            getattr(L, fn).argtypes = [V4, V4, V4, V4, V4, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_void_p]
        D = ctypes.c_double
        L.sbp_collective_cost.argtypes = [ctypes.c_int32, ctypes.c_int32, D, D, D, P(D)]
        L.sbp_boxing_cost.argtypes = [P(sbp_layout_t), P(sbp_layout_t), D, D, D, P(D),
                                      P(ctypes.c_int32)]
        L.sbp_chain_cost.argtypes = [P(sbp_chain_t), P(ctypes.c_int32), P(D)]
        L.sbp_search_strategy.argtypes = [P(sbp_chain_t), ctypes.c_int32, ctypes.c_uint64,
                                          P(ctypes.c_int32), P(D), P(D), ctypes.c_int32,
                                          P(ctypes.c_int32)]
        for fn in EXPORTS:
            if fn != "sbp_strerror":
                getattr(L, fn).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(code):
    if code != SBP_OK:
        raise SbpError(code, lib().sbp_last_hip_error() if code == SBP_ERR_HIP else 0)


# ------------------------------------------------------------------- views
def view(t, scope=SBP_GLOBAL) -> sbp_view_t:
    """sbp_view_t of a 2-D torch tensor whose columns are contiguous."""
    import torch
    if t.dim() != 2:
        raise ValueError("views are 2-D")
    if t.stride(1) != 1 and t.shape[1] > 1:
        raise ValueError("views need unit column stride")
    dt = {torch.bfloat16: SBP_BF16, torch.float32: SBP_F32}.get(t.dtype)
    if dt is None:
        raise TypeError("unsupported dtype %s" % t.dtype)
    ld = max(t.stride(0), t.shape[1], 1)
    return sbp_view_t(t.data_ptr(), t.shape[0], t.shape[1], ld, dt, scope)


def view4(t, scope=SBP_GLOBAL) -> sbp_view4_t:
    """sbp_view4_t of a 4-D torch tensor [batch][heads][rows][cols] (any
    strides with unit column stride; e.g. a permuted view into a fused QKV
    activation)."""
    import torch
    if t.dim() != 4:
        raise ValueError("view4 needs a 4-D tensor")
    if t.stride(3) != 1 and t.shape[3] > 1:
        raise ValueError("views need unit column stride")
    dt = {torch.bfloat16: SBP_BF16, torch.float32: SBP_F32}.get(t.dtype)
    if dt is None:
        raise TypeError("unsupported dtype %s" % t.dtype)
    ld = max(t.stride(2), t.shape[3], 1)
    return sbp_view4_t(t.data_ptr(), t.shape[0], t.shape[1], t.shape[2], t.shape[3],
                       t.stride(0), t.stride(1), ld, dt, scope)


def raw_view(ptr, rows, cols, ld, dtype, scope=SBP_GLOBAL) -> sbp_view_t:
    return sbp_view_t(ptr, rows, cols, ld, dtype, scope)


def current_stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


_default_ws = {}


def workspace(t) -> sbp_workspace_t:
    """sbp_workspace_t over a device tensor's bytes (kept alive by the caller)."""
    return sbp_workspace_t(t.data_ptr(), t.numel() * t.element_size())


def default_workspace(stream) -> sbp_workspace_t:
    """This module's workspace for (current device, stream): SBP_WORKSPACE_BYTES
    allocated with torch on first use and kept (calls on one stream run in
    order, so they can share it)."""
    import torch
    key = (torch.cuda.current_device(), int(stream or 0))
    t = _default_ws.get(key)
    if t is None:
        t = torch.empty(SBP_WORKSPACE_BYTES, dtype=torch.uint8, device="cuda")
        _default_ws[key] = t
    return workspace(t)


def _ws(ws, stream):
    if ws is None:
        return default_workspace(stream)
    if isinstance(ws, sbp_workspace_t):
        return ws
    return workspace(ws)


# ------------------------------------------------------------- functions
def sbp_strerror(code: int) -> str:
    return lib().sbp_strerror(code).decode()


def sbp_shard_index(layout: sbp_layout_t, rows: int, cols: int) -> sbp_shard_t:
    out = sbp_shard_t()
    _check(lib().sbp_shard_index(ctypes.byref(layout), rows, cols, ctypes.byref(out)))
    return out


def sbp_signature(x: sbp_layout_t, w: sbp_layout_t):
    """(Y, dY, dX, dW) states for X in state x and W in state w."""
    y, dy, dx, dw = sbp_layout_t(), sbp_layout_t(), sbp_layout_t(), sbp_layout_t()
    _check(lib().sbp_signature(ctypes.byref(x), ctypes.byref(w), ctypes.byref(y),
                               ctypes.byref(dy), ctypes.byref(dx), ctypes.byref(dw)))
    return y, dy, dx, dw


def _compute(fn, a, la, b, lb, out, stream, ws):
    lo = type(la)()
    s = current_stream() if stream is None else stream
    w = _ws(ws, s)
    _check(getattr(lib(), fn)(ctypes.byref(a), ctypes.byref(la), ctypes.byref(b),
                              ctypes.byref(lb), ctypes.byref(out), ctypes.byref(lo),
                              ctypes.byref(w), ctypes.c_void_p(s)))
    return lo


def sbp_linear_fwd(X: sbp_view_t, lx: sbp_layout_t, W: sbp_view_t, lw: sbp_layout_t,
                   Y: sbp_view_t, stream=None, ws=None) -> sbp_layout_t:
    """Y_r = X_r W_r on `stream` (default: torch's current stream); returns Y's state."""
    return _compute("sbp_linear_fwd", X, lx, W, lw, Y, stream, ws)


def sbp_linear_bwd_data(dY: sbp_view_t, ldy: sbp_layout_t, W: sbp_view_t, lw: sbp_layout_t,
                        dX: sbp_view_t, stream=None, ws=None) -> sbp_layout_t:
    """dX_r = dY_r W_r^T; returns dX's state."""
    return _compute("sbp_linear_bwd_data", dY, ldy, W, lw, dX, stream, ws)


def sbp_linear_bwd_weight(X: sbp_view_t, lx: sbp_layout_t, dY: sbp_view_t, ldy: sbp_layout_t,
                          dW: sbp_view_t, stream=None, ws=None) -> sbp_layout_t:
    """dW_r = X_r^T dY_r; returns dW's state."""
    return _compute("sbp_linear_bwd_weight", X, lx, dY, ldy, dW, stream, ws)


def sbp_linear_bwd(dY: sbp_view_t, ldy: sbp_layout_t, X: sbp_view_t, lx: sbp_layout_t,
                   W: sbp_view_t, lw: sbp_layout_t, dX: sbp_view_t, dW: sbp_view_t,
                   stream=None, ws=None):
    """dX_r = dY_r W_r^T and dW_r = X_r^T dY_r in one call; returns (dX state, dW state)."""
    sx, sw = sbp_layout_t(), sbp_layout_t()
    s = current_stream() if stream is None else stream
    w = _ws(ws, s)
    _check(lib().sbp_linear_bwd(ctypes.byref(dY), ctypes.byref(ldy), ctypes.byref(X),
                                ctypes.byref(lx), ctypes.byref(W), ctypes.byref(lw),
                                ctypes.byref(dX), ctypes.byref(sx), ctypes.byref(dW),
                                ctypes.byref(sw), ctypes.byref(w), ctypes.c_void_p(s)))
    return sx, sw


def sbp_linear_bwd_noalloc(dY: sbp_view_t, ldy: sbp_layout_t, X: sbp_view_t, lx: sbp_layout_t,
                           W: sbp_view_t, lw: sbp_layout_t, dX: sbp_view_t, dW: sbp_view_t,
                           stream=None):
    """sbp_linear_bwd with the library's static scratch as its workspace (for
    callers that cannot allocate); returns (dX state, dW state)."""
    sx, sw = sbp_layout_t(), sbp_layout_t()
    s = current_stream() if stream is None else stream
    _check(lib().sbp_linear_bwd_noalloc(ctypes.byref(dY), ctypes.byref(ldy), ctypes.byref(X),
                                        ctypes.byref(lx), ctypes.byref(W), ctypes.byref(lw),
                                        ctypes.byref(dX), ctypes.byref(sx), ctypes.byref(dW),
                                        ctypes.byref(sw), ctypes.c_void_p(s)))
    return sx, sw


# ------------------------------------------------------------------ nd-SBP
def sbp_mesh_coords(nodes, gpus=None, node: int = 0, gpu: int = 0) -> list[int]:
    """Mesh coordinate of device (node, gpu) on a mesh whose axis a spans
    nodes[a] x gpus[a] devices (gpus None: a single-level mesh, node = rank)."""
    n = len(nodes)
    arr = ctypes.c_int32 * max(n, 1)
    c = arr()
    g = None if gpus is None else arr(*gpus)
    _check(lib().sbp_mesh_coords(n, arr(*nodes), g, node, gpu, c))
    return list(c[:n])


def sbp_nd_shard_index(layout: sbp_nd_layout_t, rows: int, cols: int) -> sbp_shard_t:
    out = sbp_shard_t()
    _check(lib().sbp_nd_shard_index(ctypes.byref(layout), rows, cols, ctypes.byref(out)))
    return out


def sbp_nd_signature(x: sbp_nd_layout_t, w: sbp_nd_layout_t):
    """(Y, dY, dX, dW) nd states for X in state x and W in state w."""
    outs = [sbp_nd_layout_t() for _ in range(4)]
    _check(lib().sbp_nd_signature(ctypes.byref(x), ctypes.byref(w),
                                  *(ctypes.byref(o) for o in outs)))
    return tuple(outs)


def sbp_nd_linear_fwd(X, lx: sbp_nd_layout_t, W, lw: sbp_nd_layout_t, Y, stream=None, ws=None):
    """Y_r = X_r W_r on nd shares; returns Y's nd state."""
    return _compute("sbp_nd_linear_fwd", X, lx, W, lw, Y, stream, ws)


def sbp_nd_linear_bwd_data(dY, ldy: sbp_nd_layout_t, W, lw: sbp_nd_layout_t, dX, stream=None,
                           ws=None):
    """dX_r = dY_r W_r^T on nd shares; returns dX's nd state."""
    return _compute("sbp_nd_linear_bwd_data", dY, ldy, W, lw, dX, stream, ws)


def sbp_nd_linear_bwd_weight(X, lx: sbp_nd_layout_t, dY, ldy: sbp_nd_layout_t, dW, stream=None,
                             ws=None):
    """dW_r = X_r^T dY_r on nd shares; returns dW's nd state."""
    return _compute("sbp_nd_linear_bwd_weight", X, lx, dY, ldy, dW, stream, ws)


def sbp_nd_linear_bwd(dY, ldy, X, lx, W, lw, dX, dW, stream=None, ws=None):
    """Both backward products on nd shares in one call; returns (dX state, dW state)."""
    sx, sw = sbp_nd_layout_t(), sbp_nd_layout_t()
    s = current_stream() if stream is None else stream
    w = _ws(ws, s)
    _check(lib().sbp_nd_linear_bwd(ctypes.byref(dY), ctypes.byref(ldy), ctypes.byref(X),
                                   ctypes.byref(lx), ctypes.byref(W), ctypes.byref(lw),
                                   ctypes.byref(dX), ctypes.byref(sx), ctypes.byref(dW),
                                   ctypes.byref(sw), ctypes.byref(w), ctypes.c_void_p(s)))
    return sx, sw


# ------------------------------------------------------- attention core
def _stream(stream):
    return ctypes.c_void_p(current_stream() if stream is None else stream)


def sbp_attn_scores(Q, K, S, p: int, r: int, stream=None):
    """S = Q K^T per (batch, local head) under a head split over p devices."""
    _check(lib().sbp_attn_scores(ctypes.byref(Q), ctypes.byref(K), ctypes.byref(S), p, r,
                                 _stream(stream)))


def sbp_attn_context(P_, V, O, p: int, r: int, stream=None):
    """O = P V per (batch, local head)."""
    _check(lib().sbp_attn_context(ctypes.byref(P_), ctypes.byref(V), ctypes.byref(O), p, r,
                                  _stream(stream)))


def sbp_attn_scores_bwd(dS, Q, K, dQ, dK, p: int, r: int, stream=None):
    """dQ = dS K and dK = dS^T Q per (batch, local head)."""
    _check(lib().sbp_attn_scores_bwd(ctypes.byref(dS), ctypes.byref(Q), ctypes.byref(K),
                                     ctypes.byref(dQ), ctypes.byref(dK), p, r, _stream(stream)))


def sbp_attn_context_bwd(dO, P_, V, dP, dV, p: int, r: int, stream=None):
    """dP = dO V^T and dV = P^T dO per (batch, local head)."""
    _check(lib().sbp_attn_context_bwd(ctypes.byref(dO), ctypes.byref(P_), ctypes.byref(V),
                                      ctypes.byref(dP), ctypes.byref(dV), p, r, _stream(stream)))


# ------------------------------------------- cost model and search
def sbp_collective_cost(coll: int, p: int, n: float, alpha: float, beta: float) -> float:
    c = ctypes.c_double()
    _check(lib().sbp_collective_cost(coll, p, n, alpha, beta, ctypes.byref(c)))
    return c.value


def sbp_boxing_cost(frm: sbp_layout_t, to: sbp_layout_t, nbytes: float, alpha: float,
                    beta: float):
    """(time, collective id or -1) of moving a tensor between two 1-D states."""
    c, k = ctypes.c_double(), ctypes.c_int32()
    _check(lib().sbp_boxing_cost(ctypes.byref(frm), ctypes.byref(to), nbytes, alpha, beta,
                                 ctypes.byref(c), ctypes.byref(k)))
    return c.value, k.value


def make_chain(p, alpha, beta, M, K, N, act_bytes=2.0, grad_bytes=4.0, in_state=(0, 0),
               out_state=(0, 0), allowed=("DP", "COL", "KS")):
    """An sbp_chain_t (the arrays are kept alive on the returned object)."""
    L = len(K)
    arr = ctypes.c_int64 * L
    net = sbp_chain_t()
    net._M, net._K, net._N = arr(*([M] * L)), arr(*K), arr(*N)
    net.layers, net.p, net.alpha, net.beta = L, p, alpha, beta
    net.M, net.K, net.N = net._M, net._K, net._N
    net.act_bytes, net.grad_bytes = act_bytes, grad_bytes
    net.in_kind, net.in_axis = in_state
    net.out_kind, net.out_axis = out_state
    net.allowed = sum(1 << SIG_IDS[a] for a in allowed)
    return net


def sbp_chain_cost(net: sbp_chain_t, sigs) -> float:
    a = (ctypes.c_int32 * len(sigs))(*sigs)
    c = ctypes.c_double()
    _check(lib().sbp_chain_cost(ctypes.byref(net), a, ctypes.byref(c)))
    return c.value


def sbp_search_strategy(net: sbp_chain_t, restarts: int = 16, seed: int = 0,
                        max_sweeps: int = 4096):
    """(signature ids, cost, per-sweep costs) of the coordinate-descent search."""
    sigs = (ctypes.c_int32 * net.layers)()
    cost = ctypes.c_double()
    sweeps = (ctypes.c_double * max_sweeps)()
    ns = ctypes.c_int32()
    _check(lib().sbp_search_strategy(ctypes.byref(net), restarts, seed, sigs, ctypes.byref(cost),
                                     sweeps, max_sweeps, ctypes.byref(ns)))
    return list(sigs), cost.value, list(sweeps[:min(ns.value, max_sweeps)])


def sbp_last_hip_error() -> int:
    return lib().sbp_last_hip_error()


KERNEL_AUTO, KERNEL_PIPELINED, KERNEL_GENERIC, KERNEL_F32, KERNEL_PIPELINED_2STAGE = 0, 1, 2, 3, 4
KERNEL_GROUPS_STAGED, KERNEL_ROWQ, KERNEL_GROUPS_ROWQ = 5, 6, 7
KERNEL_DEEP, KERNEL_GROUPS_DEEP = 8, 9
KERNEL_GROUPS_2STAGE, KERNEL_DEEP_PREFETCH = 10, 11
KERNEL_GROUPS_WIDE, KERNEL_GROUPS_WIDE_ROWQ = 12, 13


def sbp_plan(op: int, m: int, n: int, k: int, in_dtype: int, out_dtype: int):
    """(tile_m, tile_n, splits, kernel) the library would launch for this product
    with aligned operands; kernel is KERNEL_F32 or one of the bf16 instance codes
    of sbp_set_plan_override (KERNEL_PIPELINED ... KERNEL_GROUPS_WIDE_ROWQ)."""
    tm, tn, sp, kn = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check(lib().sbp_plan(op, m, n, k, in_dtype, out_dtype, ctypes.byref(tm), ctypes.byref(tn),
                          ctypes.byref(sp), ctypes.byref(kn)))
    return tm.value, tn.value, sp.value, kn.value


def sbp_plan_bwd(md, nd, kd, out_d, mw, nw, kw, out_w):
    """(grouped, tile_m, tile_n, splits_d, splits_w) of sbp_linear_bwd for aligned operands."""
    v = [ctypes.c_int32() for _ in range(5)]
    _check(lib().sbp_plan_bwd(md, nd, kd, out_d, mw, nw, kw, out_w, *(ctypes.byref(x) for x in v)))
    return tuple(x.value for x in v)


def sbp_profile_begin(capacity: int) -> None:
    _check(lib().sbp_profile_begin(capacity))


def sbp_profile_end(capacity: int):
    """[(kernel name, microseconds)] of the kernels launched since sbp_profile_begin."""
    us = (ctypes.c_float * max(capacity, 1))()
    nl = 160
    names = ctypes.create_string_buffer(max(capacity, 1) * nl)
    n = lib().sbp_profile_end(us, names, nl)
    if n < 0:
        _check(n)
    raw = names.raw
    return [(raw[i * nl:(i + 1) * nl].split(b"\0", 1)[0].decode(), us[i]) for i in range(n)]


def sbp_set_override_orients(mask: int) -> None:
    """Apply the plan override only to orientations in mask (bit 0 forward,
    1 backward-data, 2 backward-weight); cleared with the plan override."""
    _check(lib().sbp_set_override_orients(mask))


def sbp_set_bwd_override(mode: int, splits_w: int = 1) -> None:
    """How sbp_linear_bwd runs its products: 0 library's choice, 1 two launches,
    2 one grouped launch (plan override's tile/kernel; splits_w for dW)."""
    _check(lib().sbp_set_bwd_override(mode, splits_w))


def sbp_set_plan_override(tile_m: int, tile_n: int, splits: int, kernel: int = 0,
                          wgs_per_cu: int = 0) -> None:
    _check(lib().sbp_set_plan_override(tile_m, tile_n, splits, kernel, wgs_per_cu))
