"""One rank's share of a workload's linear layers as a fixed sequence of
C-ABI calls: every forward product in layer order, then both backward
products of each linear (one sbp_linear_bwd call) in reverse order, with all
buffers preallocated so the sequence can be replayed from a HIP graph. The
benchmark and the in-step plan tuner both run it."""
from __future__ import annotations

OPS = ("fwd", "bwd_data", "bwd_weight")


class Step:
    """Rank r's calls of one workload, with all buffers preallocated: every
    forward product in layer order, then both backward products of each
    linear (one sbp_linear_bwd call) in reverse order."""

    def __init__(self, wl, r, device="cuda"):
        import ctypes
        import torch
        from . import linear, sbp, workloads
        self.sbp = sbp
        self.keep = []
        fwd, bwd = [], []
        for lin in wl.linears:
            X, W, dY = workloads.make_tensors(lin, wl.dtype, device)
            L = linear.layouts(lin.sig, wl.p, r)
            self.keep += [X, W, dY]
            vX, vW, vdY = sbp.view(X), sbp.view(W), sbp.view(dY)
            outs = {}
            for op in OPS:
                out = linear.alloc_out(op, lin.sig, wl.p, r, lin.M, lin.K, lin.N, wl.dtype, device)
                self.keep.append(out)
                outs[op] = out
            prods = {}
            for op, out in outs.items():
                m, n = out.shape
                k = {"fwd": sbp.sbp_shard_index(L["x"], lin.M, lin.K).cols,
                     "bwd_data": sbp.sbp_shard_index(L["dy"], lin.M, lin.N).cols,
                     "bwd_weight": sbp.sbp_shard_index(L["x"], lin.M, lin.K).rows}[op]
                ob = 4 if out.dtype == torch.float32 else 2
                prods[op] = dict(m=m, n=n, k=k, flops=2.0 * m * n * k,
                                 bytes=2.0 * (m * k + k * n) + ob * m * n)
            vo = {op: sbp.view(out, sbp.SBP_LOCAL) for op, out in outs.items()}
            f = ("sbp_linear_fwd", (vX, L["x"], vW, L["w"], vo["fwd"]), 1)
            fwd.append((f, dict(linear=lin.name, sig=lin.sig, ops=("fwd",), lin=lin, layouts=L,
                                **prods["fwd"])))
            bcall = ("sbp_linear_bwd", (vdY, L["dy"], vX, L["x"], vW, L["w"], vo["bwd_data"]),
                     (vo["bwd_weight"],))
            pb = dict(flops=prods["bwd_data"]["flops"] + prods["bwd_weight"]["flops"],
                      bytes=prods["bwd_data"]["bytes"] + prods["bwd_weight"]["bytes"])
            bwd.append((bcall, dict(linear=lin.name, sig=lin.sig, ops=("bwd_data", "bwd_weight"),
                                    lin=lin, layouts=L, data=prods["bwd_data"],
                                    weight=prods["bwd_weight"], **pb)))
        self.calls, self.meta = [], []
        for call, meta in fwd + bwd[::-1]:
            self.calls.append(call)
            self.meta.append(meta)
        self.flops = sum(m["flops"] for m in self.meta)
        L_ = sbp.lib()
        self._lo = sbp.sbp_layout_t()
        self._lo2 = sbp.sbp_layout_t()
        lo, lo2 = ctypes.byref(self._lo), ctypes.byref(self._lo2)
        # the split reductions' workspace (caller-owned; every call of the
        # step runs in order on one stream, so they share it)
        self.ws_mem = torch.empty(sbp.SBP_WORKSPACE_BYTES, dtype=torch.uint8, device=device)
        self._ws = sbp.workspace(self.ws_mem)
        ws = ctypes.byref(self._ws)
        self._bound = []
        for name, args, extra in self.calls:
            fn = getattr(L_, name)
            refs = tuple(ctypes.byref(a) for a in args)
            if name == "sbp_linear_bwd":
                refs = refs + (lo, ctypes.byref(extra[0]), lo2, ws)
            else:
                refs = refs + (lo, ws)
            self._bound.append((fn, refs))

    def launch_all(self, stream, hook=None):
        """Launch every call in order on `stream`. hook(i, before): called
        before (True) and after (False) call i, e.g. to set and clear a plan
        override for that call while a graph is captured."""
        import ctypes
        s = ctypes.c_void_p(stream)
        for i, (fn, refs) in enumerate(self._bound):
            if hook:
                hook(i, True)
            rc = fn(*refs, s)
            if hook:
                hook(i, False)
            if rc != 0:
                raise self.sbp.SbpError(rc, self.sbp.sbp_last_hip_error())

    def profile(self, stream):
        """Per call: [(kernel name, us)] of every kernel it launched, each
        timed by events recorded with its own dispatch."""
        import ctypes
        s = ctypes.c_void_p(stream)
        out = []
        for fn, refs in self._bound:
            self.sbp.sbp_profile_begin(16)
            rc = fn(*refs, s)
            ks = self.sbp.sbp_profile_end(16)
            if rc != 0:
                raise self.sbp.SbpError(rc, self.sbp.sbp_last_hip_error())
            out.append(ks)
        return out
