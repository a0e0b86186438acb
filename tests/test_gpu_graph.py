"""Library calls captured into a HIP graph and replayed.

The benchmark times its step by replaying a graph of library calls, so the
replays must compute what the eager calls compute. A set of calls covering
every signature and operation, the split reduction (whose partials go to the
caller's workspace), the grouped backward launch and an accumulating weight
gradient is made once eagerly on a side stream and then captured on that
stream. The graph is replayed several times with other eager library calls
on the same stream (same workspace) and synchronisations in between; after
every replay each output must be bit-identical to the eager result (the
kernels are deterministic), and the eager results themselves are exact
against the oracle (integer inputs).

The library allocates nothing, so a capture needs no eager call first: the
second test captures split and grouped calls on a fresh stream, with a
workspace the caller allocated, and checks every replay against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2301_06813_amd import inputs, linear, sbp

from helpers import decode, oracle_full, out_bits, say

pytestmark = pytest.mark.gpu

M, K, N = 1024, 768, 512
P, R = 4, 1
# (name, signature, op, plan override (tile_m, tile_n, splits, kernel, wgs_per_cu) or None)
CASES = [
    ("dp fwd", "DP", "fwd", None),
    ("col fwd split", "COL", "fwd", (128, 128, 3, 4, 0)),
    ("ks fwd", "KS", "fwd", None),
    ("dp bwd_data split staged", "DP", "bwd_data", (128, 128, 4, 5, 0)),
    ("col bwd_data", "COL", "bwd_data", None),
    ("ks bwd_weight split rowq", "KS", "bwd_weight", (128, 128, 5, 7, 0)),
    ("dp bwd_weight persistent split", "DP", "bwd_weight", (64, 64, 2, 1, 2)),
    ("bb fwd", "BB", "fwd", None),
]
BWD_CASES = ["DP", "COL", "KS"]   # sbp_linear_bwd, the library's own plan (grouped)


def _inputs(seed):
    X = inputs.randint((M, K), -3, 3, seed + 1, torch.bfloat16, "cuda")
    W = inputs.randint((K, N), -3, 3, seed + 2, torch.bfloat16, "cuda")
    dY = inputs.randint((M, N), -3, 3, seed + 3, torch.bfloat16, "cuda")
    return X, W, dY


def _bits(t):
    b = out_bits(t)
    return b.view(np.uint32) if b.dtype == np.float32 else b


def test_graph_replays_match_eager():
    X, W, dY = _inputs(4000)
    X2, W2, dY2 = _inputs(4100)   # inputs of the eager calls between replays
    outs = [linear.alloc_out(op, sig, P, R, M, K, N, torch.bfloat16, "cuda")
            for _, sig, op, _ in CASES]
    bwd = [(linear.alloc_out("bwd_data", sig, P, R, M, K, N, torch.bfloat16, "cuda"),
            linear.alloc_out("bwd_weight", sig, P, R, M, K, N, torch.bfloat16, "cuda"))
           for sig in BWD_CASES]
    # an accumulating fp32 weight gradient (DP: dW is P, fp32)
    acc0 = inputs.randint((K, N), -8, 8, 4200, torch.float32, "cuda")
    acc = acc0.clone()
    acc_dx = linear.alloc_out("bwd_data", "DP", P, R, M, K, N, torch.bfloat16, "cuda")
    L_dp = linear.layouts("DP", P, R)

    def launch_all(stream):
        for (name, sig, op, ov), out in zip(CASES, outs):
            if ov is not None:
                sbp.sbp_set_plan_override(*ov)
            try:
                linear.run(op, sig, P, R, X, W, dY, out, stream)
            finally:
                sbp.sbp_set_plan_override(0, 0, 1, 0)
        for sig, (dX, dW) in zip(BWD_CASES, bwd):
            linear.run_bwd(sig, P, R, X, W, dY, dX, dW, stream)
        linear.run_bwd_L(L_dp, X, W, dY, acc_dx, acc, stream, accumulate_dw=True)

    stream = torch.cuda.Stream()
    sid = stream.cuda_stream
    say("graph: eager pass")
    with torch.cuda.stream(stream):
        launch_all(sid)
    torch.cuda.synchronize()
    want = [o.clone() for o in outs] + [t.clone() for pair in bwd for t in pair]
    want_acc = acc.clone()

    # the eager results are exact
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    for (name, sig, op, _), out in zip(CASES, outs):
        ref = oracle_full(op, sig, P, R, Xh, Wh, dYh)
        got = out_bits(out) if out.dtype == torch.bfloat16 else decode(out)
        exp = oracle.round_bf16(ref) if out.dtype == torch.bfloat16 else ref
        assert np.array_equal(got, exp), name
    for sig, (dX, dW) in zip(BWD_CASES, bwd):
        for op, out in (("bwd_data", dX), ("bwd_weight", dW)):
            ref = oracle_full(op, sig, P, R, Xh, Wh, dYh)
            got = out_bits(out) if out.dtype == torch.bfloat16 else decode(out)
            exp = oracle.round_bf16(ref) if out.dtype == torch.bfloat16 else ref
            assert np.array_equal(got, exp), (sig, op)
    ref_dw = oracle_full("bwd_weight", "DP", P, R, Xh, Wh, dYh)
    assert np.array_equal(decode(want_acc), decode(acc0) + ref_dw)

    say("graph: capture")
    graph = torch.cuda.CUDAGraph()
    acc.copy_(acc0)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=stream):
        launch_all(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()

    scratch = linear.alloc_out("bwd_data", "DP", P, R, M, K, N, torch.bfloat16, "cuda")
    for rep in range(4):
        for o in outs:
            o.fill_(7)
        for pair in bwd:
            for t in pair:
                t.fill_(7)
        acc.copy_(acc0)
        # other eager library work on the graph's stream: same workspace
        with torch.cuda.stream(stream):
            sbp.sbp_set_plan_override(128, 128, 6, 4, 0)
            try:
                linear.run("bwd_data", "DP", P, R, X2, W2, dY2, scratch, sid)
            finally:
                sbp.sbp_set_plan_override(0, 0, 1, 0)
        torch.cuda.synchronize()
        say("graph: replay", rep)
        with torch.cuda.stream(stream):
            graph.replay()
        torch.cuda.synchronize()
        got = outs + [t for pair in bwd for t in pair]
        for i, (g, w) in enumerate(zip(got, want)):
            assert np.array_equal(_bits(g), _bits(w)), (rep, i)
        assert np.array_equal(_bits(acc), _bits(want_acc)), rep


def test_capture_on_fresh_stream_without_eager_call():
    """Capture first, no eager warm-up: split plans, the grouped backward
    launch and the split reduction inside a graph on a stream the library has
    never seen; every replay is exact against the oracle."""
    X, W, dY = _inputs(4300)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    ws = torch.empty(sbp.SBP_WORKSPACE_BYTES, dtype=torch.uint8, device="cuda")
    cases = [c for c in CASES if c[3] is not None]
    outs = [linear.alloc_out(op, sig, P, R, M, K, N, torch.bfloat16, "cuda")
            for _, sig, op, _ in cases]
    bwd = [(linear.alloc_out("bwd_data", sig, P, R, M, K, N, torch.bfloat16, "cuda"),
            linear.alloc_out("bwd_weight", sig, P, R, M, K, N, torch.bfloat16, "cuda"))
           for sig in BWD_CASES]
    # the grouped plans of these pairs split their reductions
    for sig in BWD_CASES:
        L = linear.layouts(sig, P, R)
        say("fresh capture: %s backward plan" % sig,
            sbp.sbp_plan_bwd(*[int(v) for v in _pair_dims(L)]))
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    say("fresh capture: capture")
    with torch.cuda.graph(graph, stream=stream):
        sid = torch.cuda.current_stream().cuda_stream
        for (name, sig, op, ov), out in zip(cases, outs):
            sbp.sbp_set_plan_override(*ov)
            try:
                linear.run_L(op, linear.layouts(sig, P, R), X, W, dY, out, sid, ws=ws)
            finally:
                sbp.sbp_set_plan_override(0, 0, 1, 0)
        for sig, (dX, dW) in zip(BWD_CASES, bwd):
            sbp.sbp_set_plan_override(128, 128, 3, 4, 0)
            sbp.sbp_set_bwd_override(2, 4)
            try:
                linear.run_bwd_L(linear.layouts(sig, P, R), X, W, dY, dX, dW, sid, ws=ws)
            finally:
                sbp.sbp_set_plan_override(0, 0, 1, 0)
    torch.cuda.synchronize()
    for rep in range(3):
        for o in outs + [t for pair in bwd for t in pair]:
            o.fill_(7)
        torch.cuda.synchronize()
        say("fresh capture: replay", rep)
        with torch.cuda.stream(stream):
            graph.replay()
        torch.cuda.synchronize()
        checks = [(op, sig, out) for (_, sig, op, _), out in zip(cases, outs)]
        checks += [(op, sig, t) for sig, pair in zip(BWD_CASES, bwd)
                   for op, t in zip(("bwd_data", "bwd_weight"), pair)]
        for op, sig, out in checks:
            ref = oracle_full(op, sig, P, R, Xh, Wh, dYh)
            got = out_bits(out) if out.dtype == torch.bfloat16 else decode(out)
            exp = oracle.round_bf16(ref) if out.dtype == torch.bfloat16 else ref
            assert np.array_equal(got, exp), (rep, sig, op)


def _pair_dims(L):
    """(md, nd, kd, fp32 d, mw, nw, kw, fp32 w) of a backward pair at the test shape."""
    dx = linear.out_shape("bwd_data", L, M, K, N)
    dw = linear.out_shape("bwd_weight", L, M, K, N)
    kd = linear.shard(L["dy"], M, N).cols
    kw = linear.shard(L["x"], M, K).rows
    fd = 1 if linear.is_partial(L["dx"]) else 0
    fw = 1 if linear.is_partial(L["dw"]) else 0
    return dx[0], dx[1], kd, fd, dw[0], dw[1], kw, fw
