"""GPU parity with the oracle on the five workloads and on mid-size cases.

Tolerance (normwise over the compared elements, max|g - o| / max|o|):
2e-2 for bf16 inputs and 1e-5 for the fp32 path. At full workload sizes the
ranks that the benchmark times (rank 0; rank 1 too for the VGG head, whose
FC8 shards are misaligned) are compared element by element over whole
outputs, each product alone and the backward pair as one call; the other
ranks on a random sample of elements plus the corners. Integer inputs at
full step shapes, under the plans the benchmark launches (persistent grids,
grouped backward launches with split reductions, thousands of work items),
must match bit for bit. At mid sizes whole outputs are compared.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2301_06813_amd import inputs, linear, sbp, workloads

from helpers import (OP_ID, SIG_ID, decode, expect_state, normwise_rel, oracle_full, run_gpu,
                     say)

pytestmark = pytest.mark.gpu
OPS = ("fwd", "bwd_data", "bwd_weight")
TOL_BF16 = 2e-2
TOL_F32 = 1e-5


def test_tiny_fp32_all_ranks_and_reassembly():
    # Workload 1: fp32, p = 4, every signature and rank; the reassembled GPU
    # outputs also match the brute-force global products (fp64 numpy).
    for wl in workloads.tiny_fp32():
        (lin,) = wl.linears
        X, W, dY = workloads.make_tensors(lin, torch.float32, "cuda")
        Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
        Xd, Wd, dYd = (a.astype(np.float64) for a in (Xh, Wh, dYh))
        glob = {"fwd": Xd @ Wd, "bwd_data": dYd @ Wd.T, "bwd_weight": Xd.T @ dYd}
        for op in OPS:
            parts = []
            for r in wl.ranks:
                say("tiny fp32", lin.sig, op, r)
                out, st = run_gpu(op, lin.sig, wl.p, r, X, W, dY)
                expect_state(op, lin.sig, wl.p, r, st)
                got = decode(out)
                want = oracle_full(op, lin.sig, wl.p, r, Xh, Wh, dYh)
                assert normwise_rel(got, want) <= TOL_F32, (lin.sig, op, r)
                # the plain fp32 triple loop (fp32 accumulator, increasing k)
                want32 = oracle.linear_f32(SIG_ID[lin.sig], OP_ID[op], Xh, Wh, dYh, wl.p, r)
                assert normwise_rel(got, want32.astype(np.float64)) <= TOL_F32, (lin.sig, op, r)
                parts.append(got)
            _, _, kind, axis = oracle.out_shape(SIG_ID[lin.sig], OP_ID[op], lin.M, lin.K, lin.N,
                                                wl.p, 0)
            if kind == oracle.SPLIT:
                whole = np.concatenate(parts, axis=axis)
            else:
                whole = np.sum(np.stack(parts), axis=0)
            assert normwise_rel(whole, glob[op]) <= TOL_F32, (lin.sig, op)


@pytest.mark.parametrize("sig", ["DP", "COL", "KS"])
def test_midsize_bf16_full_outputs(sig):
    # several tiles in every dimension plus ragged tails and uneven shards
    M, K, N, p = 517, 389, 261, 3
    g = torch.Generator().manual_seed(77)
    X = torch.randn((M, K), generator=g).to(torch.bfloat16)
    W = (torch.randn((K, N), generator=g) / K ** 0.5).to(torch.bfloat16)
    dY = torch.randn((M, N), generator=g).to(torch.bfloat16)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    Xc, Wc, dYc = (t.cuda() for t in (X, W, dY))
    for r in range(p):
        for op in OPS:
            say("midsize", sig, op, r)
            out, st = run_gpu(op, sig, p, r, Xc, Wc, dYc)
            expect_state(op, sig, p, r, st)
            want = oracle_full(op, sig, p, r, Xh, Wh, dYh)
            assert normwise_rel(decode(out), want) <= TOL_BF16, (sig, op, r)


def _sampled_check(lin, wl, X, W, dY, Xh, Wh, dYh, ranks, nsamp=1500, seed=0):
    rng = np.random.default_rng(seed)
    worst = 0.0
    for r in ranks:
        for op in OPS:
            say(wl.name, lin.name, lin.sig, op, "rank", r)
            out, st = run_gpu(op, lin.sig, wl.p, r, X, W, dY)
            expect_state(op, lin.sig, wl.p, r, st)
            rows, cols = out.shape
            ii = rng.integers(0, rows, nsamp)
            jj = rng.integers(0, cols, nsamp)
            # always include the four corners (edge tiles)
            ii[:4] = [0, 0, rows - 1, rows - 1]
            jj[:4] = [0, cols - 1, 0, cols - 1]
            got = decode(out[torch.as_tensor(ii, device="cuda"), torch.as_tensor(jj, device="cuda")])
            want = oracle.linear_samples(SIG_ID[lin.sig], OP_ID[op], Xh, Wh, dYh, wl.p, r, ii, jj)
            rel = normwise_rel(got, want)
            worst = max(worst, rel)
            assert rel <= TOL_BF16, (wl.name, lin.name, op, r, rel)
            del out
    return worst


def _full_check(lin, wl, X, W, dY, Xh, Wh, dYh, r):
    """Rank r's whole outputs against the oracle, element by element: each
    product alone, then both backward products as one sbp_linear_bwd call
    (the benchmark's grouped launch where the plans say so)."""
    want = {}
    for op in OPS:
        say(wl.name, lin.name, lin.sig, op, "rank", r, "whole output")
        out, st = run_gpu(op, lin.sig, wl.p, r, X, W, dY)
        expect_state(op, lin.sig, wl.p, r, st)
        want[op] = oracle_full(op, lin.sig, wl.p, r, Xh, Wh, dYh)
        rel = normwise_rel(decode(out), want[op])
        assert rel <= TOL_BF16, (wl.name, lin.name, op, r, rel)
        del out
    say(wl.name, lin.name, lin.sig, "bwd pair", "rank", r, "whole outputs")
    dX, dW, (sx, sw) = linear.call_bwd(lin.sig, wl.p, r, X, W, dY)
    torch.cuda.synchronize()
    expect_state("bwd_data", lin.sig, wl.p, r, sx)
    expect_state("bwd_weight", lin.sig, wl.p, r, sw)
    for op, out in (("bwd_data", dX), ("bwd_weight", dW)):
        rel = normwise_rel(decode(out), want[op])
        assert rel <= TOL_BF16, (wl.name, lin.name, "pair", op, r, rel)
    del dX, dW


# ranks the benchmark's per-call reports time: compared over whole outputs
FULL_RANKS = {"ffn": (0,), "attention": (0,), "vgg": (0, 1)}


@pytest.mark.parametrize("make", [workloads.ffn_shard, workloads.attention_dp, workloads.vgg_head],
                         ids=["ffn", "attention", "vgg"])
def test_workload_full_size(make):
    wl = make()
    key = {2: "ffn", 3: "attention", 4: "vgg"}[wl.cid]
    full = FULL_RANKS[key]
    for lin in wl.linears:
        X, W, dY = workloads.make_tensors(lin, wl.dtype, "cpu")
        Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
        Xc, Wc, dYc = (t.cuda() for t in (X, W, dY))
        for r in full:
            _full_check(lin, wl, Xc, Wc, dYc, Xh, Wh, dYh, r)
        others = tuple(r for r in wl.ranks if r not in full)
        _sampled_check(lin, wl, Xc, Wc, dYc, Xh, Wh, dYh, others, seed=lin.seed_base)
        del Xc, Wc, dYc


def _one_per_shape(wl):
    """The first linear of each (signature, layer position) of a step: every
    distinct local product shape, hence every plan, the benchmark launches."""
    seen, picked = set(), []
    for lin in wl.linears:
        key = (lin.sig, lin.name.split("_", 1)[1])
        if key not in seen:
            seen.add(key)
            picked.append(lin)
    return picked


def test_transformer_step_full_outputs():
    # Workload 5 draws inputs on the GPU (as the benchmark does); one linear
    # per distinct (signature, qkv/out/fc1/fc2) on rank 0, whole outputs: the
    # forward and each backward product alone, and the backward pair as the
    # benchmark calls it.
    wl = workloads.transformer_step()
    picked = _one_per_shape(wl)
    assert {l.sig for l in picked} == {"DP", "COL", "KS"} and len(picked) >= 10
    for lin in picked:
        X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
        Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
        _full_check(lin, wl, X, W, dY, Xh, Wh, dYh, 0)
        del X, W, dY


def test_transformer_step_searched_full_outputs():
    # Workload 8: the same 96 linears with the signatures the strategy search
    # chooses (all DP): one linear per layer position on rank 0, whole outputs
    wl = workloads.transformer_step_searched()
    for lin in _one_per_shape(wl):
        X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
        Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
        _full_check(lin, wl, X, W, dY, Xh, Wh, dYh, 0)
        del X, W, dY


# (name, M, K, N, signature, op or "pair") at step shapes (8192 tokens,
# hidden 1024, ffn 4096, 8 devices, rank 0) whose benchmark plans stress the
# work distribution: the K-split forward with an 8192 x 4096 fp32 output
# (2048 tiles on a persistent grid of two workgroups per compute unit), the
# column-split backward pair (512 + 256 work items in one grouped launch,
# an 8-way split reduction), and a data-parallel forward with 128-wide
# reduction stages
EXACT_STEP_CASES = [("ks fc1 fwd", 8192, 1024, 4096, "KS", "fwd"),
                    ("col fc1 bwd pair", 8192, 1024, 4096, "COL", "pair"),
                    ("dp fc1 fwd", 8192, 1024, 4096, "DP", "fwd"),
                    ("ks fc2 bwd pair", 8192, 4096, 1024, "KS", "pair")]


@pytest.mark.parametrize("name,M,K,N,sig,op", EXACT_STEP_CASES,
                         ids=[c[0] for c in EXACT_STEP_CASES])
def test_exact_full_step_shapes(name, M, K, N, sig, op):
    """Integer inputs in [-3, 3]: every partial sum is an exact fp32 integer
    (|sum| <= 9 * 8192 < 2^24), so whole outputs match the oracle bit for bit
    (bf16 outputs: the oracle's rounding of the exact value)."""
    p, r = 8, 0
    seed = 7700 + 10 * EXACT_STEP_CASES.index((name, M, K, N, sig, op))
    X = inputs.randint((M, K), -3, 3, seed + 1, torch.bfloat16, "cuda")
    W = inputs.randint((K, N), -3, 3, seed + 2, torch.bfloat16, "cuda")
    dY = inputs.randint((M, N), -3, 3, seed + 3, torch.bfloat16, "cuda")
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    if op == "pair":
        L = linear.layouts(sig, p, r)
        dx = linear.out_shape("bwd_data", L, M, K, N)
        dw = linear.out_shape("bwd_weight", L, M, K, N)
        plan = sbp.sbp_plan_bwd(dx[0], dx[1], linear.shard(L["dy"], M, N).cols,
                                sbp.SBP_F32 if linear.is_partial(L["dx"]) else sbp.SBP_BF16,
                                dw[0], dw[1], linear.shard(L["x"], M, K).rows,
                                sbp.SBP_F32 if linear.is_partial(L["dw"]) else sbp.SBP_BF16)
        say(name, "plan (grouped, tile, tile, splits dX, splits dW)", plan)
        assert plan[0] == 1 and max(plan[3], plan[4]) > 1
        dX, dW, _ = linear.call_bwd(sig, p, r, X, W, dY)
        torch.cuda.synchronize()
        outs = (("bwd_data", dX), ("bwd_weight", dW))
    else:
        say(name, "plan", sbp.sbp_plan(OP_ID[op], *_mnk(op, sig, p, r, M, K, N),
                                       sbp.SBP_BF16, sbp.SBP_F32 if sig == "KS" else sbp.SBP_BF16))
        out, _ = run_gpu(op, sig, p, r, X, W, dY)
        outs = ((op, out),)
    for o, out in outs:
        ref = oracle_full(o, sig, p, r, Xh, Wh, dYh)
        if out.dtype == torch.bfloat16:
            assert np.array_equal(inputs.host_bits(out), oracle.round_bf16(ref)), (name, o)
        else:
            assert np.array_equal(decode(out), ref), (name, o)


def _mnk(op, sig, p, r, M, K, N):
    L = linear.layouts(sig, p, r)
    m, n = linear.out_shape(op, L, M, K, N)
    k = {"fwd": linear.shard(L["x"], M, K).cols, "bwd_data": linear.shard(L["dy"], M, N).cols,
         "bwd_weight": linear.shard(L["x"], M, K).rows}[op]
    return m, n, k
