"""GPU parity with the oracle on the five workloads and on mid-size cases.

Tolerance (normwise over the compared elements, max|g - o| / max|o|):
2e-2 for bf16 inputs and 1e-5 for the fp32 path. At full workload sizes the
oracle computes a random sample of output elements one by one (same launch
configuration as the benchmark); at mid sizes it computes whole outputs.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2301_06813_amd import inputs, linear, workloads

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


@pytest.mark.parametrize("make", [workloads.ffn_shard, workloads.attention_dp, workloads.vgg_head],
                         ids=["ffn", "attention", "vgg"])
def test_workload_full_size_sampled(make):
    wl = make()
    for lin in wl.linears:
        X, W, dY = workloads.make_tensors(lin, wl.dtype, "cpu")
        Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
        Xc, Wc, dYc = (t.cuda() for t in (X, W, dY))
        _sampled_check(lin, wl, Xc, Wc, dYc, Xh, Wh, dYh, wl.ranks, seed=lin.seed_base)
        del Xc, Wc, dYc


def _sampled_bwd_pair(lin, wl, X, W, dY, Xh, Wh, dYh, r, nsamp, seed):
    """Both backward products through sbp_linear_bwd (one grouped launch where
    the tuned plans say so), as the benchmark calls them; sampled outputs."""
    rng = np.random.default_rng(seed)
    say(wl.name, lin.name, lin.sig, "bwd pair", "rank", r)
    dX, dW, (sx, sw) = linear.call_bwd(lin.sig, wl.p, r, X, W, dY)
    torch.cuda.synchronize()
    expect_state("bwd_data", lin.sig, wl.p, r, sx)
    expect_state("bwd_weight", lin.sig, wl.p, r, sw)
    for op, out in (("bwd_data", dX), ("bwd_weight", dW)):
        rows, cols = out.shape
        ii = rng.integers(0, rows, nsamp)
        jj = rng.integers(0, cols, nsamp)
        ii[:4] = [0, 0, rows - 1, rows - 1]
        jj[:4] = [0, cols - 1, 0, cols - 1]
        got = decode(out[torch.as_tensor(ii, device="cuda"), torch.as_tensor(jj, device="cuda")])
        want = oracle.linear_samples(SIG_ID[lin.sig], OP_ID[op], Xh, Wh, dYh, wl.p, r, ii, jj)
        rel = normwise_rel(got, want)
        assert rel <= TOL_BF16, (wl.name, lin.name, "pair", op, r, rel)


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


def test_transformer_step_sampled_linears():
    # Workload 5 draws inputs on the GPU (as the benchmark does); one linear
    # per distinct (signature, qkv/out/fc1/fc2) on rank 0: the forward and
    # each backward product alone, and the backward pair as the benchmark
    # calls it.
    wl = workloads.transformer_step()
    picked = _one_per_shape(wl)
    assert {l.sig for l in picked} == {"DP", "COL", "KS"} and len(picked) >= 10
    for lin in picked:
        X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
        Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
        _sampled_check(lin, wl, X, W, dY, Xh, Wh, dYh, (0,), nsamp=800, seed=lin.seed_base)
        _sampled_bwd_pair(lin, wl, X, W, dY, Xh, Wh, dYh, 0, 800, lin.seed_base + 1)
        del X, W, dY


def test_transformer_step_searched_sampled_linears():
    # Workload 8: the same 96 linears with the signatures the strategy search
    # chooses (all DP): one linear per layer position on rank 0, also as a
    # backward pair
    wl = workloads.transformer_step_searched()
    for lin in _one_per_shape(wl):
        X, W, dY = workloads.make_tensors(lin, wl.dtype, "cuda")
        Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
        _sampled_check(lin, wl, X, W, dY, Xh, Wh, dYh, (0,), nsamp=600, seed=lin.seed_base)
        _sampled_bwd_pair(lin, wl, X, W, dY, Xh, Wh, dYh, 0, 600, lin.seed_base + 1)
        del X, W, dY
