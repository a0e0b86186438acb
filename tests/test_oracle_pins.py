"""Pins for the CPU oracle, against things other than the oracle itself.

* numpy.array_split fixes the balanced contiguous split;
* the reassembly invariant of the SBP states (AutoDDL Sec. 1 partial-sum
  definition, Sec. 4.1 Fig. 5 caption, Sec. 4.2 SBP matmul): concatenating
  Split outputs, summing Partial-sum outputs and taking any copy of
  Broadcast outputs over all p ranks reproduces the global product, checked
  exactly against numpy integer products on integer inputs;
* p = 1 reduces every signature to the textbook product;
* closed forms on all-ones inputs;
* the gradient-state duality (Sec. 4.3: a broadcast weight receives
  partial-sum gradients);
* worked examples under tests/golden/ (Listing 1 shard shapes; a hand-worked
  K-split example);
* bf16 rounding against torch's own fp32 -> bf16 conversion;
* planted mistakes in copies of oracle.c are caught by the same checks.
"""
import json
import os
import re

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SIGS = (oracle.DP, oracle.COL, oracle.KS)
# signatures with a Partial-sum or replicated operand and no split
LINEAR_SIGS = (oracle.PB, oracle.BP, oracle.BB)
ALL_SIGS = SIGS + LINEAR_SIGS
OPS = (oracle.FWD, oracle.BWD_DATA, oracle.BWD_WEIGHT)


def _global_product(op, X, W, dY):
    if op == oracle.FWD:
        return X @ W
    if op == oracle.BWD_DATA:
        return dY @ W.T
    return X.T @ dY


def _reassemble(orc, sig, op, Xe, We, dYe, p, M, K, N):
    """Run every rank and combine by the output state; returns the global tensor
    (or raises AssertionError when Broadcast copies differ)."""
    parts = [orc.linear(sig, op, Xe, We, dYe, p, r) for r in range(p)]
    _, _, kind, axis = orc.out_shape(sig, op, M, K, N, p, 0)
    if kind == oracle.SPLIT:
        return np.concatenate(parts, axis=axis)
    if kind == oracle.PARTIAL:
        return np.sum(np.stack(parts), axis=0)
    for q in parts[1:]:
        assert np.array_equal(q, parts[0])
    return parts[0]


SHAPES = [(13, 7, 11), (8, 16, 4), (3, 5, 2), (1, 9, 6)]


def invariant_failures(orc, encs=("f32", "bf16")):
    """Every (signature, op, p, shape, encoding) where the reassembled oracle
    output differs from the exact global product of integer inputs."""
    bad = []
    rng = np.random.default_rng(7)
    for (M, K, N) in SHAPES:
        Xi = rng.integers(-3, 4, (M, K))
        Wi = rng.integers(-3, 4, (K, N))
        dYi = rng.integers(-3, 4, (M, N))
        for enc in encs:
            if enc == "f32":
                Xe, We, dYe = (a.astype(np.float32) for a in (Xi, Wi, dYi))
            else:
                Xe, We, dYe = (torch.tensor(a, dtype=torch.bfloat16).view(torch.int16)
                               .numpy().view(np.uint16) for a in (Xi, Wi, dYi))
            for sig in SIGS:
                for op in OPS:
                    want = _global_product(op, Xi, Wi, dYi)
                    for p in (1, 2, 3, 4, 8):
                        try:
                            got = _reassemble(orc, sig, op, Xe, We, dYe, p, M, K, N)
                            ok = got.shape == want.shape and np.array_equal(got, want)
                        except (AssertionError, ValueError):
                            ok = False
                        if not ok:
                            bad.append((sig, op, p, (M, K, N), enc))
    return bad


def test_split_matches_numpy_array_split(orc):
    for D in range(0, 41):
        for p in range(1, 10):
            chunks = np.array_split(np.arange(D), p)
            for r in range(p):
                off, ln = orc.split(D, p, r)
                assert ln == len(chunks[r])
                if ln:
                    assert off == chunks[r][0]
                else:
                    assert off == sum(len(c) for c in chunks[:r])


def test_reassembly_invariant_exact_integer_inputs(orc):
    assert invariant_failures(orc) == []


def test_reassembly_invariant_random_bf16(orc):
    # N(0,1) inputs rounded to bf16; exact products summed in fp64 agree with
    # numpy's fp64 product of the decoded inputs to fp64 rounding.
    M, K, N = 37, 29, 23
    g = torch.Generator().manual_seed(11)
    X, W, dY = (torch.randn(s, generator=g).to(torch.bfloat16) for s in ((M, K), (K, N), (M, N)))
    Xb, Wb, dYb = (t.view(torch.int16).numpy().view(np.uint16) for t in (X, W, dY))
    Xd, Wd, dYd = (t.double().numpy() for t in (X, W, dY))
    for sig in SIGS:
        for op in OPS:
            want = _global_product(op, Xd, Wd, dYd)
            for p in (2, 5, 8):
                got = _reassemble(orc, sig, op, Xb, Wb, dYb, p, M, K, N)
                np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_p1_is_textbook_product(orc):
    rng = np.random.default_rng(3)
    X, W, dY = (rng.standard_normal(s).astype(np.float32) for s in ((9, 6), (6, 5), (9, 5)))
    Xd, Wd, dYd = (a.astype(np.float64) for a in (X, W, dY))
    for sig in SIGS:
        for op in OPS:
            got = orc.linear(sig, op, X, W, dY, 1, 0)
            np.testing.assert_allclose(got, _global_product(op, Xd, Wd, dYd), rtol=1e-13)


def test_closed_form_all_ones(orc):
    # With all-ones inputs every output element is the length of the local
    # reduction: K_r for the forward, N_r for backward-data, M_r for backward-weight.
    M, K, N, p = 10, 7, 9, 4
    X, W, dY = (np.ones(s, np.float32) for s in ((M, K), (K, N), (M, N)))
    for r in range(p):
        _, k_r = orc.split(K, p, r)
        _, n_r = orc.split(N, p, r)
        _, m_r = orc.split(M, p, r)
        assert np.all(orc.linear(oracle.DP, oracle.FWD, X, W, dY, p, r) == K)
        assert np.all(orc.linear(oracle.COL, oracle.FWD, X, W, dY, p, r) == K)
        assert np.all(orc.linear(oracle.KS, oracle.FWD, X, W, dY, p, r) == k_r)
        assert np.all(orc.linear(oracle.DP, oracle.BWD_DATA, X, W, dY, p, r) == N)
        assert np.all(orc.linear(oracle.COL, oracle.BWD_DATA, X, W, dY, p, r) == n_r)
        assert np.all(orc.linear(oracle.KS, oracle.BWD_DATA, X, W, dY, p, r) == N)
        assert np.all(orc.linear(oracle.DP, oracle.BWD_WEIGHT, X, W, dY, p, r) == m_r)
        assert np.all(orc.linear(oracle.COL, oracle.BWD_WEIGHT, X, W, dY, p, r) == M)
        assert np.all(orc.linear(oracle.KS, oracle.BWD_WEIGHT, X, W, dY, p, r) == M)


def test_gradient_state_duality(orc):
    # grad of Split(i) is Split(i); grad of Broadcast is Partial-sum and vice
    # versa (Sec. 4.3 states the Broadcast-weight case).
    dual = {oracle.SPLIT: oracle.SPLIT, oracle.BCAST: oracle.PARTIAL, oracle.PARTIAL: oracle.BCAST}
    for sig in ALL_SIGS:
        t = orc.tags(sig)
        X, W, Y, dY, dX, dW = t
        for fwd, grad in ((X, dX), (W, dW), (Y, dY)):
            assert grad[0] == dual[fwd[0]]
            if fwd[0] == oracle.SPLIT:
                assert grad[1] == fwd[1]


def partial_parts(rng, T, p):
    """p integer tensors that sum to the integer tensor T (a Partial-sum
    state of T over p devices)."""
    parts = [rng.integers(-3, 4, T.shape) for _ in range(p - 1)]
    return parts + [T - sum(parts, np.zeros_like(T))]


def linear_sig_failures(orc):
    """(signature, op, p, shape) where the per-rank outputs of a signature with
    a Partial-sum or replicated operand, given per-rank partial inputs whose
    sum is the true tensor, do not reassemble into the exact global product
    (Partial-sum outputs summed, Broadcast outputs equal on every rank)."""
    bad = []
    rng = np.random.default_rng(9)
    for (M, K, N) in SHAPES:
        Xi, Wi, dYi = (rng.integers(-3, 4, s) for s in ((M, K), (K, N), (M, N)))
        for sig in LINEAR_SIGS:
            t = orc.tags(sig)
            for op in OPS:
                want = _global_product(op, Xi, Wi, dYi)
                for p in (1, 2, 3):
                    # inputs in Partial-sum state get per-rank partials
                    ins = []
                    for T, st in ((Xi, t[0]), (Wi, t[1]), (dYi, t[3])):
                        ins.append(partial_parts(rng, T, p) if st[0] == oracle.PARTIAL
                                   else [T] * p)
                    try:
                        outs = [orc.linear(sig, op, *(a[r].astype(np.float32) for a in ins), p, r)
                                for r in range(p)]
                        kind = orc.out_shape(sig, op, M, K, N, p, 0)[2]
                        if kind == oracle.PARTIAL:
                            got = np.sum(np.stack(outs), axis=0)
                        else:
                            assert all(np.array_equal(o, outs[0]) for o in outs)
                            got = outs[0]
                        ok = np.array_equal(got, want)
                    except (AssertionError, ValueError):
                        ok = False
                    if not ok:
                        bad.append((sig, op, p, (M, K, N)))
    return bad


def test_partial_and_replicated_signatures_reassemble(orc):
    # By linearity: (P, B) -> P and (B, P) -> P, (B, B) -> B; their backward
    # states follow the duality (a Broadcast tensor's gradient is Partial-sum)
    assert linear_sig_failures(orc) == []


def test_forward_rule_is_a_factor_of_the_3d_rule(orc):
    # Sec. 4.2: I ~ (S0:p0, B:p1, S1:p2), W ~ (B:p0, S1:p1, S0:p2),
    # O ~ (S0:p0, S1:p1, P:p2). Keeping one mesh axis gives one 1-D signature;
    # p1 = p2 = 1 is data parallelism.
    rule = {  # mesh axis -> (I state, W state, O state) as (kind, axis)
        0: ((oracle.SPLIT, 0), (oracle.BCAST, -1), (oracle.SPLIT, 0)),
        1: ((oracle.BCAST, -1), (oracle.SPLIT, 1), (oracle.SPLIT, 1)),
        2: ((oracle.SPLIT, 1), (oracle.SPLIT, 0), (oracle.PARTIAL, -1)),
    }
    for mesh_axis, sig in ((0, oracle.DP), (1, oracle.COL), (2, oracle.KS)):
        X, W, Y = orc.tags(sig)[:3]
        assert (X, W, Y) == rule[mesh_axis]


def test_golden_listing1_shard_shapes(orc):
    with open(os.path.join(GOLDEN, "listing1_shards.json")) as f:
        g = json.load(f)
    rows, cols = g["tensor_shape"]
    f_s1, f_s0, f_b = g["factors"]
    for r in range(f_s1["p"]):
        off, ln = orc.split(cols, f_s1["p"], r)
        assert (rows, ln) == tuple(f_s1["local_shape"]) and off == f_s1["col_offsets"][r]
    for r in range(f_s0["p"]):
        off, ln = orc.split(rows, f_s0["p"], r)
        assert (ln, cols) == tuple(f_s0["local_shape"]) and off == f_s0["row_offsets"][r]
    # composing the two split factors gives the 2 x 2 local block of every device
    for a in range(f_s1["p"]):
        for b in range(f_s0["p"]):
            _, nc = orc.split(cols, f_s1["p"], a)
            _, nr = orc.split(rows, f_s0["p"], b)
            assert [nr, nc] == g["composed_local_shape"]
    assert f_b["p"] == g["copies_per_block"]


def test_golden_ksplit_worked_example(orc):
    with open(os.path.join(GOLDEN, "ksplit_worked_example.json")) as f:
        g = json.load(f)
    X = np.array(g["X"], np.float32)
    W = np.array(g["W"], np.float32)
    p = g["p"]
    total = 0
    for r in range(p):
        part = orc.linear(oracle.KS, oracle.FWD, X, W, None, p, r)
        assert np.array_equal(part, np.array(g["partials"][r], np.float64))
        total = total + part
    assert np.array_equal(total, np.array(g["sum"], np.float64))
    _, _, kind, _ = orc.out_shape(oracle.KS, oracle.FWD, 2, 3, 2, p, 0)
    assert kind == oracle.PARTIAL


def test_samples_match_blocks(orc):
    rng = np.random.default_rng(5)
    M, K, N, p = 40, 24, 33, 3
    X, W, dY = (rng.standard_normal(s).astype(np.float32) for s in ((M, K), (K, N), (M, N)))
    for sig in SIGS:
        for op in OPS:
            for r in range(p):
                full = orc.linear(sig, op, X, W, dY, p, r)
                ii = rng.integers(0, full.shape[0], 50)
                jj = rng.integers(0, full.shape[1], 50)
                got = orc.linear_samples(sig, op, X, W, dY, p, r, ii, jj)
                assert np.array_equal(got, full[ii, jj])
                blk = orc.linear(sig, op, X, W, dY, p, r, rows=range(2, 7), cols=range(1, 4))
                assert np.array_equal(blk, full[2:7, 1:4])


def test_bad_arguments_raise(orc):
    X = np.ones((4, 4), np.float32)
    with pytest.raises(ValueError):
        orc.linear(6, 0, X, X, X, 2, 0)       # unknown signature
    with pytest.raises(ValueError):
        orc.linear(0, 0, X, X, X, 2, 2)       # rank out of range
    with pytest.raises(ValueError):
        orc.linear(0, 0, X, X, X, 2, 0, rows=range(0, 5))  # outside the output


def test_round_bf16_matches_torch_conversion(orc):
    # fp32 values (so fp64 -> bf16 and torch's fp32 -> bf16 round the same
    # number): random, exact ties in both directions, and near-ties.
    g = torch.Generator().manual_seed(9)
    vals = [torch.randn(4000, generator=g) * 10.0 ** torch.randint(-20, 20, (4000,), generator=g)]
    base = torch.randint(0, 1 << 16, (3000,), generator=g, dtype=torch.int32) << 16
    base = base[(base.view(torch.float32).isfinite())]
    for low in (0x8000, 0x7FFF, 0x8001, 0x0001, 0xFFFF):
        vals.append((base | low).view(torch.float32))
    v = torch.cat(vals)
    v = v[torch.isfinite(v) & (v.abs() > 1e-37) & (v.abs() < 3.3e38)]
    want = v.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = orc.round_bf16(v.double().numpy())
    assert np.array_equal(got, want)


MUTATIONS = [
    ("split offset ignores the remainder", "(r < rem ? r : rem)", "(r < rem ? r : 0)"),
    ("forward drops the last reduction term", "k < pl->x.nc; ++k", "k + 1 < pl->x.nc; ++k"),
    ("backward-weight sign flipped", "acc += decode(X, enc, (pl->x.r0 + t) * K + (pl->x.c0 + i))",
     "acc -= decode(X, enc, (pl->x.r0 + t) * K + (pl->x.c0 + i))"),
    ("forward reads a fixed column of X", "decode(X, enc, (pl->x.r0 + i) * K + (pl->x.c0 + k))",
     "decode(X, enc, (pl->x.r0 + i) * K + (pl->x.c0))"),
    ("data-parallel weight gradient tagged Broadcast",
     "{ORC_SPLIT,   ORC_BCAST,   ORC_SPLIT,   ORC_SPLIT,   ORC_SPLIT,   ORC_PARTIAL}",
     "{ORC_SPLIT,   ORC_BCAST,   ORC_SPLIT,   ORC_SPLIT,   ORC_SPLIT,   ORC_BCAST  }"),
    ("K-split output tagged Broadcast",
     "{ORC_SPLIT,   ORC_SPLIT,   ORC_PARTIAL, ORC_BCAST,   ORC_SPLIT,   ORC_SPLIT  }",
     "{ORC_SPLIT,   ORC_SPLIT,   ORC_BCAST,   ORC_BCAST,   ORC_SPLIT,   ORC_SPLIT  }"),
    ("replicated product's gradients tagged Broadcast",
     "{ORC_BCAST,   ORC_BCAST,   ORC_BCAST,   ORC_PARTIAL, ORC_PARTIAL, ORC_PARTIAL}",
     "{ORC_BCAST,   ORC_BCAST,   ORC_BCAST,   ORC_BCAST,   ORC_BCAST,   ORC_BCAST  }"),
    ("partial-input output tagged Broadcast",
     "{ORC_PARTIAL, ORC_BCAST,   ORC_PARTIAL, ORC_BCAST,   ORC_BCAST,   ORC_PARTIAL}",
     "{ORC_PARTIAL, ORC_BCAST,   ORC_BCAST,   ORC_BCAST,   ORC_BCAST,   ORC_PARTIAL}"),
]


def f32_failures(orc):
    """Pins of the fp32-accumulating loop (orc_linear_block_f32), each fixed
    by arithmetic rather than by the loop itself:
    * integer inputs: every partial sum is an integer below 2^24, so the fp32
      result equals the exact (fp64) one;
    * a reduction of length 1 (K-split with p = K): the result is the single
      product rounded once to fp32;
    * recursive summation in increasing reduction order: [2^24, 1, -2^24] .
      [1, 1, 1] gives fl(fl(2^24 + 1) - 2^24) = 0 in fp32, where the exact
      sum is 1 (any other order, or a wider accumulator, gives 1);
    * the error bound of recursive summation of products (Higham, Accuracy
      and Stability of Numerical Algorithms, Sec. 3.1): |c - s| <=
      gamma_n sum |a_k b_k|, gamma_n = n u / (1 - n u), u = 2^-24, for random
      inputs, every op."""
    bad = []
    rng = np.random.default_rng(11)
    M, K, N = 9, 14, 7
    Xi, Wi, dYi = (rng.integers(-3, 4, s).astype(np.float32) for s in ((M, K), (K, N), (M, N)))
    for sig in (oracle.DP, oracle.COL, oracle.KS):
        for op in OPS:
            a = orc.linear_f32(sig, op, Xi, Wi, dYi, 3, 1)
            b = orc.linear(sig, op, Xi, Wi, dYi, 3, 1)
            if a.dtype != np.float32 or not np.array_equal(a.astype(np.float64), b):
                bad.append(("integer", sig, op))
    X1 = rng.standard_normal((5, 4)).astype(np.float32)
    W1 = rng.standard_normal((4, 6)).astype(np.float32)
    for r in range(4):
        got = orc.linear_f32(oracle.KS, oracle.FWD, X1, W1, None, 4, r, N=6)
        want = (X1[:, r:r + 1].astype(np.float64) * W1[r:r + 1, :].astype(np.float64))
        if not np.array_equal(got, want.astype(np.float32)):
            bad.append(("single product", r))
    Xo = np.array([[2.0 ** 24, 1.0, -(2.0 ** 24)]], dtype=np.float32)
    Wo = np.ones((3, 1), dtype=np.float32)
    if orc.linear_f32(oracle.DP, oracle.FWD, Xo, Wo, None, 1, 0, N=1)[0, 0] != 0.0:
        bad.append("summation order")
    if orc.linear(oracle.DP, oracle.FWD, Xo, Wo, None, 1, 0, N=1)[0, 0] != 1.0:
        bad.append("exact reference of the order case")
    Xr = rng.standard_normal((12, 40)).astype(np.float32)
    Wr = rng.standard_normal((40, 10)).astype(np.float32)
    dYr = rng.standard_normal((12, 10)).astype(np.float32)
    u = 2.0 ** -24
    for op in OPS:
        got = orc.linear_f32(oracle.DP, op, Xr, Wr, dYr, 1, 0).astype(np.float64)
        exact = orc.linear(oracle.DP, op, Xr, Wr, dYr, 1, 0)
        absmag = orc.linear(oracle.DP, op, np.abs(Xr), np.abs(Wr), np.abs(dYr), 1, 0)
        n = {oracle.FWD: 40, oracle.BWD_DATA: 10, oracle.BWD_WEIGHT: 12}[op]
        gamma = n * u / (1 - n * u)
        # the fp64 reference's own error is far below this bound
        if np.any(np.abs(got - exact) > gamma * absmag * (1 + 1e-9)):
            bad.append(("error bound", op))
    return bad


def test_f32_accumulation_pins(orc):
    assert f32_failures(orc) == []


F32_MUTATIONS = [
    ("fp32 loop accumulates in fp64", "    float acc = 0.0f;", "    double acc = 0.0;"),
    ("fp32 loop sums in decreasing order", "        for (int64_t t = 0; t < pl->x.nc; ++t) {",
     "        for (int64_t t = pl->x.nc - 1; t >= 0; --t) {"),
    ("fp32 loop reads X's neighbour column",
     "(float)decode(X, enc, (pl->x.r0 + i) * K + (pl->x.c0 + t))",
     "(float)decode(X, enc, (pl->x.r0 + i) * K + (pl->x.c0 + t + 1) % K)"),
]


@pytest.mark.parametrize("name,old,new", F32_MUTATIONS, ids=[m[0] for m in F32_MUTATIONS])
def test_planted_f32_mistakes_are_caught(tmp_path, name, old, new):
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, "mutation anchor not found: " + name
    mut = tmp_path / "oracle_mut.c"
    mut.write_text(src.replace(old, new))
    lib = oracle.build(force=True, src=str(mut), out=str(tmp_path / "liboracle_mut.so"))
    assert f32_failures(oracle.Oracle(lib)), "planted mistake not caught: " + name


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistakes_are_caught(tmp_path, name, old, new):
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, "mutation anchor not found: " + name
    mut = tmp_path / "oracle_mut.c"
    mut.write_text(src.replace(old, new))
    lib = oracle.build(force=True, src=str(mut), out=str(tmp_path / "liboracle_mut.so"))
    bad = oracle.Oracle(lib)
    caught = bool(invariant_failures(bad, encs=("f32",))) or bool(linear_sig_failures(bad))
    if not caught:
        # a mistake in the state table shows up in the duality check instead
        try:
            test_gradient_state_duality(bad)
            test_forward_rule_is_a_factor_of_the_3d_rule(bad)
        except AssertionError:
            caught = True
    assert caught, "planted mistake not caught: " + name
