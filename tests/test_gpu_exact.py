"""Bit-exact GPU checks through the C ABI.

Integer inputs in [-3, 3] make every product and every partial sum an exact
fp32 integer (|sum| <= 9 K < 2^24), so the library's fp32 result must equal
the oracle's exactly in any summation order, and a bf16 output must equal
the oracle's round-to-nearest-even of that exact integer. This covers every
signature, operation, tile shape and split count, ragged sizes, uneven
shards and misaligned shard views.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2301_06813_amd import inputs, linear, sbp

from helpers import (EXTRA_TILE_KERNELS, KERNELS, TILES, decode, expect_state, oracle_full,
                     out_bits, run_gpu, say)

pytestmark = pytest.mark.gpu
SIGS = ("DP", "COL", "KS")
OPS = ("fwd", "bwd_data", "bwd_weight")


def _int_inputs(M, K, N, seed, device="cuda"):
    X = inputs.randint((M, K), -3, 3, seed + 1, torch.bfloat16, device)
    W = inputs.randint((K, N), -3, 3, seed + 2, torch.bfloat16, device)
    dY = inputs.randint((M, N), -3, 3, seed + 3, torch.bfloat16, device)
    return X, W, dY


def _check_exact(op, sig, p, r, X, W, dY, Xh, Wh, dYh):
    out, st = run_gpu(op, sig, p, r, X, W, dY)
    expect_state(op, sig, p, r, st)
    want = oracle_full(op, sig, p, r, Xh, Wh, dYh)
    assert out.shape == want.shape, (op, sig, p, r, out.shape, want.shape)
    if out.dtype == torch.bfloat16:
        assert np.array_equal(out_bits(out), oracle.round_bf16(want)), (op, sig, p, r)
    else:
        assert np.array_equal(decode(out), want), (op, sig, p, r)


@pytest.mark.parametrize("shape", [(300, 1000, 270), (64, 64, 64), (1, 70, 9), (517, 129, 33)])
def test_exact_all_signatures_default_plan(shape):
    M, K, N = shape
    X, W, dY = _int_inputs(M, K, N, 100)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    for p in (1, 3, 8):
        for r in sorted({0, p // 2, p - 1}):
            for sig in SIGS:
                for op in OPS:
                    say("exact", shape, p, r, sig, op)
                    _check_exact(op, sig, p, r, X, W, dY, Xh, Wh, dYh)


@pytest.mark.parametrize("shape", [(300, 1000, 270), (1, 70, 9)])
def test_exact_partial_and_replicated_signatures(shape):
    # (P,B)->P, (B,P)->P, (B,B)->B: full-size local operands on every rank
    M, K, N = shape
    X, W, dY = _int_inputs(M, K, N, 150)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    for p in (1, 4):
        for r in sorted({0, p - 1}):
            for sig in ("PB", "BP", "BB"):
                for op in OPS:
                    say("exact", shape, p, r, sig, op)
                    _check_exact(op, sig, p, r, X, W, dY, Xh, Wh, dYh)
                say("exact bwd pair", shape, p, r, sig)
                _check_exact_bwd(sig, p, r, X, W, dY, Xh, Wh, dYh)


def _accumulate_case(op, sig, p, r, X, W, dY, Xh, Wh, dYh, seed):
    """An fp32 output holding integers gets the product added (SBP_ACCUMULATE);
    the result must equal old + the oracle's product exactly."""
    L = linear.layouts(sig, p, r)
    M, K = X.shape
    N = W.shape[1]
    rows, cols = linear.out_shape(op, L, M, K, N)
    old = inputs.randint((rows, cols), -8, 8, seed, torch.float32, "cuda")
    out = old.clone()
    linear.run_L(op, L, X, W, dY, out, accumulate=True)
    torch.cuda.synchronize()
    want = old.double().cpu().numpy() + oracle_full(op, sig, p, r, Xh, Wh, dYh)
    assert np.array_equal(decode(out), want), (op, sig, p, r)


# (tile, kernel, splits) plans that reach every epilogue: direct, staged,
# row-quad, the generic kernel, and the split reduction
ACC_PLANS = [None, ((128, 128), 1, 1), ((128, 128), 1, 3), ((128, 128), 5, 1), ((64, 64), 7, 1),
             ((256, 256), 6, 1), ((128, 128), 2, 1), ((64, 64), 2, 2)]


@pytest.mark.parametrize("plan", ACC_PLANS, ids=[str(p_) for p_ in ACC_PLANS])
def test_exact_accumulate(plan):
    M, K, N = 304, 1104, 272
    X, W, dY = _int_inputs(M, K, N, 300)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    try:
        if plan is not None:
            (bm, bn), code, splits = plan
            sbp.sbp_set_plan_override(bm, bn, splits, code)
        for p, r in ((2, 1), (3, 0)):
            for sig in ("DP", "COL", "KS", "PB"):
                for op in OPS:
                    say("accumulate", plan, p, r, sig, op)
                    _accumulate_case(op, sig, p, r, X, W, dY, Xh, Wh, dYh, 310 + r)
    finally:
        sbp.sbp_set_plan_override(0, 0, 1)


def test_exact_accumulate_grouped_backward():
    # gradient accumulation over two micro-batches through the two-product
    # call: dW = X1^T dY1 + X2^T dY2 (dX overwritten each time)
    M, K, N = 256, 384, 320
    X1, W, dY1 = _int_inputs(M, K, N, 400)
    X2, _, dY2 = _int_inputs(M, K, N, 410)
    for grouped in (1, 2):
        for sig, p, r in (("DP", 4, 1), ("KS", 2, 0), ("COL", 4, 3)):
            say("accumulate grouped", grouped, sig, p, r)
            L = linear.layouts(sig, p, r)
            dX = linear.alloc_out("bwd_data", sig, p, r, M, K, N, X1.dtype, "cuda")
            dW = linear.alloc_out("bwd_weight", sig, p, r, M, K, N, X1.dtype, "cuda").float()
            dW.zero_()
            try:
                sbp.sbp_set_plan_override(128, 128, 2, 1)
                sbp.sbp_set_bwd_override(grouped, 3)
                for X, dY in ((X1, dY1), (X2, dY2)):
                    linear.run_bwd_L(L, X, W, dY, dX, dW, accumulate_dw=True)
                torch.cuda.synchronize()
            finally:
                sbp.sbp_set_plan_override(0, 0, 1)
            want = sum(oracle_full("bwd_weight", sig, p, r, *(inputs.host_bits(t) for t in
                                                              (X, W, dY)))
                       for X, dY in ((X1, dY1), (X2, dY2)))
            assert np.array_equal(decode(dW), want), (grouped, sig)
            want_dx = oracle_full("bwd_data", sig, p, r, *(inputs.host_bits(t) for t in
                                                          (X2, W, dY2)))
            got_dx = decode(dX)
            if dX.dtype == torch.bfloat16:
                assert np.array_equal(out_bits(dX), oracle.round_bf16(want_dx))
            else:
                assert np.array_equal(got_dx, want_dx)


def test_exact_accumulate_fp32_inputs():
    g = torch.Generator().manual_seed(5)
    X, W, dY = (torch.randint(-3, 4, s, generator=g).float().cuda() for s in
                ((64, 128), (128, 256), (64, 256)))
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    for sig in ("DP", "COL", "KS"):
        for op in OPS:
            say("accumulate fp32", sig, op)
            _accumulate_case(op, sig, 4, 2, X, W, dY, Xh, Wh, dYh, 500)


TILE_KERNELS = [(t, k) for k in KERNELS for t in TILES] + EXTRA_TILE_KERNELS
TK_IDS = ["%dx%d-k%d" % (t[0], t[1], k) for t, k in TILE_KERNELS]


@pytest.mark.parametrize("tile,kernel", TILE_KERNELS, ids=TK_IDS)
def test_exact_every_tile_and_split(tile, kernel):
    # sizes are multiples of 8 (so the pipelined kernel is eligible) but not
    # of any tile: every dimension has a ragged last tile
    M, K, N = 304, 1104, 272
    X, W, dY = _int_inputs(M, K, N, 200)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    p, r = 2, 1
    try:
        for splits in (1, 3, 7):
            sbp.sbp_set_plan_override(tile[0], tile[1], splits, kernel)
            for sig in SIGS:
                for op in OPS:
                    say("tile", tile, "kernel", kernel, "splits", splits, sig, op)
                    _check_exact(op, sig, p, r, X, W, dY, Xh, Wh, dYh)
    finally:
        sbp.sbp_set_plan_override(0, 0, 1)


def _check_exact_bwd(sig, p, r, X, W, dY, Xh, Wh, dYh):
    dX, dW, (sx, sw) = linear.call_bwd(sig, p, r, X, W, dY)
    torch.cuda.synchronize()
    expect_state("bwd_data", sig, p, r, sx)
    expect_state("bwd_weight", sig, p, r, sw)
    for op, out in (("bwd_data", dX), ("bwd_weight", dW)):
        want = oracle_full(op, sig, p, r, Xh, Wh, dYh)
        assert out.shape == want.shape
        if out.dtype == torch.bfloat16:
            assert np.array_equal(out_bits(out), oracle.round_bf16(want)), (op, sig, p, r)
        else:
            assert np.array_equal(decode(out), want), (op, sig, p, r)


@pytest.mark.parametrize("shape", [(304, 1104, 272), (300, 1000, 270), (8192, 256, 1024)])
def test_exact_grouped_backward_default_plan(shape):
    # sbp_linear_bwd: one grouped launch when eligible (multiples of 8),
    # separate launches otherwise; both outputs exact
    M, K, N = shape
    X, W, dY = _int_inputs(M, K, N, 800)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    for p in (1, 2, 8):
        for r in sorted({0, p - 1}):
            for sig in SIGS:
                say("grouped bwd", shape, p, r, sig)
                _check_exact_bwd(sig, p, r, X, W, dY, Xh, Wh, dYh)


GROUP_TILES = [(t, 1) for t in TILES] + EXTRA_TILE_KERNELS


@pytest.mark.parametrize("tile,kernel", GROUP_TILES,
                         ids=["%dx%d-k%d" % (t[0], t[1], k) for t, k in GROUP_TILES])
def test_exact_grouped_backward_every_tile(tile, kernel):
    M, K, N = 304, 1104, 272
    X, W, dY = _int_inputs(M, K, N, 900)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    try:
        for splits in (1, 3):
            sbp.sbp_set_plan_override(tile[0], tile[1], splits, kernel)
            for sig in SIGS:
                say("grouped bwd tile", tile, splits, sig)
                _check_exact_bwd(sig, 2, 1, X, W, dY, Xh, Wh, dYh)
    finally:
        sbp.sbp_set_plan_override(0, 0, 1)


def test_exact_long_reduction_split():
    # reduction of 8192 (the longest in the workloads), |sum| <= 9 * 8192 < 2^24
    M, K, N = 8192, 256, 200
    X, W, dY = _int_inputs(M, K, N, 300)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    for sig in ("COL", "KS"):
        say("long reduction", sig)
        _check_exact("bwd_weight", sig, 8, 3, X, W, dY, Xh, Wh, dYh)


def test_exact_misaligned_column_shards():
    # COL with N = 1000 over 8 ranks: W and dY column shards start at 125 r,
    # i.e. byte offsets 250 r, not 16-byte aligned for odd r.
    M, K, N = 96, 256, 1000
    X, W, dY = _int_inputs(M, K, N, 400)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    for r in range(8):
        for op in OPS:
            say("misaligned", r, op)
            _check_exact(op, "COL", 8, r, X, W, dY, Xh, Wh, dYh)


# the instances with a shifted form: direct and staged epilogues, 64- and
# 128-wide stages, one and two reduction groups
SHIFT_INSTANCES = [((64, 64), 1), ((128, 128), 4), ((64, 64), 12), ((128, 64), 12),
                   ((64, 128), 12), ((128, 128), 12)]


@pytest.mark.parametrize("tile,kernel", SHIFT_INSTANCES,
                         ids=["%dx%d-k%d" % (t[0], t[1], k) for t, k in SHIFT_INSTANCES])
def test_exact_shifted_operand_views(tile, kernel):
    """Shards that start inside a 16-byte block run on the pipelined kernel
    in a shifted index space: the column shards of a 1000-wide W and dY over
    8 ranks (125 r, as the VGG head's FC8) -- an n-major operand shifted
    along the output columns (forward, backward-weight) and both k-major
    operands shifted along a 125-long reduction (backward-data, with its
    boundary chunks masked) -- and the K split of a 1000-wide X (an m-major
    operand shifted along the output rows, backward-weight). Every rank,
    splits 1 and 3, the backward pair as one grouped launch; the profile
    shows the pipelined kernel ran (its shifted form on the ranks whose
    shards need it); results bit-exact. An instance without a shifted form
    falls back to the generic kernel on those ranks."""
    M, K, N, p = 200, 1000, 1000, 8
    X, W, dY = _int_inputs(M, K, N, 1700)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    cases = [("COL", "fwd"), ("COL", "bwd_data"), ("COL", "bwd_weight"), ("KS", "bwd_weight"),
             ("KS", "bwd_data")]
    try:
        for splits in (1, 3):
            sbp.sbp_set_plan_override(tile[0], tile[1], splits, kernel)
            for r in range(p):
                for sig, op in cases:
                    say("shifted", tile, kernel, splits, r, sig, op)
                    names = _kernel_names(
                        lambda: _check_exact(op, sig, p, r, X, W, dY, Xh, Wh, dYh))
                    assert any(n.startswith("gemm_bf16_dma_kernel") for n in names), names
                    # 125-wide shards: every product except the K split's
                    # backward-data (aligned operands, a 1000-long reduction)
                    # needs the shifted form, whose kernel name has a twelfth
                    # template argument
                    shifted = any(n.startswith("gemm_bf16_dma_kernel") and n.count(",") == 11
                                  for n in names)
                    assert shifted == (not (sig == "KS" and op == "bwd_data")), names
                sbp.sbp_set_bwd_override(2, splits)
                names = _kernel_names(lambda: _check_exact_bwd("COL", p, r, X, W, dY, Xh, Wh, dYh))
                assert any(n.startswith("gemm_bf16_dma_bwd_kernel") for n in names), names
                sbp.sbp_set_bwd_override(0, 1)
    finally:
        sbp.sbp_set_plan_override(0, 0, 1)


def test_exact_local_scope_padded_ld():
    # LOCAL views with ld > cols and an odd element offset; the result must
    # equal the GLOBAL-scope call on the same share.
    M, K, N, p, r = 130, 96, 72, 4, 2
    X, W, dY = _int_inputs(M, K, N, 500)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    want = oracle_full("fwd", "DP", p, r, Xh, Wh, dYh)
    sh = sbp.sbp_shard_index(sbp.split(0, p, r), M, K)
    buf = torch.zeros((sh.rows + 1, K + 9), dtype=torch.bfloat16, device="cuda")
    Xr = buf[1:, 3:3 + K]
    Xr.copy_(X[sh.row_off:sh.row_off + sh.rows])
    out = torch.empty((sh.rows, N), dtype=torch.float32, device="cuda")
    L = linear.layouts("DP", p, r)
    sbp.sbp_linear_fwd(sbp.view(Xr, sbp.SBP_LOCAL), L["x"], sbp.view(W), L["w"],
                       sbp.view(out, sbp.SBP_LOCAL))
    torch.cuda.synchronize()
    assert np.array_equal(decode(out), want)


def test_k_zero_share_writes_zeros():
    # K = 3 over p = 4: rank 3 holds an empty reduction share, so its
    # Partial-sum forward output is all zeros (and must be written).
    M, K, N, p, r = 40, 3, 50, 4, 3
    X, W, dY = _int_inputs(M, K, N, 600)
    out = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    linear.run("fwd", "KS", p, r, X, W, dY, out)
    torch.cuda.synchronize()
    assert torch.all(out == 0)


def test_shard_readback_identity():
    # With an identity weight the forward output is the selected share of X,
    # bit for bit (x 1.0 and + 0.0 are exact): checks the shard views through
    # the kernel for every signature and rank.
    M, K, p = 200, 136, 8
    g = torch.Generator(device="cuda").manual_seed(7)
    X = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    I = torch.eye(K, dtype=torch.bfloat16, device="cuda")
    for r in range(p):
        for sig in SIGS:
            say("readback", sig, r)
            out, _ = run_gpu("fwd", sig, p, r, X, I, None)
            xs = sbp.sbp_shard_index(linear.layouts(sig, p, r)["x"], M, K)
            ws = sbp.sbp_shard_index(linear.layouts(sig, p, r)["w"], K, K)
            want = torch.zeros((xs.rows, ws.cols), dtype=torch.float32, device="cuda")
            # X_r I_r: the columns of X_r that meet the ones of the identity share
            Xr = X[xs.row_off:xs.row_off + xs.rows, xs.col_off:xs.col_off + xs.cols].float()
            for j in range(ws.cols):
                kk = ws.col_off + j - ws.row_off
                if 0 <= kk < xs.cols:
                    want[:, j] = Xr[:, kk]
            assert torch.equal(out.float(), want), (sig, r)


def test_guard_bands_untouched():
    # Outputs inside a NaN-filled buffer (ld > cols, rows above and below):
    # the guard stays NaN and every element of the share is written.
    M, K, N, p = 150, 200, 140, 3
    X, W, dY = _int_inputs(M, K, N, 700)
    for tile, kernel in TILE_KERNELS:
        sbp.sbp_set_plan_override(tile[0], tile[1], 2, kernel)
        try:
            for sig in SIGS:
                for op in OPS:
                    r = 1
                    L = linear.layouts(sig, p, r)
                    rows, cols = linear.out_shape(op, L, M, K, N)
                    dt = linear.out_dtype(op, L, torch.bfloat16)
                    buf = torch.full((rows + 2, cols + 7), float("nan"), dtype=dt, device="cuda")
                    out = buf[1:rows + 1, 2:2 + cols]
                    linear.run(op, sig, p, r, X, W, dY, out)
                    torch.cuda.synchronize()
                    guard = torch.ones_like(buf, dtype=torch.bool)
                    guard[1:rows + 1, 2:2 + cols] = False
                    assert torch.all(torch.isnan(buf[guard])), (tile, kernel, sig, op)
                    assert not torch.any(torch.isnan(out)), (tile, kernel, sig, op)
        finally:
            sbp.sbp_set_plan_override(0, 0, 1)


def _guarded(rows, cols, dt, extra_ld, col_off):
    """A NaN canvas with the output view inside it: one guard row above and
    below, col_off guard columns on the left and the rest of the row (ld =
    cols + extra_ld) on the right."""
    buf = torch.full((rows + 2, cols + extra_ld), float("nan"), dtype=dt, device="cuda")
    out = buf[1:rows + 1, col_off:col_off + cols]
    guard = torch.ones_like(buf, dtype=torch.bool)
    guard[1:rows + 1, col_off:col_off + cols] = False
    return buf, out, guard


def _kernel_names(fn):
    """Names of the kernels the library launches in fn()."""
    sbp.sbp_profile_begin(8)
    try:
        fn()
    finally:
        names = [n for n, _ in sbp.sbp_profile_end(8)]
    return names


# pipelined instances (kernel codes other than the generic 2), each with a
# split reduction, plus persistent launches of two of them
PIPE_CASES = [(t, k, 0) for (t, k) in TILE_KERNELS if k != 2] + [((128, 128), 1, 2),
                                                               ((64, 64), 12, 1)]


@pytest.mark.parametrize("extra_ld,col_off", [(7, 2), (8, 8)], ids=["unaligned", "aligned"])
def test_guard_bands_pipelined_kernels(extra_ld, col_off):
    """Shapes every pipelined instance can read (all shares and leading
    dimensions multiples of 8): outputs inside a NaN canvas keep the canvas
    NaN and are exact, through each epilogue (direct, staged, row-quad; split
    partials and their reduction; persistent grids) and the grouped backward
    launch. The profile of each call shows that a pipelined kernel ran. The
    aligned canvas takes the 16-byte store paths, the unaligned one the
    element stores."""
    M, K, N, p, r = 176, 208, 144, 2, 1
    X, W, dY = _int_inputs(M, K, N, 720)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    for tile, kernel, occ in PIPE_CASES:
        sbp.sbp_set_plan_override(tile[0], tile[1], 2, kernel, occ)
        try:
            for sig in SIGS:
                L = linear.layouts(sig, p, r)
                for op in OPS:
                    rows, cols = linear.out_shape(op, L, M, K, N)
                    dt = linear.out_dtype(op, L, torch.bfloat16)
                    buf, out, guard = _guarded(rows, cols, dt, extra_ld, col_off)
                    names = _kernel_names(lambda: linear.run(op, sig, p, r, X, W, dY, out))
                    torch.cuda.synchronize()
                    assert any(n.startswith("gemm_bf16_dma_kernel") for n in names), names
                    assert torch.all(torch.isnan(buf[guard])), (tile, kernel, occ, sig, op)
                    want = oracle_full(op, sig, p, r, Xh, Wh, dYh)
                    got = out_bits(out) if dt == torch.bfloat16 else decode(out)
                    exp = oracle.round_bf16(want) if dt == torch.bfloat16 else want
                    assert np.array_equal(got, exp), (tile, kernel, occ, sig, op)
                if occ:
                    continue
                # both backward products in one grouped launch, each split
                sbp.sbp_set_bwd_override(2, 3)
                bufs = {}
                for op in ("bwd_data", "bwd_weight"):
                    rows, cols = linear.out_shape(op, L, M, K, N)
                    bufs[op] = _guarded(rows, cols, linear.out_dtype(op, L, torch.bfloat16),
                                        extra_ld, col_off)
                names = _kernel_names(lambda: linear.run_bwd(
                    sig, p, r, X, W, dY, bufs["bwd_data"][1], bufs["bwd_weight"][1]))
                torch.cuda.synchronize()
                assert any(n.startswith("gemm_bf16_dma_bwd_kernel") for n in names), names
                for op, (buf, out, guard) in bufs.items():
                    assert torch.all(torch.isnan(buf[guard])), (tile, kernel, sig, "pair", op)
                    want = oracle_full(op, sig, p, r, Xh, Wh, dYh)
                    got = out_bits(out) if out.dtype == torch.bfloat16 else decode(out)
                    exp = oracle.round_bf16(want) if out.dtype == torch.bfloat16 else want
                    assert np.array_equal(got, exp), (tile, kernel, sig, "pair", op)
        finally:
            sbp.sbp_set_plan_override(0, 0, 1)


def test_split_reduction_is_deterministic():
    M, K, N = 384, 4096, 320
    g = torch.Generator(device="cuda").manual_seed(3)
    X = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    dY = torch.randn((M, N), generator=g, device="cuda").to(torch.bfloat16)
    try:
        for sig, kernel in (("DP", 1), ("COL", 1), ("DP", 2), ("COL", 2)):
            sbp.sbp_set_plan_override(128, 128, 5, kernel)
            a, _ = run_gpu("bwd_weight", sig, 1, 0, X, None, dY)
            b, _ = run_gpu("bwd_weight", sig, 1, 0, X, None, dY)
            assert torch.equal(a, b)
    finally:
        sbp.sbp_set_plan_override(0, 0, 1)


PERSISTENT = [((128, 128), 1), ((256, 256), 6), ((128, 128), 6), ((128, 128), 7),
              ((256, 128), 7), ((128, 256), 7), ((256, 256), 8), ((128, 128), 9)]


def test_exact_persistent_launches():
    # grids capped at one workgroup per compute unit: each workgroup takes
    # several work items in turn (more items than compute units), reusing its
    # LDS pipeline and leaving each item's stores in flight
    M, K, N = 4096, 200, 2176
    X, W, dY = _int_inputs(M, K, N, 1300)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    cases = [("DP", 1, 0), ("KS", 2, 1)]
    want = {(sig, op, p, r): oracle_full(op, sig, p, r, Xh, Wh, dYh)
            for sig, p, r in cases for op in OPS}
    try:
        for tile, kernel in PERSISTENT:
            for splits in (1, 5):
                sbp.sbp_set_plan_override(tile[0], tile[1], splits, kernel, 1)
                for sig, p, r in cases:
                    for op in OPS:
                        say("persistent", tile, kernel, splits, sig, p, r, op)
                        out, st = run_gpu(op, sig, p, r, X, W, dY)
                        expect_state(op, sig, p, r, st)
                        w = want[(sig, op, p, r)]
                        if out.dtype == torch.bfloat16:
                            assert np.array_equal(out_bits(out), oracle.round_bf16(w)), \
                                (tile, kernel, splits, sig, op)
                        else:
                            assert np.array_equal(decode(out), w), (tile, kernel, splits, sig, op)
    finally:
        sbp.sbp_set_plan_override(0, 0, 1)


@pytest.mark.parametrize("tile,kernel", [((128, 128), 1), ((128, 128), 5), ((64, 64), 1),
                                         ((256, 128), 5)],
                         ids=["128x128-k1", "128x128-k5", "64x64-k1", "256x128-k5"])
def test_exact_grouped_backward_own_splits(tile, kernel):
    # one grouped launch whose two products use different reduction splits
    M, K, N = 304, 1104, 272
    X, W, dY = _int_inputs(M, K, N, 1400)
    Xh, Wh, dYh = (inputs.host_bits(t) for t in (X, W, dY))
    try:
        for sd, sw in ((1, 5), (3, 1), (2, 4)):
            sbp.sbp_set_plan_override(tile[0], tile[1], sd, kernel)
            sbp.sbp_set_bwd_override(2, sw)
            for sig in SIGS:
                say("grouped own splits", tile, kernel, sd, sw, sig)
                _check_exact_bwd(sig, 2, 1, X, W, dY, Xh, Wh, dYh)
    finally:
        sbp.sbp_set_plan_override(0, 0, 1)
