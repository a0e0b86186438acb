"""Host-side checks of the C ABI (no GPU needed).

* libsbp.so loads and exports every function include/sbp.h declares;
* sbp_shard_index agrees bit for bit with the oracle's own split and with
  numpy.array_split (AutoDDL Sec. 4.1 states; balanced-split reading);
* sbp_signature agrees with the oracle's independent state table, and every
  other pair of input states is rejected (Sec. 4.2 rule, Sec. 4.3 gradients);
* every validation error is returned before any HIP call. Each case below
  has exactly one defect, so no call here ever reaches a kernel launch; the
  fake device addresses are never dereferenced, and the module is skipped
  wherever a GPU is visible.
"""
import os
import re

import numpy as np
import pytest

import oracle
from paper_2301_06813_amd import sbp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


# These tests pass fake device addresses that must never reach a kernel. They
# check host logic only, so they run where no GPU is visible; on a GPU machine a
# mistaken case could launch a kernel on those addresses.
pytestmark = pytest.mark.skipif(_gpu_visible(), reason="host-only ABI tests use fake device "
                                "addresses; run them where no GPU is visible")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(sbp.LIB_PATH):
        from paper_2301_06813_amd import build
        build.build(verbose=False)
    return sbp.lib()


def test_exports_every_declared_symbol(L):
    hdr = open(os.path.join(ROOT, "include", "sbp.h")).read()
    declared = set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(sbp_\w+)\s*\(", hdr, re.M))
    assert declared, "no declarations parsed"
    assert declared == set(sbp.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def test_shard_index_matches_oracle_and_numpy(L, orc):
    for D in range(0, 30):
        for p in range(1, 10):
            chunks = np.array_split(np.arange(D), p)
            for r in range(p):
                off, ln = orc.split(D, p, r)
                s0 = sbp.sbp_shard_index(sbp.split(0, p, r), D, 7)
                s1 = sbp.sbp_shard_index(sbp.split(1, p, r), 5, D)
                assert (s0.row_off, s0.rows, s0.col_off, s0.cols) == (off, ln, 0, 7)
                assert (s1.col_off, s1.cols, s1.row_off, s1.rows) == (off, ln, 0, 5)
                assert ln == len(chunks[r])
                for lay in (sbp.broadcast(p, r), sbp.partial(p, r)):
                    s = sbp.sbp_shard_index(lay, D, 3)
                    assert (s.row_off, s.col_off, s.rows, s.cols) == (0, 0, D, 3)


def test_shard_index_fc8_offsets(L):
    # VGG FC8 column shards of a 4096 x 1000 weight over 8 devices: 125 columns
    # each, starting at 125 r (the odd byte offsets the kernel must handle).
    for r in range(8):
        s = sbp.sbp_shard_index(sbp.split(1, 8, r), 4096, 1000)
        assert (s.row_off, s.col_off, s.rows, s.cols) == (0, 125 * r, 4096, 125)


def _lay(kind, axis, p=4, r=1):
    return sbp.sbp_layout_t(kind, axis, p, r)


ALL_STATES = [(sbp.SBP_SPLIT, 0), (sbp.SBP_SPLIT, 1), (sbp.SBP_BROADCAST, -1),
              (sbp.SBP_PARTIAL, -1)]
ORC_KIND = {sbp.SBP_SPLIT: oracle.SPLIT, sbp.SBP_BROADCAST: oracle.BCAST,
            sbp.SBP_PARTIAL: oracle.PARTIAL}


def test_signature_table_matches_oracle(L, orc):
    expected = {}
    for sig in (oracle.DP, oracle.COL, oracle.KS, oracle.PB, oracle.BP, oracle.BB):
        t = orc.tags(sig)
        expected[(t[0], t[1])] = t[2:]
    for xs in ALL_STATES:
        for ws in ALL_STATES:
            x, w = _lay(*xs), _lay(*ws)
            key = ((ORC_KIND[xs[0]], xs[1]), (ORC_KIND[ws[0]], ws[1]))
            if key in expected:
                got = sbp.sbp_signature(x, w)
                for g, e in zip(got, expected[key]):
                    assert (ORC_KIND[g.kind], g.axis) == e
                    assert (g.p, g.r) == (4, 1)
            else:
                with pytest.raises(sbp.SbpError) as ei:
                    sbp.sbp_signature(x, w)
                assert ei.value.code == sbp.SBP_ERR_SIGNATURE


def test_layout_errors(L):
    bad = [sbp.sbp_layout_t(sbp.SBP_SPLIT, 0, 0, 0), sbp.sbp_layout_t(sbp.SBP_SPLIT, 0, 4, 4),
           sbp.sbp_layout_t(sbp.SBP_SPLIT, 0, 4, -1), sbp.sbp_layout_t(sbp.SBP_SPLIT, 2, 4, 0),
           sbp.sbp_layout_t(sbp.SBP_BROADCAST, 0, 4, 0), sbp.sbp_layout_t(7, -1, 4, 0)]
    for l in bad:
        with pytest.raises(sbp.SbpError) as ei:
            sbp.sbp_shard_index(l, 8, 8)
        assert ei.value.code == sbp.SBP_ERR_LAYOUT
    # layouts of one call must agree on p and r
    with pytest.raises(sbp.SbpError) as ei:
        sbp.sbp_signature(sbp.split(0, 4, 1), sbp.broadcast(4, 2))
    assert ei.value.code == sbp.SBP_ERR_LAYOUT
    with pytest.raises(sbp.SbpError) as ei:
        sbp.sbp_shard_index(sbp.split(0, 2, 0), -1, 3)
    assert ei.value.code == sbp.SBP_ERR_SHAPE


# Fake, never-dereferenced device addresses in disjoint ranges.
XA, WA, YA = 0x10000000, 0x20000000, 0x30000000
BF, F32 = sbp.SBP_BF16, sbp.SBP_F32


def _fwd_case(**kw):
    """A forward DP call (p=4, r=1, M=64, K=32, N=48) with one field changed."""
    c = dict(x=sbp.raw_view(XA, 64, 32, 32, BF), lx=sbp.split(0, 4, 1),
             w=sbp.raw_view(WA, 32, 48, 48, BF), lw=sbp.broadcast(4, 1),
             y=sbp.raw_view(YA, 16, 48, 48, BF, sbp.SBP_LOCAL))
    c.update(kw)
    return c


def _code(c, fn="sbp_linear_fwd"):
    import ctypes
    lo = sbp.sbp_layout_t()
    args = [c["x"], c["lx"], c["w"], c["lw"], c["y"]]
    return getattr(sbp.lib(), fn)(*(ctypes.byref(a) if a is not None else None for a in args),
                                  ctypes.byref(lo), None, None)


ERR_CASES = [
    ("null X", dict(x=None), sbp.SBP_ERR_NULL),
    ("null layout", dict(lw=None), sbp.SBP_ERR_NULL),
    ("null data", dict(x=sbp.raw_view(None, 64, 32, 32, BF)), sbp.SBP_ERR_NULL),
    ("r >= p", dict(lx=sbp.split(0, 4, 4)), sbp.SBP_ERR_LAYOUT),
    ("p mismatch", dict(lw=sbp.broadcast(8, 1)), sbp.SBP_ERR_LAYOUT),
    ("r mismatch", dict(lw=sbp.broadcast(4, 2)), sbp.SBP_ERR_LAYOUT),
    ("bad signature (P,S0)", dict(lx=sbp.partial(4, 1), lw=sbp.split(0, 4, 1)),
     sbp.SBP_ERR_SIGNATURE),
    ("bad signature (S0,S0)", dict(lw=sbp.split(0, 4, 1)), sbp.SBP_ERR_SIGNATURE),
    ("accumulate into bf16", dict(y=sbp.raw_view(YA, 16, 48, 48, BF, sbp.SBP_ACCUMULATE)),
     sbp.SBP_ERR_DTYPE),
    ("partial input, split weight", dict(lx=sbp.partial(4, 1), lw=sbp.split(1, 4, 1)),
     sbp.SBP_ERR_SIGNATURE),
    # (P, B) -> P resolves, so a bf16 output of the right shape is refused
    ("partial input, bf16 output", dict(lx=sbp.partial(4, 1),
                                        y=sbp.raw_view(YA, 64, 48, 48, BF, sbp.SBP_LOCAL)),
     sbp.SBP_ERR_DTYPE),
    ("inner dims", dict(w=sbp.raw_view(WA, 33, 48, 48, BF)), sbp.SBP_ERR_SHAPE),
    ("ld < cols", dict(x=sbp.raw_view(XA, 64, 32, 31, BF)), sbp.SBP_ERR_SHAPE),
    ("negative rows", dict(x=sbp.raw_view(XA, -1, 32, 32, BF)), sbp.SBP_ERR_SHAPE),
    ("huge cols", dict(w=sbp.raw_view(WA, 32, 1 << 31, 1 << 31, BF)), sbp.SBP_ERR_SHAPE),
    ("bad scope", dict(x=sbp.raw_view(XA, 64, 32, 32, BF, 5)), sbp.SBP_ERR_SHAPE),
    ("wrong output rows", dict(y=sbp.raw_view(YA, 64, 48, 48, BF)), sbp.SBP_ERR_SHAPE),
    ("wrong output cols", dict(y=sbp.raw_view(YA, 16, 47, 48, BF)), sbp.SBP_ERR_SHAPE),
    ("output ld < cols", dict(y=sbp.raw_view(YA, 16, 48, 40, BF)), sbp.SBP_ERR_SHAPE),
    ("mixed input dtype", dict(w=sbp.raw_view(WA, 32, 48, 48, F32)), sbp.SBP_ERR_DTYPE),
    ("unknown dtype", dict(x=sbp.raw_view(XA, 64, 32, 32, 9)), sbp.SBP_ERR_DTYPE),
    ("fp32 in, bf16 out", dict(x=sbp.raw_view(XA, 64, 32, 32, F32),
                               w=sbp.raw_view(WA, 32, 48, 48, F32)), sbp.SBP_ERR_DTYPE),
    ("misaligned bf16", dict(x=sbp.raw_view(XA + 1, 64, 32, 32, BF)), sbp.SBP_ERR_ALIGN),
    ("misaligned f32 out", dict(y=sbp.raw_view(YA + 2, 16, 48, 48, F32)), sbp.SBP_ERR_ALIGN),
    ("output overlaps X share", dict(y=sbp.raw_view(XA + 16 * 32 * 2 + 64, 16, 48, 48, BF)),
     sbp.SBP_ERR_ALIAS),
    ("output overlaps W", dict(y=sbp.raw_view(WA + 100, 16, 48, 48, BF)), sbp.SBP_ERR_ALIAS),
]


@pytest.mark.parametrize("name,change,code", ERR_CASES, ids=[c[0] for c in ERR_CASES])
def test_forward_validation_errors(L, name, change, code):
    assert _code(_fwd_case(**change)) == code


WS_ERR_CASES = [
    ("negative size", sbp.sbp_workspace_t(0x60000000, -16), sbp.SBP_ERR_SHAPE),
    ("null data", sbp.sbp_workspace_t(None, 4096), sbp.SBP_ERR_NULL),
    ("misaligned", sbp.sbp_workspace_t(0x60000008, 4096), sbp.SBP_ERR_ALIGN),
    ("overlaps X", sbp.sbp_workspace_t(XA + 1024, 4096), sbp.SBP_ERR_ALIAS),
    ("overlaps W", sbp.sbp_workspace_t(WA - 1024, 4096), sbp.SBP_ERR_ALIAS),
    ("overlaps Y", sbp.sbp_workspace_t(YA, 16), sbp.SBP_ERR_ALIAS),
]


@pytest.mark.parametrize("name,ws,code", WS_ERR_CASES, ids=[c[0] for c in WS_ERR_CASES])
def test_workspace_validation(L, name, ws, code):
    """The caller's workspace is checked on the host before any HIP call:
    size, pointer, 16-byte alignment, and no overlap with the call's
    operands or output."""
    import ctypes
    c = _fwd_case()
    lo = sbp.sbp_layout_t()
    args = [c["x"], c["lx"], c["w"], c["lw"], c["y"]]
    rc = L.sbp_linear_fwd(*(ctypes.byref(a) for a in args), ctypes.byref(lo), ctypes.byref(ws),
                          None)
    assert rc == code
    # the two-product call checks it against both products
    dy = sbp.raw_view(YA, 64, 48, 48, BF)
    dx = sbp.raw_view(0x40000000, 16, 32, 32, BF, sbp.SBP_LOCAL)
    dw = sbp.raw_view(0x50000000, 32, 48, 48, F32, sbp.SBP_LOCAL)
    if name == "overlaps Y":
        ws = sbp.sbp_workspace_t(0x50000000 + 64, 16)   # inside dW
    rc = L.sbp_linear_bwd(ctypes.byref(dy), ctypes.byref(sbp.split(0, 4, 1)), ctypes.byref(c["x"]),
                          ctypes.byref(c["lx"]), ctypes.byref(c["w"]), ctypes.byref(c["lw"]),
                          ctypes.byref(dx), ctypes.byref(lo), ctypes.byref(dw), ctypes.byref(lo),
                          ctypes.byref(ws), None)
    assert rc == code, (name, rc)


def test_partial_output_must_be_fp32(L):
    # K-split forward: X S(1), W S(0) -> P; a bf16 output is rejected.
    c = dict(x=sbp.raw_view(XA, 64, 32, 32, BF), lx=sbp.split(1, 4, 1),
             w=sbp.raw_view(WA, 32, 48, 48, BF), lw=sbp.split(0, 4, 1),
             y=sbp.raw_view(YA, 64, 48, 48, BF, sbp.SBP_LOCAL))
    assert _code(c) == sbp.SBP_ERR_DTYPE


def test_global_inner_dims_checked(L):
    # K-split with global X of 33 columns and global W of 32 rows: the local
    # shares both have 8 reduction elements, but the globals disagree.
    c = dict(x=sbp.raw_view(XA, 64, 33, 33, BF), lx=sbp.split(1, 4, 1),
             w=sbp.raw_view(WA, 32, 48, 48, BF), lw=sbp.split(0, 4, 1),
             y=sbp.raw_view(YA, 64, 48, 48, F32, sbp.SBP_LOCAL))
    assert _code(c) == sbp.SBP_ERR_SHAPE


def test_backward_signature_errors(L):
    import ctypes
    lo = sbp.sbp_layout_t()
    dy = sbp.raw_view(XA, 64, 48, 48, BF)
    w = sbp.raw_view(WA, 32, 48, 48, BF)
    dx = sbp.raw_view(YA, 16, 32, 32, BF, sbp.SBP_LOCAL)
    # bwd_data: (dY P, W S(0)) is no signature (dY is P only under BB, with W B)
    rc = sbp.lib().sbp_linear_bwd_data(ctypes.byref(dy), ctypes.byref(sbp.partial(4, 1)),
                                       ctypes.byref(w), ctypes.byref(sbp.split(0, 4, 1)),
                                       ctypes.byref(dx), ctypes.byref(lo), None, None)
    assert rc == sbp.SBP_ERR_SIGNATURE
    # bwd_weight: (X S(0), dY B) is no signature
    x = sbp.raw_view(XA, 64, 32, 32, BF)
    dw = sbp.raw_view(YA, 32, 48, 48, F32, sbp.SBP_LOCAL)
    rc = sbp.lib().sbp_linear_bwd_weight(ctypes.byref(x), ctypes.byref(sbp.split(0, 4, 1)),
                                         ctypes.byref(dy), ctypes.byref(sbp.broadcast(4, 1)),
                                         ctypes.byref(dw), ctypes.byref(lo), None, None)
    assert rc == sbp.SBP_ERR_SIGNATURE
    # bwd_weight DP: the dW output is Partial-sum, so a bf16 dW is rejected
    dyl = sbp.raw_view(XA + (1 << 20), 64, 48, 48, BF)
    dwb = sbp.raw_view(YA, 32, 48, 48, BF, sbp.SBP_LOCAL)
    rc = sbp.lib().sbp_linear_bwd_weight(ctypes.byref(x), ctypes.byref(sbp.split(0, 4, 1)),
                                         ctypes.byref(dyl), ctypes.byref(sbp.split(0, 4, 1)),
                                         ctypes.byref(dwb), ctypes.byref(lo), None, None)
    assert rc == sbp.SBP_ERR_DTYPE


def test_empty_output_is_a_noop(L):
    # M = 3 rows over p = 4: rank 3 holds no rows, so the DP forward has an
    # empty output and returns success without touching the device.
    c = dict(x=sbp.raw_view(XA, 3, 32, 32, BF), lx=sbp.split(0, 4, 3),
             w=sbp.raw_view(WA, 32, 48, 48, BF), lw=sbp.broadcast(4, 3),
             y=sbp.raw_view(None, 0, 48, 48, BF, sbp.SBP_LOCAL))
    assert _code(c) == sbp.SBP_OK


def test_strerror_and_plan(L):
    for code in range(-8, 1):
        assert sbp.sbp_strerror(code) and "unknown" not in sbp.sbp_strerror(code)
    assert "unknown" in sbp.sbp_strerror(-99)
    tm, tn, s, kn = sbp.sbp_plan(2, 1024, 384, 8192, sbp.SBP_BF16, sbp.SBP_BF16)
    assert (tm, tn) in {(256, 256), (256, 128), (128, 256), (128, 128), (128, 64), (64, 128),
                        (64, 64)}
    assert s >= 1 and kn in (1, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13)   # pipelined bf16 instances
    # a reduction that is not a multiple of 8 cannot use the pipelined kernel
    assert sbp.sbp_plan(0, 256, 256, 125, BF, BF)[3] == sbp.KERNEL_GENERIC
    assert sbp.sbp_plan(0, 64, 64, 64, F32, F32)[3] == sbp.KERNEL_F32
    with pytest.raises(sbp.SbpError):
        sbp.sbp_set_plan_override(96, 96, 1)
    with pytest.raises(sbp.SbpError):
        sbp.sbp_set_plan_override(64, 64, 1, 8)
    sbp.sbp_set_plan_override(64, 64, 3)
    assert sbp.sbp_plan(0, 128, 128, 1024, BF, BF) == (64, 64, 3, sbp.KERNEL_PIPELINED)
    sbp.sbp_set_plan_override(256, 256, 2, sbp.KERNEL_GENERIC)
    assert sbp.sbp_plan(0, 128, 128, 1024, BF, BF) == (256, 128, 2, sbp.KERNEL_GENERIC)
    sbp.sbp_set_plan_override(256, 256, 2, sbp.KERNEL_PIPELINED)
    assert sbp.sbp_plan(0, 128, 128, 1024, BF, BF) == (256, 256, 2, sbp.KERNEL_PIPELINED)
    with pytest.raises(sbp.SbpError):
        sbp.sbp_set_plan_override(512, 256, 1)
    # the two-stage instances exist for tiles up to 128x128 only
    with pytest.raises(sbp.SbpError):
        sbp.sbp_set_plan_override(256, 128, 1, sbp.KERNEL_PIPELINED_2STAGE)
    with pytest.raises(sbp.SbpError):
        sbp.sbp_set_plan_override(128, 128, 1, sbp.KERNEL_F32)
    sbp.sbp_set_plan_override(128, 128, 3, sbp.KERNEL_PIPELINED_2STAGE)
    assert sbp.sbp_plan(0, 512, 512, 1024, BF, BF) == (128, 128, 3,
                                                       sbp.KERNEL_PIPELINED_2STAGE)
    # operands the pipelined kernel cannot read fall back to the generic kernel
    assert sbp.sbp_plan(0, 512, 512, 1001, BF, BF)[3] == sbp.KERNEL_GENERIC
    # every listed (tile, instance) pair is accepted and reported back
    for tile, code in (((128, 128), 5), ((256, 128), 5), ((128, 256), 5), ((256, 256), 6),
                       ((128, 128), 6), ((128, 128), 7), ((256, 128), 7), ((128, 256), 7),
                       ((256, 256), 8), ((256, 128), 9), ((128, 256), 9), ((128, 128), 9),
                       ((128, 128), 10), ((128, 64), 11), ((64, 128), 11), ((64, 64), 11),
                       ((128, 64), 5), ((64, 128), 5), ((64, 64), 5), ((128, 64), 7),
                       ((64, 128), 7), ((64, 64), 7), ((128, 128), 12), ((128, 64), 12),
                       ((64, 128), 12), ((64, 64), 12), ((128, 128), 13), ((128, 64), 13),
                       ((64, 128), 13), ((64, 64), 13)):
        sbp.sbp_set_plan_override(tile[0], tile[1], 2, code, 1)
        assert sbp.sbp_plan(0, 2048, 2048, 1024, BF, BF) == (tile[0], tile[1], 2, code)
    for tile, code in (((64, 64), 6), ((256, 256), 5), ((64, 128), 9), ((256, 128), 10),
                       ((128, 128), 3), ((128, 128), 11), ((256, 128), 12),
                       ((256, 256), 13), ((64, 64), 14)):
        with pytest.raises(sbp.SbpError):
            sbp.sbp_set_plan_override(tile[0], tile[1], 1, code)
    with pytest.raises(sbp.SbpError):
        sbp.sbp_set_plan_override(128, 128, 1, 1, 9)     # at most 8 workgroups per CU
    with pytest.raises(sbp.SbpError):
        sbp.sbp_set_plan_override(128, 128, 0, 1)        # splits >= 1
    sbp.sbp_set_plan_override(0, 0, 1)
    # backward override: modes 0..2, splits_w >= 1
    for mode in (0, 1, 2):
        sbp.sbp_set_bwd_override(mode, 3)
    for mode, sw in ((3, 1), (-1, 1), (2, 0)):
        with pytest.raises(sbp.SbpError):
            sbp.sbp_set_bwd_override(mode, sw)
    sbp.sbp_set_bwd_override(0, 1)


def _bwd_code(dy, ldy, x, lx, w, lw, dx, dw):
    import ctypes
    a, b = sbp.sbp_layout_t(), sbp.sbp_layout_t()
    return sbp.lib().sbp_linear_bwd(ctypes.byref(dy), ctypes.byref(ldy), ctypes.byref(x),
                                    ctypes.byref(lx), ctypes.byref(w), ctypes.byref(lw),
                                    ctypes.byref(dx), ctypes.byref(a), ctypes.byref(dw),
                                    ctypes.byref(b), None, None)


def test_grouped_backward_validation(L):
    # DP, p=4, r=1: X 64x32 (S0), W 32x48 (B), dY 64x48 (S0); dX 16x32 bf16, dW 32x48 fp32
    x = sbp.raw_view(XA, 64, 32, 32, BF)
    w = sbp.raw_view(WA, 32, 48, 48, BF)
    dy = sbp.raw_view(YA, 64, 48, 48, BF)
    dx = sbp.raw_view(0x40000000, 16, 32, 32, BF, sbp.SBP_LOCAL)
    dw = sbp.raw_view(0x50000000, 32, 48, 48, F32, sbp.SBP_LOCAL)
    s0, b = sbp.split(0, 4, 1), sbp.broadcast(4, 1)
    # dY given as B does not match the DP signature of (X, W)
    assert _bwd_code(dy, b, x, s0, w, b, dx, dw) == sbp.SBP_ERR_SIGNATURE
    # dX and dW overlapping
    dw_ov = sbp.raw_view(0x40000000 + 64, 32, 48, 48, F32, sbp.SBP_LOCAL)
    assert _bwd_code(dy, s0, x, s0, w, b, dx, dw_ov) == sbp.SBP_ERR_ALIAS
    # dX written over rank 1's share of X (rows 16..31), the input only the
    # weight product reads
    dx_ov = sbp.raw_view(XA + 16 * 32 * 2 + 64, 16, 32, 32, BF, sbp.SBP_LOCAL)
    assert _bwd_code(dy, s0, x, s0, w, b, dx_ov, dw) == sbp.SBP_ERR_ALIAS
    # P dW must be fp32
    dw_bf = sbp.raw_view(0x50000000, 32, 48, 48, BF, sbp.SBP_LOCAL)
    assert _bwd_code(dy, s0, x, s0, w, b, dx, dw_bf) == sbp.SBP_ERR_DTYPE
    # an empty rank (M = 3 rows over p = 4, r = 3) succeeds without launching
    x3 = sbp.raw_view(XA, 3, 32, 32, BF)
    dy3 = sbp.raw_view(YA, 3, 48, 48, BF)
    dx0 = sbp.raw_view(None, 0, 32, 32, BF, sbp.SBP_LOCAL)
    dw3 = sbp.raw_view(0x50000000, 32, 48, 48, F32, sbp.SBP_LOCAL)
    s3, b3 = sbp.split(0, 4, 3), sbp.broadcast(4, 3)
    # dW of an empty share is an all-zero output: a launch is needed, so only
    # check the empty dX path through the data product alone
    import ctypes
    lo = sbp.sbp_layout_t()
    assert sbp.lib().sbp_linear_bwd_data(ctypes.byref(dy3), ctypes.byref(s3), ctypes.byref(w),
                                         ctypes.byref(b3), ctypes.byref(dx0), ctypes.byref(lo),
                                         None, None) == sbp.SBP_OK


def test_plan_bwd(L):
    g, tm, tn, sd, sw = sbp.sbp_plan_bwd(1024, 1024, 3072, BF, 1024, 3072, 1024, F32)
    assert g in (0, 1) and sd >= 1 and sw >= 1
    assert (tm, tn) in {(256, 256), (256, 128), (128, 256), (128, 128), (128, 64), (64, 128),
                        (64, 64)}


def _table_rows(name):
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "paper_2301_06813_amd", "csrc", name)
    rows = []
    for line in open(path):
        m = re.match(r"\{([^}]*)\}", line.strip())
        if m:
            rows.append([int(x) for x in m.group(1).split(",")])
    return rows


def test_tuned_tables_name_built_instances(L):
    # every tuned plan names a (tile, kernel) pair the library has, and the
    # library then reports that plan back for the product
    singles = _table_rows("tuned_plans.inc")
    pairs = _table_rows("tuned_bwd_plans.inc")
    assert len(singles) > 50 and len(pairs) > 15
    try:
        from paper_2301_06813_amd.tune import SHIFT_CODES
        for orient, f32, m, n, k, dma, bm, bn, code, splits, occ, *nb in singles:
            sbp.sbp_set_plan_override(bm, bn, 1, code)     # raises for an unknown pair
            assert splits >= 1 and 0 <= occ <= 8 and dma in (0, 1, 2)
            sbp.sbp_set_plan_override(0, 0, 1)
            if dma == 2:   # shifted-form products: an instance that has that form
                assert ((bm, bn), code) in SHIFT_CODES, (orient, m, n, k, bm, bn, code)
            if dma == 1 and not nb:
                out = F32 if f32 else BF
                tm, tn, s, kn = sbp.sbp_plan(orient, m, n, k, BF, out)
                assert (tm, tn, s, kn) == (bm, bn, splits, code), (orient, m, n, k)
        for md, nd, kd, fd, mw, nw, kw, fw, bm, bn, code, sd, sw in pairs:
            sbp.sbp_set_plan_override(bm, bn, sd, code)
            sbp.sbp_set_plan_override(0, 0, 1)
            if kd % 8 or mw % 8 or nw % 8:
                continue   # not plannable with tight leading dimensions
            g, tm, tn, psd, psw = sbp.sbp_plan_bwd(md, nd, kd, F32 if fd else BF,
                                                     mw, nw, kw, F32 if fw else BF)
            assert (g, tm, tn, psd, psw) == (1, bm, bn, sd, sw), (md, nd, kd)
    finally:
        sbp.sbp_set_plan_override(0, 0, 1)
