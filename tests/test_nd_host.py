"""Host-side checks of the nd-SBP part of the C ABI (no GPU needed).

* sbp_mesh_coords agrees with the oracle's own mesh-coordinate mapping
  (pinned there to the heterogeneous GPU mapping example of Sec. 4.2);
* sbp_nd_shard_index agrees with the oracle's nested split on random nd
  layouts, meshes of 1 to 4 axes;
* sbp_nd_signature agrees with the oracle's per-axis factor table for every
  combination of per-axis input states on 2-axis meshes, errors included;
* the nd compute calls validate their arguments before any HIP call (fake
  device addresses, skipped wherever a GPU is visible).
"""
import itertools

import numpy as np
import pytest

import oracle
from paper_2301_06813_amd import linear, sbp

STATES = {"S0": (sbp.SBP_SPLIT, 0), "S1": (sbp.SBP_SPLIT, 1), "B": (sbp.SBP_BROADCAST, -1),
          "P": (sbp.SBP_PARTIAL, -1)}
# the oracle numbers states the same way but defines them itself
ORC = {"S0": (oracle.SPLIT, 0), "S1": (oracle.SPLIT, 1), "B": (oracle.BCAST, -1),
       "P": (oracle.PARTIAL, -1)}


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="module")
def L():
    return sbp.lib()


def test_mesh_coords_match_oracle(L):
    for nodes, gpus in (([4], None), ([2, 3], None), ([2, 3, 4], None), ([1, 2], [2, 2]),
                        ([2, 1, 2], [1, 3, 2]), ([2, 2, 1, 2], [1, 2, 2, 1])):
        nn = int(np.prod(nodes))
        ng = 1 if gpus is None else int(np.prod(gpus))
        for node in range(nn):
            for gpu in range(ng):
                got = sbp.sbp_mesh_coords(nodes, gpus, node, gpu)
                assert got == oracle.mesh_coord(nodes, gpus, node, gpu)
    for bad in (([2, 2], None, 4, 0), ([2, 2], [1, 2], 0, 2), ([0, 2], None, 0, 0),
                ([2] * 5, None, 0, 0)):
        with pytest.raises(sbp.SbpError) as ei:
            sbp.sbp_mesh_coords(*bad)
        assert ei.value.code == sbp.SBP_ERR_LAYOUT


def test_nd_shard_index_matches_oracle(L):
    rng = np.random.default_rng(21)
    names = list(STATES)
    for _ in range(400):
        d = int(rng.integers(1, 5))
        mesh = [int(x) for x in rng.integers(1, 5, d)]
        st = [names[int(i)] for i in rng.integers(0, 4, d)]
        rows, cols = (int(x) for x in rng.integers(0, 40, 2))
        for c in itertools.islice(itertools.product(*(range(p) for p in mesh)), 12):
            s = sbp.sbp_nd_shard_index(sbp.nd_layout(st, mesh, c), rows, cols)
            want = oracle.nd_share([ORC[n] for n in st], mesh, c, rows, cols)
            assert (s.row_off, s.col_off, s.rows, s.cols) == want


def test_nd_one_axis_equals_1d(L):
    for p in (1, 3, 8):
        for r in range(p):
            for name, (k, a) in STATES.items():
                one = sbp.sbp_shard_index(sbp.sbp_layout_t(k, a, p, r), 29, 17)
                nd = sbp.sbp_nd_shard_index(sbp.nd_layout([name], [p], [r]), 29, 17)
                assert (one.row_off, one.col_off, one.rows, one.cols) == \
                       (nd.row_off, nd.col_off, nd.rows, nd.cols)


def test_nd_signature_matches_oracle(L):
    names = list(STATES)
    mesh, c = [2, 3], [1, 2]
    accepted = 0
    for xs in itertools.product(names, repeat=2):
        for ws in itertools.product(names, repeat=2):
            x, w = sbp.nd_layout(xs, mesh, c), sbp.nd_layout(ws, mesh, c)
            try:
                want = oracle.nd_tags([ORC[n] for n in xs], [ORC[n] for n in ws])
            except ValueError:
                want = None
            if want is None:
                with pytest.raises(sbp.SbpError) as ei:
                    sbp.sbp_nd_signature(x, w)
                assert ei.value.code == sbp.SBP_ERR_SIGNATURE
                continue
            accepted += 1
            got = sbp.sbp_nd_signature(x, w)
            for t, g in enumerate(got):
                assert g.states() == want[2 + t]
                assert list(g.p[:2]) == mesh and list(g.c[:2]) == c
    assert accepted == 36   # six 1-D signatures per axis


def test_nd_layout_errors(L):
    ok = sbp.nd_layout(["S0", "B"], [2, 2], [1, 0])
    w = sbp.nd_layout(["B", "S1"], [2, 2], [1, 0])
    sbp.sbp_nd_signature(ok, w)
    for bad in (sbp.nd_layout(["S0", "B"], [2, 2], [2, 0]),     # coordinate out of range
                sbp.nd_layout(["S0", "B"], [0, 2], [0, 0]),     # empty mesh axis
                sbp.nd_layout([(sbp.SBP_SPLIT, 2), "B"], [2, 2], [0, 0]),
                sbp.nd_layout([(sbp.SBP_BROADCAST, 0), "B"], [2, 2], [0, 0])):
        with pytest.raises(sbp.SbpError) as ei:
            sbp.sbp_nd_signature(bad, w)
        assert ei.value.code == sbp.SBP_ERR_LAYOUT
    bad = sbp.nd_layout(["S0", "B"], [2, 2], [1, 0])
    bad.ndim = 5
    with pytest.raises(sbp.SbpError) as ei:
        sbp.sbp_nd_shard_index(bad, 4, 4)
    assert ei.value.code == sbp.SBP_ERR_LAYOUT
    # layouts of one call must agree on the mesh and the coordinate
    for mesh, c in (([2, 2], [0, 0]), ([2, 4], [1, 0])):
        with pytest.raises(sbp.SbpError) as ei:
            sbp.sbp_nd_signature(ok, sbp.nd_layout(["B", "S1"], mesh, c))
        assert ei.value.code == sbp.SBP_ERR_LAYOUT


def test_3d_rule_states(L):
    Lz = linear.nd_layouts(("DP", "COL", "KS"), (2, 2, 2), (1, 0, 1))
    S0, S1, B, P = (STATES[n] for n in ("S0", "S1", "B", "P"))
    assert Lz["y"].states() == [S0, S1, P]
    assert Lz["dy"].states() == [S0, S1, B]
    assert Lz["dx"].states() == [S0, P, S1]
    assert Lz["dw"].states() == [P, S1, S0]


XA, WA, YA = 0x10000000, 0x20000000, 0x30000000
BF, F32 = sbp.SBP_BF16, sbp.SBP_F32


@pytest.mark.skipif(_gpu_visible(), reason="uses fake device addresses")
def test_nd_call_validation(L):
    # 3-D rule on a 2 x 2 x 2 mesh, device (1, 0, 1): X 64 x 32 -> share
    # rows [32, 64) x cols [16, 32); W 32 x 48 -> rows [16, 32) x cols [0, 24)
    mesh, c = (2, 2, 2), (1, 0, 1)
    lx, lw = linear.nd_input_layouts(("DP", "COL", "KS"), mesh, c)
    X = sbp.raw_view(XA, 64, 32, 32, BF)
    W = sbp.raw_view(WA, 32, 48, 48, BF)

    def call(y, x=X, w=W, llx=lx, llw=lw):
        with pytest.raises(sbp.SbpError) as ei:
            sbp.sbp_nd_linear_fwd(x, llx, w, llw, y, stream=0, ws=sbp.NO_WORKSPACE)
        return ei.value.code

    # Y is Partial-sum on mesh axis 2, so a bf16 output is refused
    assert call(sbp.raw_view(YA, 32, 24, 24, BF, sbp.SBP_LOCAL)) == sbp.SBP_ERR_DTYPE
    # wrong local output shape
    assert call(sbp.raw_view(YA, 32, 48, 48, F32, sbp.SBP_LOCAL)) == sbp.SBP_ERR_SHAPE
    # layouts disagree on the coordinate
    other = sbp.nd_layout(["B", "S1", "S0"], mesh, (0, 0, 1))
    assert call(sbp.raw_view(YA, 32, 24, 24, F32, sbp.SBP_LOCAL), llw=other) == sbp.SBP_ERR_LAYOUT
    # no signature on mesh axis 2: (S1, S1)
    bad_w = sbp.nd_layout(["B", "S1", "S1"], mesh, c)
    assert call(sbp.raw_view(YA, 32, 24, 24, F32, sbp.SBP_LOCAL), llw=bad_w) == \
        sbp.SBP_ERR_SIGNATURE
    # output overlapping the X share
    assert call(sbp.raw_view(XA + 32 * 32 * 2, 32, 24, 24, F32, sbp.SBP_LOCAL)) == \
        sbp.SBP_ERR_ALIAS
    # backward: three states of different signatures
    ldy = sbp.nd_layout(["S0", "S1", "S0"], mesh, c)
    dY = sbp.raw_view(YA, 64, 48, 48, BF)
    with pytest.raises(sbp.SbpError) as ei:
        sbp.sbp_nd_linear_bwd(dY, ldy, X, lx, W, lw, sbp.raw_view(0x40000000, 32, 16, 16, BF, 1),
                              sbp.raw_view(0x50000000, 16, 24, 24, F32, 1), stream=0,
                              ws=sbp.NO_WORKSPACE)
    assert ei.value.code == sbp.SBP_ERR_SIGNATURE
