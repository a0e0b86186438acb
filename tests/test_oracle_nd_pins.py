"""Pins for the oracle's nd-SBP functions (device meshes with one SBP state
per mesh axis), against things other than the oracle itself:

* Listing 1 (Sec. 4.1): a 6 x 4 tensor in [S(1), S(0), B] on a 2 x 3 x 4
  mesh leaves a 2 x 2 block on every device, each block on 4 devices, and
  the blocks tile the tensor (tests/golden/listing1_shards.json);
* the heterogeneous GPU mapping example of Sec. 4.2
  (tests/golden/hetero_mapping.json);
* nested splits against numpy.array_split applied twice, and against one
  split over p1*p2 when it divides the extent;
* the 3-D rule of Sec. 4.2 (its printed output state (S0, S1, P));
* the mesh reassembly invariant: over all devices of the mesh, output
  blocks placed at their shares, summed over Partial-sum axes, with
  Broadcast copies equal, give the exact global product of integer inputs;
* a 1-axis mesh, or a mesh whose other axes have one device, reduces to the
  1-D oracle;
* planted mistakes in copies of oracle.c are caught by these checks.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
S0, S1, B, P = (oracle.SPLIT, 0), (oracle.SPLIT, 1), (oracle.BCAST, -1), (oracle.PARTIAL, -1)
NAMES = {"S0": S0, "S1": S1, "B": B, "P": P}
# per-axis states of X and W for each factor (the oracle's 1-D table)
FACTOR = {"DP": (S0, B), "COL": (B, S1), "KS": (S1, S0), "PB": (P, B), "BP": (B, P),
          "BB": (B, B)}
OPS = (oracle.FWD, oracle.BWD_DATA, oracle.BWD_WEIGHT)


def _global(op, X, W, dY):
    if op == oracle.FWD:
        return X @ W
    if op == oracle.BWD_DATA:
        return dY @ W.T
    return X.T @ dY


def coords(mesh):
    return list(itertools.product(*(range(p) for p in mesh)))


def partial_inputs(rng, T, states, mesh):
    """Per device coordinate, the tensor a device holds of the integer tensor
    T in per-axis states `states`: on the Partial-sum axes, integer parts
    that sum to T over those axes' coordinates (the full T elsewhere)."""
    pax = [a for a, st in enumerate(states) if st == P]
    combos = list(itertools.product(*(range(mesh[a]) for a in pax)))
    parts = [rng.integers(-3, 4, T.shape) for _ in combos[:-1]]
    parts.append(T - sum(parts, np.zeros_like(T)))
    by = dict(zip(combos, parts))
    return lambda c: by[tuple(c[a] for a in pax)].astype(np.float32)


def nd_reassemble(orc, op, factors, mesh, Xi, Wi, dYi, M, K, N, rng=None):
    """All devices' outputs of op combined by the output's per-axis states.
    Inputs in a Partial-sum state get per-device integer parts of the given
    integer tensors. Raises AssertionError when Broadcast copies differ or
    blocks do not tile."""
    rng = np.random.default_rng(1) if rng is None else rng
    xs = [FACTOR[f][0] for f in factors]
    ws = [FACTOR[f][1] for f in factors]
    t = orc.nd_tags(xs, ws)
    xin, win, dyin = (partial_inputs(rng, T, st, mesh) for T, st in
                      ((Xi, t[0]), (Wi, t[1]), (dYi, t[3])))
    grow, gcol = {oracle.FWD: (M, N), oracle.BWD_DATA: (M, K), oracle.BWD_WEIGHT: (K, N)}[op]
    total = np.zeros((grow, gcol))
    cover = np.zeros((grow, gcol), dtype=np.int64)
    first = {}
    for c in coords(mesh):
        part = orc.nd_linear(op, xin(c), win(c), dyin(c), xs, ws, mesh, c)
        rows, cols, st = orc.nd_out_shape(op, M, K, N, xs, ws, mesh, c)
        assert part.shape == (rows, cols)
        r0, c0, nr, nc = orc.nd_share(st, mesh, c, grow, gcol)
        assert (nr, nc) == (rows, cols)
        # a device whose coordinate on some Broadcast axis is not 0 holds a
        # copy: it must equal the copy at coordinate 0 on those axes
        base = tuple(0 if st[a] == B else c[a] for a in range(len(mesh)))
        if base != c:
            assert np.array_equal(part, first[base])
            continue
        first[c] = part
        total[r0:r0 + nr, c0:c0 + nc] += part
        if all(st[a] != P or c[a] == 0 for a in range(len(mesh))):
            cover[r0:r0 + nr, c0:c0 + nc] += 1
    assert np.all(cover == 1), "output blocks do not tile the global tensor"
    return total


CASES = [
    ((2, 2, 2), ("DP", "COL", "KS")),
    ((2, 2, 2), ("KS", "DP", "COL")),
    ((3, 2), ("KS", "COL")),
    ((2, 3), ("DP", "DP")),
    ((2, 2), ("KS", "KS")),
    ((3, 2), ("COL", "COL")),
    ((2, 3), ("COL", "BB")),
    ((1, 3, 2), ("BB", "DP", "KS")),
    ((2, 1, 2, 2), ("DP", "BB", "COL", "KS")),
    ((2, 3), ("PB", "COL")),
    ((3, 2), ("DP", "BP")),
    ((2, 2, 2), ("PB", "BP", "BB")),
]
SHAPES = [(13, 11, 7), (8, 12, 6)]


def nd_invariant_failures(orc, cases=CASES):
    bad = []
    rng = np.random.default_rng(17)
    for (M, K, N) in SHAPES:
        Xi, Wi, dYi = (rng.integers(-3, 4, s) for s in ((M, K), (K, N), (M, N)))
        for mesh, factors in cases:
            for op in OPS:
                try:
                    got = nd_reassemble(orc, op, factors, mesh, Xi, Wi, dYi, M, K, N, rng)
                    ok = np.array_equal(got, _global(op, Xi, Wi, dYi))
                except (AssertionError, ValueError):
                    ok = False
                if not ok:
                    bad.append((mesh, factors, op, (M, K, N)))
    return bad


def test_nd_reassembly_invariant(orc):
    assert nd_invariant_failures(orc) == []


def test_listing1_blocks(orc):
    with open(os.path.join(GOLDEN, "listing1_shards.json")) as f:
        g = json.load(f)
    rows, cols = g["tensor_shape"]
    states = [NAMES[s.replace("(", "").replace(")", "")] for s in
              (f_["state"] for f_ in g["factors"])]
    mesh = [f_["p"] for f_ in g["factors"]]
    blocks = {}
    for c in coords(mesh):
        r0, c0, nr, nc = orc.nd_share(states, mesh, c, rows, cols)
        assert [nr, nc] == g["composed_local_shape"]
        blocks.setdefault((r0, c0), []).append(c)
    # every block is held by copies_per_block devices, which differ only on
    # the Broadcast mesh axis
    for held in blocks.values():
        assert len(held) == g["copies_per_block"]
        assert len({c[:2] for c in held}) == 1
    cover = np.zeros((rows, cols), dtype=int)
    for (r0, c0) in blocks:
        cover[r0:r0 + 2, c0:c0 + 2] += 1
    assert np.all(cover == 1)


def test_hetero_mapping_golden(orc):
    with open(os.path.join(GOLDEN, "hetero_mapping.json")) as f:
        g = json.load(f)
    mesh = [n * q for n, q in zip(g["nodes"], g["gpus"])]
    states = [NAMES[s] for s in g["states"]]
    for split, gpus in enumerate(g["split_gpus"]):
        for node, gpu in gpus:
            c = orc.mesh_coord(g["nodes"], g["gpus"], node, gpu)
            assert c[0] == split
            # the device holds rows split `split` of a tensor split on mesh axis 0
            r0, _, nr, _ = orc.nd_share(states, mesh, c, 2 * mesh[0], 3)
            assert (r0, nr) == (2 * split, 2)
    # the two lists name every GPU of the 2 x 4 system once
    allg = sorted(tuple(x) for s in g["split_gpus"] for x in s)
    assert allg == [(n, q) for n in range(2) for q in range(4)]


def test_mesh_coord_is_a_bijection(orc):
    for nodes, gpus in (([2, 3], [1, 1]), ([1, 2], [2, 2]), ([2, 1, 2], [1, 3, 2])):
        seen = set()
        nn, ng = int(np.prod(nodes)), int(np.prod(gpus))
        for node in range(nn):
            for gpu in range(ng):
                c = tuple(orc.mesh_coord(nodes, gpus, node, gpu))
                assert all(0 <= c[a] < nodes[a] * gpus[a] for a in range(len(c)))
                seen.add(c)
        assert len(seen) == nn * ng
    with pytest.raises(ValueError):
        orc.mesh_coord([2, 2], None, 4, 0)


def test_nested_split_matches_numpy(orc):
    for D in range(0, 30):
        for p1 in range(1, 5):
            for p2 in range(1, 5):
                for c1 in range(p1):
                    outer = np.array_split(np.arange(D), p1)[c1]
                    for c2 in range(p2):
                        want = np.array_split(outer, p2)[c2]
                        r0, _, nr, _ = orc.nd_share([S0, S0], [p1, p2], [c1, c2], D, 1)
                        _, q0, _, nq = orc.nd_share([S1, S1], [p1, p2], [c1, c2], 1, D)
                        assert nr == len(want) and nq == len(want)
                        if nr:
                            assert r0 == want[0] and q0 == want[0]
                        # a split over p1*p2 when it divides D
                        if D % (p1 * p2) == 0:
                            flat = np.array_split(np.arange(D), p1 * p2)[c1 * p2 + c2]
                            assert nr == len(flat) and (nr == 0 or r0 == flat[0])


def test_3d_rule_output_state(orc):
    # Sec. 4.2: I (S0, B, S1) and W (B, S1, S0) give O (S0, S1, P)
    t = orc.nd_tags([S0, B, S1], [B, S1, S0])
    assert t[2] == [S0, S1, P]
    # p1 = p2 = 1 reduces to data parallelism: same local product as 1-D DP
    rng = np.random.default_rng(3)
    X, W = rng.integers(-3, 4, (10, 6)).astype(np.float32), rng.integers(-3, 4, (6, 5)).astype(np.float32)
    for r in range(4):
        nd = orc.nd_linear(oracle.FWD, X, W, None, [S0, B, S1], [B, S1, S0], [4, 1, 1], [r, 0, 0])
        assert np.array_equal(nd, orc.linear(oracle.DP, oracle.FWD, X, W, None, 4, r))


def test_single_axis_mesh_reduces_to_1d(orc):
    rng = np.random.default_rng(4)
    M, K, N = 11, 9, 7
    X, W, dY = (rng.standard_normal(s).astype(np.float32) for s in ((M, K), (K, N), (M, N)))
    for name, sig in (("DP", oracle.DP), ("COL", oracle.COL), ("KS", oracle.KS)):
        xs, ws = FACTOR[name]
        for p in (1, 3, 4):
            for r in range(p):
                for op in OPS:
                    want = orc.linear(sig, op, X, W, dY, p, r)
                    got1 = orc.nd_linear(op, X, W, dY, [xs], [ws], [p], [r])
                    got3 = orc.nd_linear(op, X, W, dY, [B, xs, B], [B, ws, B], [1, p, 1], [0, r, 0])
                    assert np.array_equal(got1, want) and np.array_equal(got3, want)


def test_nd_samples_match_blocks(orc):
    rng = np.random.default_rng(6)
    M, K, N = 20, 14, 18
    X, W, dY = (rng.standard_normal(s).astype(np.float32) for s in ((M, K), (K, N), (M, N)))
    xs, ws = [S0, B, S1], [B, S1, S0]
    for c in ((1, 0, 1), (0, 1, 0)):
        for op in OPS:
            full = orc.nd_linear(op, X, W, dY, xs, ws, (2, 2, 2), c)
            ii = rng.integers(0, full.shape[0], 30)
            jj = rng.integers(0, full.shape[1], 30)
            got = orc.nd_linear_samples(op, X, W, dY, xs, ws, (2, 2, 2), c, ii, jj)
            assert np.array_equal(got, full[ii, jj])


def test_bad_nd_arguments_raise(orc):
    X = np.ones((4, 4), np.float32)
    with pytest.raises(ValueError):
        orc.nd_tags([S0, P], [B, P])                       # two Partial-sum operands
    with pytest.raises(ValueError):
        orc.nd_tags([S1], [S1])                            # no factor
    with pytest.raises(ValueError):
        orc.nd_linear(oracle.FWD, X, X, None, [S0], [B], [2], [2])   # coordinate out of range
    with pytest.raises(ValueError):
        orc.nd_share([(oracle.BCAST, 0)], [2], [0], 4, 4)  # Broadcast with an axis


ND_MUTATIONS = [
    ("nested split cuts the full extent", "orc_split(s.nr, p[a], c[a], &off, &len);",
     "orc_split(rows, p[a], c[a], &off, &len);"),
    ("nested offsets overwrite instead of accumulate", "s.c0 += off;", "s.c0 = off;"),
    ("last mesh axis varies fastest",
     "int64_t node_stride = 1, gpu_stride = 1;\n    for (int a = 0; a < d; ++a) {",
     "int64_t node_stride = 1, gpu_stride = 1;\n    for (int a = d - 1; a >= 0; --a) {"),
    ("factor search skips the partial-input signatures", "for (int sig = 0; sig < 6; ++sig) {",
     "for (int sig = 0; sig < 3; ++sig) {"),
    ("dY share taken from W's states", "pl->dy = nd_share_of(d, kinds + 3 * d, axes + 3 * d",
     "pl->dy = nd_share_of(d, kinds + 1 * d, axes + 1 * d"),
]


@pytest.mark.parametrize("name,old,new", ND_MUTATIONS, ids=[m[0] for m in ND_MUTATIONS])
def test_planted_nd_mistakes_are_caught(tmp_path, name, old, new):
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, "mutation anchor not found: " + name
    mut = tmp_path / "oracle_mut.c"
    mut.write_text(src.replace(old, new))
    lib = oracle.build(force=True, src=str(mut), out=str(tmp_path / "liboracle_mut.so"))
    bad = oracle.Oracle(lib)
    checks = (lambda: test_listing1_blocks(bad), lambda: test_hetero_mapping_golden(bad),
              lambda: test_nested_split_matches_numpy(bad), lambda: test_3d_rule_output_state(bad))
    caught = bool(nd_invariant_failures(bad))
    for chk in checks:
        if caught:
            break
        try:
            chk()
        except (AssertionError, ValueError):
            caught = True
    assert caught, "planted mistake not caught: " + name
