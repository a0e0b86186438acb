"""Pins for the oracle's attention-core products (Sec. 2: multi-head
attention reduces to batched matrix products; the head dimension split over
p devices), against things other than the oracle itself:

* one device (p = 1): every product equals numpy's batched matmul of the
  textbook definition (S = Q K^T, O = P V, dQ = dS K, dK = dS^T Q,
  dP = dO V^T, dV = P^T dO), exactly on integer inputs;
* the head split: the devices' outputs concatenated over heads equal the
  one-device output, for uneven head counts;
* the adjoint identities that tie each backward product to its forward
  product: <dS, Q K^T> = <dS K, Q> = <dS^T Q, K> and
  <dO, P V> = <dO V^T, P> = <P^T dO, V>, exactly on integer inputs;
* planted mistakes in copies of oracle.c are caught by these checks.
"""
import numpy as np
import pytest

import oracle

B, H, SQ, SK, D = 2, 5, 7, 6, 4


def _ints(rng, *shape):
    return rng.integers(-3, 4, shape).astype(np.float32)


def _operands(rng):
    return dict(Q=_ints(rng, B, H, SQ, D), K=_ints(rng, B, H, SK, D), V=_ints(rng, B, H, SK, D),
                P=_ints(rng, B, H, SQ, SK), dS=_ints(rng, B, H, SQ, SK),
                dO=_ints(rng, B, H, SQ, D))


# product -> (operand names in the oracle's order, numpy definition)
def _mt(x):
    return np.swapaxes(x, -1, -2)


PRODUCTS = {
    oracle.ATT_S: (("Q", "K"), lambda q, k: q @ _mt(k)),
    oracle.ATT_O: (("P", "V"), lambda p_, v: p_ @ v),
    oracle.ATT_DQ: (("dS", "K"), lambda ds, k: ds @ k),
    oracle.ATT_DK: (("dS", "Q"), lambda ds, q: _mt(ds) @ q),
    oracle.ATT_DP: (("dO", "V"), lambda do, v: do @ _mt(v)),
    oracle.ATT_DV: (("P", "dO"), lambda p_, do: _mt(p_) @ do),
}


def attn_failures(orc):
    bad = []
    rng = np.random.default_rng(12)
    t = _operands(rng)
    td = {k: v.astype(np.float64) for k, v in t.items()}
    for which, (names, ref) in PRODUCTS.items():
        try:
            one = orc.attn(which, t[names[0]], t[names[1]], 1, 0, SQ, SK, D)
            if not np.array_equal(one, ref(td[names[0]], td[names[1]])):
                bad.append((which, "p=1"))
                continue
            for p in (2, 3, 4):
                parts = [orc.attn(which, t[names[0]], t[names[1]], p, r, SQ, SK, D)
                         for r in range(p)]
                if not np.array_equal(np.concatenate(parts, axis=1), one):
                    bad.append((which, "p=%d" % p))
        except ValueError:
            bad.append((which, "error"))
    # adjoint identities, per device of a 3-way head split
    for r in range(3):
        try:
            S = orc.attn(oracle.ATT_S, t["Q"], t["K"], 3, r, SQ, SK, D)
            dQ = orc.attn(oracle.ATT_DQ, t["dS"], t["K"], 3, r, SQ, SK, D)
            dK = orc.attn(oracle.ATT_DK, t["dS"], t["Q"], 3, r, SQ, SK, D)
            O = orc.attn(oracle.ATT_O, t["P"], t["V"], 3, r, SQ, SK, D)
            dP = orc.attn(oracle.ATT_DP, t["dO"], t["V"], 3, r, SQ, SK, D)
            dV = orc.attn(oracle.ATT_DV, t["P"], t["dO"], 3, r, SQ, SK, D)
        except ValueError:
            bad.append(("adjoint", r))
            continue
        off, hr = orc.split(H, 3, r)
        sl = slice(off, off + hr)
        ds, q, k = td["dS"][:, sl], td["Q"][:, sl], td["K"][:, sl]
        do, p_, v = td["dO"][:, sl], td["P"][:, sl], td["V"][:, sl]
        if not (np.sum(ds * S) == np.sum(dQ * q) == np.sum(dK * k)):
            bad.append(("adjoint scores", r))
        if not (np.sum(do * O) == np.sum(dP * p_) == np.sum(dV * v)):
            bad.append(("adjoint context", r))
    return bad


def test_attention_products_pinned(orc):
    assert attn_failures(orc) == []


def test_attention_random_fp32_close(orc):
    rng = np.random.default_rng(3)
    Q, K = (rng.standard_normal(s).astype(np.float32) for s in ((2, 3, 33, 16), (2, 3, 17, 16)))
    got = orc.attn(oracle.ATT_S, Q, K, 1, 0, 33, 17, 16)
    np.testing.assert_allclose(got, Q.astype(np.float64) @ _mt(K.astype(np.float64)),
                               rtol=1e-12, atol=1e-12)


def test_attention_bad_arguments(orc):
    Q = np.ones((1, 2, 3, 4), np.float32)
    with pytest.raises(ValueError):
        orc.attn(6, Q, Q, 1, 0, 3, 3, 4)
    with pytest.raises(ValueError):
        orc.attn(oracle.ATT_S, Q, Q, 2, 2, 3, 3, 4)


ATT_MUTATIONS = [
    ("scores read K transposed",
     "acc += decode(T1, enc, m1 + i * c1 + t) * decode(T2, enc, m2 + j * c2 + t);\n                        break;\n                    case ORC_ATT_O:",
     "acc += decode(T1, enc, m1 + i * c1 + t) * decode(T2, enc, m2 + t * c2 + j);\n                        break;\n                    case ORC_ATT_O:"),
    ("head offset ignored", "const int64_t m1 = (b * nh + h0 + h) * s1, m2 = (b * nh + h0 + h) * s2;",
     "const int64_t m1 = (b * nh + h) * s1, m2 = (b * nh + h) * s2;"),
    ("transposed-A products sum over the key length", "for (int64_t t = 0; t < sq; ++t)\n                            acc += decode(T1, enc, m1 + t * c1 + i)",
     "for (int64_t t = 0; t < sk && t < sq; ++t)\n                            acc += decode(T1, enc, m1 + t * c1 + i)"),
    ("dP shape swapped", "case ORC_ATT_DP: *orow = sq; *ocol = sk;", "case ORC_ATT_DP: *orow = sk; *ocol = sq;"),
]


@pytest.mark.parametrize("name,old,new", ATT_MUTATIONS, ids=[m[0] for m in ATT_MUTATIONS])
def test_planted_attention_mistakes_are_caught(tmp_path, name, old, new):
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, "mutation anchor not found: " + name
    mut = tmp_path / "oracle_mut.c"
    mut.write_text(src.replace(old, new))
    lib = oracle.build(force=True, src=str(mut), out=str(tmp_path / "liboracle_mut.so"))
    assert attn_failures(oracle.Oracle(lib)), "planted mistake not caught: " + name
