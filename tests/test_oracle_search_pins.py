"""Pins for the oracle's cost model (oracle/search.py) against what the
paper states about specific strategies:

* pure data parallelism moves no activations: its whole cost is one
  AllReduce of every weight gradient (Sec. 4.3: replicated weights receive
  partial-sum gradients that are all-reduced);
* the Megatron MLP pattern -- column split, then K-split (Sec. 2, Fig. 2) --
  between replicated activations costs exactly one AllReduce of the output
  in the forward pass and one in the backward pass, and no weight sync;
* every redistribution's backward move uses the dual collective: AllGather
  and ReduceScatter pair up, AllReduce and AlltoAll are their own duals
  (Sec. 4.2: the redistributions of the forward path recur in the backward
  path), and moves the same data, so it costs the same;
* data parallelism followed by a column split all-gathers the activation
  forward and reduce-scatters its gradient backward (Sec. 4.2);
* the AlltoAll of a split-axis change sends each device's share, so its
  bandwidth term is the tensor over p;
* every collective's time equals Table 2's formula evaluated by hand at fixed
  points (tests/golden/table2_collectives.json), where latency-only and
  bandwidth-only points separate each coefficient;
* planted mistakes in copies of search.py are caught by these checks, one
  per coefficient of Table 2 among them.
"""
import importlib.util
import itertools
import json
import os

import pytest

import oracle
from oracle import search as S

S0, S1, B, P = (oracle.SPLIT, 0), (oracle.SPLIT, 1), (oracle.BCAST, -1), (oracle.PARTIAL, -1)
STATES = (S0, S1, B, P)
TABLE2 = os.path.join(os.path.dirname(__file__), "golden", "table2_collectives.json")


def table2_cases():
    with open(TABLE2) as f:
        return json.load(f)["cases"]


def _net(K, N, p=8, alpha=1e-5, beta=1e-10, M=4096, ins=S0, outs=S0):
    return dict(p=p, alpha=alpha, beta=beta, M=M, K=list(K), N=list(N), act_bytes=2.0,
                grad_bytes=4.0, in_state=ins, out_state=outs)


def checks(mod):
    """Names of the pins that fail for search module `mod`."""
    bad = []
    # Table 2 as printed, evaluated by hand (exact in binary floating point)
    names = (("allreduce", mod.ALLREDUCE), ("allgather", mod.ALLGATHER),
             ("reducescatter", mod.REDUCESCATTER), ("alltoall", mod.ALLTOALL))
    for c in table2_cases():
        for name, coll in names:
            got = mod.collective(coll, c["p"], c["n"], c["alpha"], c["beta"])
            if abs(got - c[name]) > 1e-12 * max(1.0, abs(c[name])):
                bad.append("table 2 %s at p=%d n=%g alpha=%g beta=%g" % (
                    name, c["p"], c["n"], c["alpha"], c["beta"]))
    for p in (2, 4, 8):
        net = _net([1024, 3072, 1024], [3072, 1024, 4096], p=p)
        dp = mod.chain_cost(net, [oracle.DP] * 3)
        ar = sum(mod.collective(mod.ALLREDUCE, p, k * n * 4.0, net["alpha"], net["beta"])
                 for k, n in zip(net["K"], net["N"]))
        if abs(dp - ar) > 1e-15 * max(1.0, ar):
            bad.append("data parallelism")
        mlp = _net([1024, 4096], [4096, 1024], p=p, ins=B, outs=B)
        y = mod.chain_cost(mlp, [oracle.COL, oracle.KS])
        want = 2 * mod.collective(mod.ALLREDUCE, p, mlp["M"] * 1024 * 2.0, mlp["alpha"],
                                  mlp["beta"])
        if abs(y - want) > 1e-15 * max(1.0, want):
            bad.append("megatron mlp")
    # data parallel then column split: the activation is all-gathered in the
    # forward pass and its gradient reduce-scattered in the backward pass
    # (Sec. 4.2), on top of the data-parallel weight's AllReduce
    for p in (2, 8):
        net = _net([1024, 2048], [2048, 512], p=p, outs=S1)
        act = net["M"] * 2048 * 2.0
        want = (mod.collective(mod.ALLREDUCE, p, 1024 * 2048 * 4.0, net["alpha"], net["beta"]) +
                mod.collective(mod.ALLGATHER, p, act, net["alpha"], net["beta"]) +
                mod.collective(mod.REDUCESCATTER, p, act, net["alpha"], net["beta"]))
        got = mod.chain_cost(net, [oracle.DP, oracle.COL])
        if abs(got - want) > 1e-15 * max(1.0, want):
            bad.append("dp then column")
    dual = {None: None, mod.ALLGATHER: mod.REDUCESCATTER, mod.REDUCESCATTER: mod.ALLGATHER,
            mod.ALLREDUCE: mod.ALLREDUCE, mod.ALLTOALL: mod.ALLTOALL}
    for a, b in itertools.product(STATES, STATES):
        f = mod.boxing_collective(a, b)
        g = mod.boxing_collective(mod.grad_state(b), mod.grad_state(a))
        if dual[f] != g:
            bad.append("duality %s->%s" % (a, b))
    # an AllGather and the ReduceScatter that mirrors it move the same data:
    # a redistribution and its backward move cost the same
    for a, b in itertools.product(STATES, STATES):
        for p in (2, 8):
            f = mod.boxing(a, b, 3e6, p, 1e-5, 1e-10)
            g = mod.boxing(mod.grad_state(b), mod.grad_state(a), 3e6, p, 1e-5, 1e-10)
            if abs(f - g) > 1e-18:
                bad.append("mirror cost %s->%s" % (a, b))
    # AlltoAll: bandwidth term of a split-axis change is bytes / p
    for p in (2, 8):
        c = mod.boxing(S0, S1, 1e6, p, 0.0, 1.0)
        if abs(c - 1e6 / p) > 1e-9:
            bad.append("alltoall share")
    # a split into another split, a broadcast into a split and a split into a
    # partial sum need no communication only where stated
    if mod.boxing(B, S0, 1e6, 8, 1.0, 1.0) != 0 or mod.boxing(S1, P, 1e6, 8, 1.0, 1.0) != 0:
        bad.append("local moves")
    if mod.boxing(S0, B, 1e6, 8, 0.0, 1.0) == 0 or mod.boxing(P, S1, 1e6, 8, 0.0, 1.0) == 0:
        bad.append("gathers and reductions")
    return bad


def test_search_oracle_pins():
    assert checks(S) == []


def test_exhaustive_is_a_lower_bound():
    net = _net([512, 2048, 512, 1024], [2048, 512, 1024, 768])
    c, sigs = S.exhaustive(net, (oracle.DP, oracle.COL, oracle.KS))
    assert abs(S.chain_cost(net, sigs) - c) == 0
    for other in itertools.product((oracle.DP, oracle.COL, oracle.KS), repeat=4):
        assert S.chain_cost(net, other) >= c


def test_partial_input_rejected():
    with pytest.raises(ValueError):
        S.chain_cost(_net([64], [64]), [oracle.PB])


SEARCH_MUTATIONS = [
    ("allgather priced as an alltoall", "    if coll in (ALLGATHER, REDUCESCATTER):",
     "    if coll == ALLGATHER:\n        return (p - 1) * alpha + n * beta\n    if coll in (REDUCESCATTER,):"),
    ("weight sync dropped", "        if dW[0] == oracle.PARTIAL:", "        if False:"),
    ("backward moves dropped", "        total += boxing(grad_state(X), grad_state(prev), nbytes, p, a, b)",
     "        total += 0.0"),
    ("alltoall sends the whole tensor", "    n = nbytes / p if coll == ALLTOALL else nbytes",
     "    n = nbytes"),
    ("allreduce latency term as an allgather's",
     "        return (2 * p - 1) * alpha + 2 * (p - 1) / p * n * beta",
     "        return (p - 1) * alpha + 2 * (p - 1) / p * n * beta"),
    ("allreduce bandwidth term without its factor 2",
     "        return (2 * p - 1) * alpha + 2 * (p - 1) / p * n * beta",
     "        return (2 * p - 1) * alpha + (p - 1) / p * n * beta"),
    ("allreduce priced as an allgather",
     "        return (2 * p - 1) * alpha + 2 * (p - 1) / p * n * beta",
     "        return (p - 1) * alpha + (p - 1) / p * n * beta"),
    ("allgather/reducescatter bandwidth term without (p-1)/p",
     "        return (p - 1) * alpha + (p - 1) / p * n * beta",
     "        return (p - 1) * alpha + n * beta"),
    ("allgather/reducescatter latency term with p",
     "        return (p - 1) * alpha + (p - 1) / p * n * beta",
     "        return p * alpha + (p - 1) / p * n * beta"),
    ("alltoall bandwidth term with (p-1)/p",
     "        return (p - 1) * alpha + n * beta",
     "        return (p - 1) * alpha + (p - 1) / p * n * beta"),
    ("alltoall latency term dropped",
     "        return (p - 1) * alpha + n * beta",
     "        return n * beta"),
    ("gradient of a broadcast stays broadcast",
     "    return {oracle.BCAST: (oracle.PARTIAL, -1), oracle.PARTIAL: (oracle.BCAST, -1)}.get(k, st)",
     "    return {oracle.PARTIAL: (oracle.BCAST, -1)}.get(k, st)"),
]


@pytest.mark.parametrize("name,old,new", SEARCH_MUTATIONS, ids=[m[0] for m in SEARCH_MUTATIONS])
def test_planted_search_mistakes_are_caught(tmp_path, name, old, new):
    src = open(S.__file__).read()
    assert src.count(old) == 1, "mutation anchor not found: " + name
    path = tmp_path / "search_mut.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("search_mut", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    try:
        caught = bool(checks(mod))
    except (ValueError, KeyError):
        caught = True
    assert caught, "planted mistake not caught: " + name
