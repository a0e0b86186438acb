"""Cost model and exhaustive strategy search, for checking the library's
coordinate-descent search.

TEST INFRASTRUCTURE ONLY (like the rest of this package): the tests may
import it; the product path never does.

What it computes (AutoDDL Sec. 3.1 and Table 2; Sec. 4.2-4.4):

* collective times of the alpha-beta model, as printed in Table 2: with n
  the message size (ReduceScatter's input, the other collectives' output,
  per device),
      AllReduce               (2p - 1) a + 2 (p - 1) / p n b
      AllGather, ReduceScatter (p - 1) a + (p - 1) / p n b
      AlltoAll                 (p - 1) a + n b
* redistribution of a tensor between 1-D states (the collectives named in
  Sec. 4.2 and 4.3): Split -> other Split: AlltoAll (each device ends with
  1/p of the tensor); Split -> Broadcast: AllGather; Partial-sum -> Split:
  ReduceScatter; Partial-sum -> Broadcast: AllReduce; anything else local;
* a chain of linear layers, one signature each, costs the forward
  redistributions between consecutive layers, the backward moves of their
  gradients (the gradient of S is S, of B is P, of P is B), and an AllReduce
  of every weight gradient left Partial-sum (Sec. 4.3);
* exhaustive search over every assignment of signatures.

States are (kind, axis) pairs in the oracle's numbering; signatures are the
oracle's ids (oracle.DP, ...), whose X, Y and dW states come from
oracle.tags().
"""
from __future__ import annotations

import itertools

import oracle

ALLREDUCE, ALLGATHER, REDUCESCATTER, ALLTOALL = 0, 1, 2, 3


def collective(coll, p, n, alpha, beta):
    if coll == ALLREDUCE:
        return (2 * p - 1) * alpha + 2 * (p - 1) / p * n * beta
    if coll in (ALLGATHER, REDUCESCATTER):
        return (p - 1) * alpha + (p - 1) / p * n * beta
    if coll == ALLTOALL:
        return (p - 1) * alpha + n * beta
    raise ValueError(coll)


def boxing_collective(frm, to):
    """The collective that moves a tensor from state frm to state to, or None."""
    (fk, fa), (tk, ta) = frm, to
    if fk == oracle.SPLIT and tk == oracle.SPLIT and fa != ta:
        return ALLTOALL
    if fk == oracle.SPLIT and tk == oracle.BCAST:
        return ALLGATHER
    if fk == oracle.PARTIAL and tk == oracle.SPLIT:
        return REDUCESCATTER
    if fk == oracle.PARTIAL and tk == oracle.BCAST:
        return ALLREDUCE
    return None


def boxing(frm, to, nbytes, p, alpha, beta):
    coll = boxing_collective(frm, to)
    if coll is None:
        return 0.0
    n = nbytes / p if coll == ALLTOALL else nbytes
    return collective(coll, p, n, alpha, beta)


def grad_state(st):
    k, a = st
    return {oracle.BCAST: (oracle.PARTIAL, -1), oracle.PARTIAL: (oracle.BCAST, -1)}.get(k, st)


def chain_cost(net, sigs):
    """Communication time of one step of the chain `net` (a dict: p, alpha,
    beta, M, K (list), N (list), act_bytes, grad_bytes, in_state, out_state)
    under signatures sigs."""
    p, a, b = net["p"], net["alpha"], net["beta"]
    total = 0.0
    prev = net["in_state"]
    nbytes = net["M"] * net["K"][0] * net["act_bytes"]
    for l, sig in enumerate(sigs):
        X, W, Y, dY, dX, dW = oracle.tags(sig)
        if X[0] == oracle.PARTIAL:
            raise ValueError("a chain link never takes a Partial-sum input")
        total += boxing(prev, X, nbytes, p, a, b)                       # forward
        total += boxing(grad_state(X), grad_state(prev), nbytes, p, a, b)   # backward
        if dW[0] == oracle.PARTIAL:
            total += collective(ALLREDUCE, p, net["K"][l] * net["N"][l] * net["grad_bytes"], a, b)
        prev = Y
        nbytes = net["M"] * net["N"][l] * net["act_bytes"]
    out = net["out_state"]
    total += boxing(prev, out, nbytes, p, a, b) + boxing(grad_state(out), grad_state(prev),
                                                         nbytes, p, a, b)
    return total


def exhaustive(net, choices):
    """(minimum cost, one minimising assignment) over every assignment of the
    signatures in `choices` to the layers."""
    best = None
    for sigs in itertools.product(choices, repeat=len(net["K"])):
        c = chain_cost(net, sigs)
        if best is None or c < best[0]:
            best = (c, sigs)
    return best
