"""Shared helpers for the GPU tests: run one local product through the C ABI
and compare it with the oracle."""
import sys

import numpy as np
import torch

import oracle
from paper_2301_06813_amd import inputs, linear, sbp

SIG_ID = {"DP": oracle.DP, "COL": oracle.COL, "KS": oracle.KS, "PB": oracle.PB,
          "BP": oracle.BP, "BB": oracle.BB}
OP_ID = {"fwd": oracle.FWD, "bwd_data": oracle.BWD_DATA, "bwd_weight": oracle.BWD_WEIGHT}
TILES = [(256, 256), (256, 192), (256, 128), (128, 256), (128, 128), (128, 64), (64, 128), (64, 64)]
KERNELS = (1, 2)   # pipelined direct-to-LDS, generic
# (tile, kernel) pairs beyond TILES x KERNELS: the two-stage pipelined 128x128,
# the eight-wave instances with two reduction groups (staged and row-quad
# epilogues) and the row-quad instances with one group
EXTRA_TILE_KERNELS = [((128, 128), 4), ((128, 128), 5), ((256, 128), 5), ((128, 256), 5),
                      ((256, 256), 6), ((128, 128), 6), ((128, 128), 7), ((256, 128), 7),
                      ((128, 256), 7), ((256, 256), 8), ((256, 128), 9), ((128, 256), 9),
                      ((128, 128), 9), ((128, 128), 10), ((128, 64), 4), ((64, 128), 4),
                      ((64, 64), 4), ((128, 64), 11), ((64, 128), 11), ((64, 64), 11),
                      ((128, 64), 5), ((64, 128), 5), ((64, 64), 5), ((128, 64), 7),
                      ((64, 128), 7), ((64, 64), 7), ((128, 128), 12), ((128, 64), 12),
                      ((64, 128), 12), ((64, 64), 12), ((128, 128), 13), ((128, 64), 13),
                      ((64, 128), 13), ((64, 64), 13)]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def out_bits(t: torch.Tensor) -> np.ndarray:
    return inputs.host_bits(t)


def decode(t: torch.Tensor) -> np.ndarray:
    """GPU output as fp64 (bf16 decoded exactly)."""
    b = out_bits(t)
    if b.dtype == np.uint16:
        return oracle.bf16_to_f64(b)
    return b.astype(np.float64)


def normwise_rel(got: np.ndarray, want: np.ndarray) -> float:
    """max |g - o| / max(max |o|, 2^-126) over the compared elements."""
    if want.size == 0:
        return 0.0
    den = max(float(np.max(np.abs(want))), 2.0 ** -126)
    return float(np.max(np.abs(got - want))) / den


def run_gpu(op, sig, p, r, X, W, dY, stream=None):
    out, st = linear.call(op, sig, p, r, X, W, dY, stream)
    torch.cuda.synchronize()
    return out, st


def expect_state(op, sig, p, r, st):
    """The state the oracle's table assigns to the output."""
    t = oracle.tags(SIG_ID[sig])
    kind, axis = t[{"fwd": 2, "bwd_data": 4, "bwd_weight": 5}[op]]
    to_abi = {oracle.SPLIT: sbp.SBP_SPLIT, oracle.BCAST: sbp.SBP_BROADCAST,
              oracle.PARTIAL: sbp.SBP_PARTIAL}
    assert (st.kind, st.axis, st.p, st.r) == (to_abi[kind], axis, p, r), (op, sig, st)


def oracle_full(op, sig, p, r, Xh, Wh, dYh):
    return oracle.linear(SIG_ID[sig], OP_ID[op], Xh, Wh, dYh, p, r)
