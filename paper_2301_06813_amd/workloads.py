"""The workloads: shapes, SBP signatures, seeds and value distributions.

Each workload is a list of linear layers ``Y = X W`` with global
X (M x K), W (K x N) and upstream gradient dY (M x N), a device count p and
one SBP signature per linear (AutoDDL Sec. 4.2; each layer gets its own
strategy, Sec. 4.4). Only rank r's share of each linear runs on the GPU.

Signatures (1-D factors of the 3-D SBP matmul rule of Sec. 4.2):
    "DP"  (S(0), B)    -> S(0)   data parallel
    "COL" (B,    S(1)) -> S(1)   column split of W
    "KS"  (S(1), S(0)) -> P      split of the reduction dimension

Workload 6 runs on a 2 x 2 x 2 device mesh: each linear carries one factor
per mesh axis (nd-SBP, Sec. 4.1 Listing 1 and the 3-D rule of Sec. 4.2),
and its "ranks" are mesh coordinates.

Seeds: tensor t of linear l in workload c uses ``1000*c + 10*l + t`` with
t = 1 (X), 2 (W), 3 (dY); workload 5 draws its signatures from seed 5000.
Weights are N(0, gain/K) with K the global fan-in.

The paper names no dataset; these synthetic tensors stand in for the layer
shapes of its Transformer (Sec. 5, small GPT-style model on 32 A100s: 24
layers, hidden 1024, 16 heads) and of the VGG classifier head.
"""
from __future__ import annotations

import dataclasses
import math
import random

import torch

from . import inputs

SIGS = ("DP", "COL", "KS")


@dataclasses.dataclass(frozen=True)
class Linear:
    name: str
    M: int            # tokens (global)
    K: int            # fan-in (global)
    N: int            # fan-out (global)
    sig: str          # "DP" | "COL" | "KS"
    seed_base: int    # seeds are seed_base + 1 (X), + 2 (W), + 3 (dY)
    x_std: float = 1.0
    x_relu: bool = False
    w_gain: float = 1.0   # W ~ N(0, w_gain / K)
    dy_std: float = 1.0
    factors: tuple = ()   # nd workloads: one signature name per mesh axis

    @property
    def w_std(self) -> float:
        return math.sqrt(self.w_gain / self.K)

    def flops_per_op(self, p: int) -> float:
        """2 m n k of one of the three local GEMMs (all three are equal)."""
        return 2.0 * self.M * self.K * self.N / p


@dataclasses.dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    dtype: torch.dtype
    p: int
    linears: tuple
    ranks: tuple          # ranks (nd workloads: mesh coordinates) that parity covers
    mesh: tuple = ()      # nd workloads: devices per mesh axis (p = their product)


def tiny_fp32() -> list[Workload]:
    """Workload 1: global X 64x128, W 128x256, dY 64x256, all N(0,1), p = 4,
    fp32, every signature and every rank."""
    out = []
    for sig in SIGS:
        lin = Linear("tiny_" + sig, 64, 128, 256, sig, 1000, w_gain=128.0)
        out.append(Workload(1, "tiny_fp32_" + sig, torch.float32, 4, (lin,), (0, 1, 2, 3)))
    return out


def ffn_shard() -> Workload:
    """Workload 2: Transformer FFN, 8192 tokens, hidden 1024, ffn 4096, p = 8.
    FC1 under (B,S(1))->S(1); FC2 under (S(1),S(0))->P."""
    fc1 = Linear("fc1", 8192, 1024, 4096, "COL", 2000)
    fc2 = Linear("fc2", 8192, 4096, 1024, "KS", 2010)
    return Workload(2, "transformer_ffn_p8", torch.bfloat16, 8, (fc1, fc2), tuple(range(8)))


def attention_dp() -> Workload:
    """Workload 3: attention projections under data parallelism, 64 x 512 tokens,
    hidden 1024, p = 8 (4096 tokens per rank)."""
    qkv = Linear("qkv", 64 * 512, 1024, 3072, "DP", 3000)
    o = Linear("out", 64 * 512, 1024, 1024, "DP", 3010)
    return Workload(3, "attention_proj_dp_p8", torch.bfloat16, 8, (qkv, o), tuple(range(8)))


def vgg_head() -> Workload:
    """Workload 4: VGG classifier head, global batch 256, p = 8. FC6 25088->4096
    K-split (P output), FC7 4096->4096 and FC8 4096->1000 column split.
    Inputs ReLU(N(0,1)), W ~ N(0, 2/K)."""
    fc6 = Linear("fc6", 256, 25088, 4096, "KS", 4000, x_relu=True, w_gain=2.0)
    fc7 = Linear("fc7", 256, 4096, 4096, "COL", 4010, x_relu=True, w_gain=2.0)
    fc8 = Linear("fc8", 256, 4096, 1000, "COL", 4020, x_relu=True, w_gain=2.0)
    return Workload(4, "vgg_fc_head_p8", torch.bfloat16, 8, (fc6, fc7, fc8), tuple(range(8)))


def transformer_step(layers: int = 24) -> Workload:
    """Workload 5: the linears of a 24-layer Transformer (hidden 1024, ffn 4096,
    16 heads, 8192 tokens, p = 8); one seeded signature per linear; rank 0."""
    rnd = random.Random(5000)
    lins = []
    dims = (("qkv", 1024, 3072), ("out", 1024, 1024), ("fc1", 1024, 4096), ("fc2", 4096, 1024))
    ell = 0
    for layer in range(layers):
        for nm, k, n in dims:
            sig = SIGS[rnd.randrange(3)]
            lins.append(Linear("L%02d_%s" % (layer, nm), 8192, k, n, sig, 5000 + 10 * ell))
            ell += 1
    return Workload(5, "transformer_24L_step_rank0_p8", torch.bfloat16, 8, tuple(lins), (0,))


# Network parameters the search assumes for one node of 8 MI355X GPUs (a
# reading, not a measurement: the paper fits alpha and beta on its own
# clusters): 10 us per message, and one xGMI link's ~153 GB/s per byte, as
# a ring algorithm is bound by one link.
XGMI_ALPHA = 10e-6
XGMI_BETA = 1.0 / 153e9


def searched_signatures(layers: int = 24, p: int = 8, tokens: int = 8192, restarts: int = 64,
                        seed: int = 8000):
    """Per-linear signatures of the 24-layer Transformer chosen by the
    library's coordinate-descent search (Sec. 4.4) over DP, COL and KS,
    minimising the alpha-beta communication cost (Table 2) of one step:
    tokens enter and leave data parallel (S0); bf16 activations, fp32 weight
    gradients. Returns (signature names, modelled seconds per step)."""
    from . import sbp
    dims = (("qkv", 1024, 3072), ("out", 1024, 1024), ("fc1", 1024, 4096), ("fc2", 4096, 1024))
    K = [k for _ in range(layers) for _, k, _ in dims]
    N = [n for _ in range(layers) for _, _, n in dims]
    net = sbp.make_chain(p, XGMI_ALPHA, XGMI_BETA, tokens, K, N, 2.0, 4.0,
                         (sbp.SBP_SPLIT, 0), (sbp.SBP_SPLIT, 0), ("DP", "COL", "KS"))
    ids, cost, _ = sbp.sbp_search_strategy(net, restarts=restarts, seed=seed)
    names = {v: k for k, v in sbp.SIG_IDS.items()}
    return [names[i] for i in ids], cost


def transformer_step_searched(layers: int = 24) -> Workload:
    """Workload 8: workload 5's 96 linears with the signatures the strategy
    search picks (searched_signatures) instead of a random draw; rank 0."""
    sigs, _ = searched_signatures(layers)
    dims = (("qkv", 1024, 3072), ("out", 1024, 1024), ("fc1", 1024, 4096), ("fc2", 4096, 1024))
    lins = []
    ell = 0
    for layer in range(layers):
        for nm, k, n in dims:
            lins.append(Linear("L%02d_%s" % (layer, nm), 8192, k, n, sigs[ell], 8000 + 10 * ell))
            ell += 1
    return Workload(8, "transformer_24L_step_searched_rank0_p8", torch.bfloat16, 8, tuple(lins),
                    (0,))


def transformer_3d() -> Workload:
    """Workload 6: the four linears of one Transformer layer (8192 tokens,
    hidden 1024, ffn 4096) on a 2 x 2 x 2 mesh of 8 devices, each under the
    3-D rule of Sec. 4.2: X (S0, B, S1), W (B, S1, S0) -> Y (S0, S1, P), so
    every device multiplies a (M/2) x (K/2) share of X by a (K/2) x (N/2)
    share of W (the paper prefers a 3-D strategy for attention layers,
    Sec. 4.5). Parity covers all eight devices; the benchmark reports device
    (0, 0, 0)."""
    mesh = (2, 2, 2)
    f3 = ("DP", "COL", "KS")
    dims = (("qkv", 1024, 3072), ("out", 1024, 1024), ("fc1", 1024, 4096), ("fc2", 4096, 1024))
    lins = tuple(Linear(nm, 8192, k, n, "3D", 6000 + 10 * i, factors=f3)
                 for i, (nm, k, n) in enumerate(dims))
    coords = tuple((a, b, c) for a in range(2) for b in range(2) for c in range(2))
    return Workload(6, "transformer_layer_3d_mesh2x2x2", torch.bfloat16, 8, lins, coords, mesh)


@dataclasses.dataclass(frozen=True)
class AttentionCore:
    """The attention core of a Transformer layer under a head split: per
    sequence and local head, scores S = Q K^T, context O = P V and their
    backward products (Sec. 2: multi-head attention reduces to batched
    matrix products)."""
    name: str
    batch: int        # sequences
    heads: int        # global heads H
    seq: int
    head_dim: int
    p: int            # devices splitting the heads
    seed_base: int


def attention_core() -> AttentionCore:
    """Workload 7: the attention core of the 24-layer Transformer (16 heads of
    64, sequence 1024) for 8 sequences (the 8192 tokens of workload 5), heads
    split over 8 devices (2 per device). Q, K and V are views into a fused
    [batch][seq][3][heads][head_dim] QKV activation drawn N(0,1); P is a
    row-softmax of N(0,1) logits; dS and dO are N(0,1)."""
    return AttentionCore("attention_core_h16x64_s1024_b8_p8", 8, 16, 1024, 64, 8, 7000)


def all_workloads() -> list[Workload]:
    return tiny_fp32() + [ffn_shard(), attention_dp(), vgg_head(), transformer_step(),
                          transformer_3d()]


def make_tensors(lin: Linear, dtype, device="cpu"):
    """Global X, W, dY of one linear, drawn by the recipe in this module's docstring."""
    X = inputs.randn((lin.M, lin.K), lin.x_std, lin.seed_base + 1, dtype, device, lin.x_relu)
    W = inputs.randn((lin.K, lin.N), lin.w_std, lin.seed_base + 2, dtype, device)
    dY = inputs.randn((lin.M, lin.N), lin.dy_std, lin.seed_base + 3, dtype, device)
    return X, W, dY
