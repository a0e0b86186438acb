"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no arithmetic of the SBP linear layer: it only draws
tensors. The library and the oracle both consume exactly the bits drawn
here (bf16 inputs are rounded once, on the device that drew them, by
torch's round-to-nearest-even conversion).

Recipe: ``torch.Generator(device).manual_seed(seed)``, then
``torch.randn(shape) * std`` in fp32, optionally ``relu``, then ``.to(bf16)``
for bf16 workloads. Integer-valued inputs (exact-arithmetic tests) are
``torch.randint(lo, hi + 1)`` cast to the input dtype.
"""
from __future__ import annotations

import numpy as np
import torch


def randn(shape, std: float, seed: int, dtype=torch.bfloat16, device="cpu",
          relu: bool = False) -> torch.Tensor:
    """N(0, std^2) values (ReLU-ed if asked), drawn in fp32 and rounded once to dtype."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    t = torch.randn(tuple(shape), generator=g, dtype=torch.float32, device=device)
    if std != 1.0:
        t.mul_(std)
    if relu:
        t.clamp_(min=0.0)
    return t.to(dtype)


def randint(shape, lo: int, hi: int, seed: int, dtype=torch.bfloat16,
            device="cpu") -> torch.Tensor:
    """Integers drawn uniformly from [lo, hi], stored exactly in dtype."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    t = torch.randint(lo, hi + 1, tuple(shape), generator=g, device=device,
                      dtype=torch.int32)
    return t.to(dtype)


def host_bits(t: torch.Tensor) -> np.ndarray:
    """Host copy in the oracle's input encoding: uint16 bit patterns for bf16, fp32 as is."""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.numpy()
    raise TypeError("unsupported input dtype %s" % t.dtype)
