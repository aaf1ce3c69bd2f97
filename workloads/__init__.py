"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This module holds none of the attention arithmetic: it only draws random
numbers (q, k, v ~ N(0, 1)) and per-KV-head elastic-rule parameters
(alpha, beta), and names the workload shapes.  Both the CPU oracle and the
HIP library receive exactly the tensors produced here.

The elastic rule is the per-head span law of the method (paper, Sec. 3.2,
Eq. 2: span = alpha + beta * N).  Sampling draws alpha from
{256, 512, 1024, 2048} and beta from {0, .25, .5, .75} per KV head, then
multiplies both by one common factor f so that the (continuous, unrounded)
mean of min(N, f * (alpha + beta * N)) over heads equals the target mean
window (N/2 or N/4).  The integer windows themselves are produced by the
plan (library) or the oracle's plan, never here.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

ALPHA_CHOICES = (256.0, 512.0, 1024.0, 2048.0)
BETA_CHOICES = (0.0, 0.25, 0.5, 0.75)


def randn(shape: Sequence[int], seed: int, dtype=None, device="cpu"):
    """N(0, 1) tensor from a seeded torch generator, rounded to ``dtype``.

    Draws in float32 with a generator on ``device`` and rounds to ``dtype``
    (round-to-nearest-even for bfloat16).  The same (shape, seed, device)
    always gives the same values.
    """
    import torch

    dtype = dtype or torch.float32
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    x = torch.randn(tuple(int(s) for s in shape), generator=gen, device=device,
                    dtype=torch.float32)
    return x.to(dtype)


def sample_rules(seed: int, num_kv_heads: int, n: int,
                 target_mean: float) -> Tuple[np.ndarray, np.ndarray]:
    """Seeded per-KV-head (alpha, beta), rescaled to a target mean window.

    Returns float64 arrays (alpha', beta') = (f * alpha, f * beta) where f is
    found by bisection so that mean_g min(n, f * (alpha_g + beta_g * n)) is
    ``target_mean`` (continuous, before the plan floors and clips).
    """
    rng = np.random.default_rng(seed)
    alpha = rng.choice(np.array(ALPHA_CHOICES), size=num_kv_heads)
    beta = rng.choice(np.array(BETA_CHOICES), size=num_kv_heads)
    raw = alpha + beta * float(n)

    def mean_at(f: float) -> float:
        return float(np.minimum(float(n), f * raw).mean())

    lo, hi = 0.0, 1.0
    while mean_at(hi) < target_mean and hi < 1e9:
        hi *= 2.0
    if mean_at(hi) < target_mean:
        raise ValueError("target mean window not reachable")
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if mean_at(mid) < target_mean:
            lo = mid
        else:
            hi = mid
    f = hi
    return (f * alpha).astype(np.float64), (f * beta).astype(np.float64)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic attention-layer workload."""

    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    num_sink: int
    n: int                      # length N at which the elastic rule is evaluated
    dtype: str                  # "f32" or "bf16"
    prefill_batch: int
    decode_batch: int
    decode_steps: int
    seed: int
    alpha: Tuple[float, ...]
    beta: Tuple[float, ...]

    def torch_dtype(self):
        import torch
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


def _elastic(name, hq, hkv, n, mean_frac, prefill_batch, decode_batch, steps, seed,
             d=128, sink=64, dtype="bf16") -> Workload:
    a, b = sample_rules(seed, hkv, n, mean_frac * n)
    return Workload(name, hq, hkv, d, sink, n, dtype, prefill_batch, decode_batch,
                    steps, seed, tuple(float(x) for x in a), tuple(float(x) for x in b))


def workloads() -> List[Workload]:
    """The workload shapes (index 0 is the small oracle-checkable case; index 5 is
    the long-context batch-1 decode case)."""
    small = Workload("small-mha4-d64-n512-f32", 4, 4, 64, 4, 512, "f32", 1, 1, 16, 0,
                     (64.0, 128.0, 256.0, 512.0), (0.0, 0.0, 0.0, 0.0))
    return [
        small,
        _elastic("vicuna7b-prefill-n4096", 32, 32, 4096, 0.5, 1, 1, 0, 1),
        _elastic("vicuna7b-decode-b32-ctx8192", 32, 32, 8192, 0.5, 32, 32, 256, 2),
        _elastic("llama3-8b-gqa-n16384", 32, 8, 16384, 0.5, 1, 16, 256, 3),
        _elastic("llama3-70b-gqa-n32768", 64, 8, 32768, 0.25, 1, 8, 512, 4),
        _elastic("vicuna7b-decode-b1-ctx131072", 32, 32, 131072, 0.5, 1, 1, 512, 5),
    ]


def workload(name_or_index) -> Workload:
    ws = workloads()
    if isinstance(name_or_index, int):
        return ws[name_or_index]
    for w in ws:
        if w.name == name_or_index:
            return w
    raise KeyError(name_or_index)
