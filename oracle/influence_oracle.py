"""Plain fp64 CPU oracle for MoA attention-influence profiling.

TEST INFRASTRUCTURE ONLY.  Only the test-suite and the benchmark's CPU
baseline may import this module.  It shares no code with the HIP library.

What it computes, in the paper's terms (Sec. 3.3 "Attention Influence
Profiling", Eq. 3; Appendix "Derivation of Attention Influence"):

* Attention influence: the first-order estimate of the change in the loss L
  when attention value A_ij is masked and the rest of row i renormalised.
  Masking sets A_ij to 0 and scales every other entry of the row by
  1 / (1 - A_ij); summing dL/dA times those changes gives
      E_ij = -A_ij / (1 - A_ij) * (G_ij - sum_n G_in A_in),   G = dL/dA.
  The derivation's last line carries the minus sign; the matrix form printed
  after it omits it.  The minus sign is taken (it is the one the first-order
  expansion gives, and the pins below check it against the exact change).
  E_ij is 0 where A_ij = 0 (nothing to mask) and where A_ij = 1 (the row's
  only weight: masking it leaves nothing to renormalise).
* Dense causal attention of the profiled model: A = softmax(scale * Q K^T +
  causal mask) per query head, O = A V.  For a loss that reaches A through O,
  dL/dA = dO V^T (chain rule through O = A V).
* Block granularity (Appendix "Main Setup"): the influence is averaged over
  64 x 64 blocks (all entries of the block that exist, zeros above the
  diagonal included) and over the calibration items.

All arithmetic is float64 on the exact stored input values.

Parity status: every function is pinned by the CPU tests (an exact masking
identity for losses linear in A, torch autograd for dL/dA, a hand-worked
row, torch pooling for the block average, planted mistakes).
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np

from .moa_oracle import _as64


def influence_ref(a: np.ndarray, g: np.ndarray) -> np.ndarray:
    """E = -A / (1 - A) * (G - rowsum(G * A)) elementwise over the last two
    axes (rows i, columns j); 0 where A is 0 or 1."""
    a = np.asarray(a, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    d = (g * a).sum(axis=-1, keepdims=True)          # sum_n G_in A_in, per row
    inside = (a > 0.0) & (a < 1.0)
    ratio = np.divide(a, 1.0 - a, out=np.zeros_like(a), where=inside)
    return np.where(inside, -ratio * (g - d), 0.0)


def causal_probabilities(q, k, scale: Optional[float] = None) -> np.ndarray:
    """A [B, H_q, n, n] = softmax(scale * Q K^T) under the causal mask."""
    q, k = _as64(q), _as64(k)
    bsz, n, hq, d = q.shape
    group = hq // k.shape[2]
    sc = 1.0 / math.sqrt(d) if not scale else float(scale)
    causal = np.tril(np.ones((n, n), dtype=bool))
    out = np.zeros((bsz, hq, n, n), dtype=np.float64)
    for b in range(bsz):
        for h in range(hq):
            s = (q[b, :, h, :] @ k[b, :, h // group, :].T) * sc
            z = np.where(causal, s, -np.inf)
            e = np.exp(z - z.max(axis=-1, keepdims=True))
            out[b, h] = e / e.sum(axis=-1, keepdims=True)
    return out


def grad_wrt_probabilities(v, dout, num_q_heads: int) -> np.ndarray:
    """dL/dA [B, H_q, n, n] = dO V^T for a loss that reaches A through O = A V."""
    v, dout = _as64(v), _as64(dout)
    bsz, n, hkv, _ = v.shape
    group = num_q_heads // hkv
    out = np.zeros((bsz, num_q_heads, n, n), dtype=np.float64)
    for b in range(bsz):
        for h in range(num_q_heads):
            out[b, h] = dout[b, :, h, :] @ v[b, :, h // group, :].T
    return out


def block_average_ref(e: np.ndarray, block: int = 64) -> np.ndarray:
    """Mean of E [B, H, n, n] over the items and over each block x block tile
    (a tile at the edge averages over the entries that exist): [H, nb, nb]."""
    e = np.asarray(e, dtype=np.float64)
    bsz, h, n, _ = e.shape
    nb = -(-n // block)
    out = np.zeros((h, nb, nb), dtype=np.float64)
    for bi in range(nb):
        for bj in range(nb):
            tile = e[:, :, bi * block:(bi + 1) * block, bj * block:(bj + 1) * block]
            out[:, bi, bj] = tile.sum(axis=(0, 2, 3)) / (bsz * tile.shape[2] * tile.shape[3])
    return out


def influence_profile_ref(q, k, v, dout, scale: Optional[float] = None, block: int = 64) -> np.ndarray:
    """Block-averaged attention influence [H_q, nb, nb] of dense causal
    attention, averaged over the batch of calibration items."""
    a = causal_probabilities(q, k, scale)
    g = grad_wrt_probabilities(v, dout, a.shape[1])
    return block_average_ref(influence_ref(a, g), block)


def influence_rows_ref(q, k, v, dout, b: int, h: int, rows, scale: Optional[float] = None) -> np.ndarray:
    """E[b, h, rows, :] ([len(rows), n]) of dense causal attention, each row from
    its own softmax and its own dL/dA row, so long inputs can be checked on
    sampled row blocks."""
    d = q.shape[-1]
    n = q.shape[1]
    group = q.shape[2] // k.shape[2]
    g = h // group
    sc = 1.0 / math.sqrt(d) if not scale else float(scale)
    kg, vg = _as64(k[b, :, g, :]), _as64(v[b, :, g, :])
    out = np.zeros((len(rows), n), dtype=np.float64)
    for r, i in enumerate(rows):
        i = int(i)
        s = (kg[: i + 1] @ _as64(q[b, i, h, :])) * sc
        e = np.exp(s - s.max())
        a_row = np.zeros(n)
        a_row[: i + 1] = e / e.sum()
        g_row = vg @ _as64(dout[b, i, h, :])
        out[r] = influence_ref(a_row[None, :], g_row[None, :])[0]
    return out

