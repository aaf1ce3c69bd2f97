"""Plain fp64 CPU oracle for Mixture-of-Attention-Spans (MoA) attention.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the package's smoke check and
the benchmark's CPU-baseline leg may import this module.  It shares no code
with the HIP library and the library never calls it.

What it computes, step by step, in the paper's terms:

* Elastic rule (Sec. 3.2, Eq. 2): the sliding-window length of KV head g at
  input length N is alpha_g + beta_g * N.  Reading adopted: the rule gives the
  band width; the always-visible initial (sink) tokens are added on top; the
  value is floored and clipped to [1, N] (Appendix "Main Setup" clips spans to
  the input length; 1 instead of 0 keeps the diagonal so no row is empty).
* Attention span / mask (Sec. 3.2 and Appendix "Attention Span"): a query at
  position i sees key j iff j <= i (causal) and (j < s, the sink prefix, or
  i - j < w_g, the diagonal band).  The band includes the query itself.
* Attention (Sec. 2.1, Eq. 1): S = Q K^T (times the usual 1/sqrt(D)),
  A = softmax(S + M) with M = 0 where visible and -inf elsewhere, O = A V.
  Each head applies its own mask independently (Appendix "Application of
  Attention Masks"); under grouped queries, query head h uses KV head
  h // (H_q / H_kv).
* Decode (Sec. 2.1): the new token at position t is row t of the same
  computation over the full history 0..t.
* Static KV cache (Appendix "Efficiency Experiment Setup" and "Memory and
  Throughput Breakdown"): each KV head keeps at most s + w_g entries; once
  full, the newest token replaces the oldest non-sink entry in place.

Two variants of the paper's own kernel setting (Appendix "Main Setup" and
"Efficiency Experiment Setup"), selected by arguments:

* span_includes_sinks: the rule gives the whole span S = alpha + beta * N,
  sinks included (Sec. 3.2: span = sliding window + initially unmasked
  tokens).  S is floored and clipped to [0, N]; the band is w = S - s, at
  least 1.
* block: the band is counted in blocks of `block` tokens (the paper's
  prefill uses 64-token blocks): query i sees key j iff j <= i and (j < s or
  i // block - j // block < ceil(w / block)).  Decode keeps the token-exact
  band, as the paper's cache replaces the oldest token one at a time.

All floating point work is float64 on the exact stored input values.

Parity status: every function here is pinned by the CPU tests (brute force,
closed forms, library reductions, invariants); no function is unpinned.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np


# ----------------------------------------------------------------------------
# Elastic rule -> per-head window table (Sec. 3.2, Eq. 2; Appendix clipping)
# ----------------------------------------------------------------------------

def window_ref(alpha: float, beta: float, n: int, num_sink: int = 0,
               span_includes_sinks: bool = False) -> int:
    """Band width of one head, from the rule alpha + beta * N in IEEE double.

    Default: w = min(max(floor(alpha + beta * N), 1), N).
    span_includes_sinks: S = min(max(floor(alpha + beta * N), 0), N) and
    w = max(S - num_sink, 1).
    """
    x = float(alpha) + float(beta) * float(n)   # Python floats: no fused multiply-add
    if span_includes_sinks:
        if not (x >= 0.0):
            span = 0
        elif x >= float(n):
            span = int(n)
        else:
            span = int(math.floor(x))
        return max(span - int(num_sink), 1)
    if not (x >= 1.0):
        return 1
    if x >= float(n):
        return int(n)
    return int(math.floor(x))


def plan_ref(alpha: Sequence[float], beta: Sequence[float], n: int,
             num_sink: int, span_includes_sinks: bool = False) -> Dict[str, np.ndarray]:
    """Per-KV-head window, cache capacity (sinks + window) and cache row offset."""
    window = np.array([window_ref(a, b, n, num_sink, span_includes_sinks) for a, b in zip(alpha, beta)],
                      dtype=np.int32)
    capacity = (window.astype(np.int64) + int(num_sink)).astype(np.int32)
    offset = np.zeros(len(window) + 1, dtype=np.int64)
    offset[1:] = np.cumsum(capacity.astype(np.int64))
    return {"window": window, "capacity": capacity, "offset": offset}


# ----------------------------------------------------------------------------
# Mask (Sec. 3.2 span definition; Appendix "Attention Mask")
# ----------------------------------------------------------------------------

def band_blocks(w: int, block: int) -> int:
    """Band length in blocks: ceil(w / block)."""
    return -(-int(w) // int(block))


def visible(i: int, j: int, w: int, s: int, block: int = 0) -> bool:
    """Key j is visible to query i: causal, and in the sink prefix or the band
    (counted in tokens, or in blocks of `block` tokens when block > 0)."""
    if block:
        return j <= i and (j < s or i // block - j // block < band_blocks(w, block))
    return j <= i and (j < s or i - j < w)


def visible_mask(n_q: int, n_k: int, w: int, s: int, q_start: int = 0, block: int = 0) -> np.ndarray:
    """Boolean [n_q, n_k] mask for query positions q_start.. and keys 0..n_k-1."""
    i = np.arange(q_start, q_start + n_q, dtype=np.int64)[:, None]
    j = np.arange(n_k, dtype=np.int64)[None, :]
    if block:
        band = (i // block - j // block) < band_blocks(w, block)
    else:
        band = (i - j) < w
    return (j <= i) & ((j < s) | band)


# ----------------------------------------------------------------------------
# Attention (Sec. 2.1, Eq. 1, with the per-head MoA mask)
# ----------------------------------------------------------------------------

def _scale(head_dim: int, scale: Optional[float]) -> float:
    return 1.0 / math.sqrt(head_dim) if not scale else float(scale)


def _as64(x) -> np.ndarray:
    """Exact float64 copy of a numpy array or torch tensor (bf16 upcasts exactly)."""
    if hasattr(x, "detach"):
        import torch
        x = x.detach().to("cpu", torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


def masked_softmax_rows(s_rows: np.ndarray, mask_rows: np.ndarray) -> np.ndarray:
    """A = softmax(S + M) row by row, M = 0 on visible entries and -inf elsewhere."""
    m = np.where(mask_rows, 0.0, -np.inf)
    z = s_rows + m
    zmax = z.max(axis=-1, keepdims=True)
    e = np.exp(z - zmax)
    return e / e.sum(axis=-1, keepdims=True)


def attention_ref(q, k, v, window: Sequence[int], num_sink: int,
                  scale: Optional[float] = None, row_block: int = 1024, block: int = 0) -> np.ndarray:
    """Prefill output O [B, n, H_q, D] in float64.

    q: [B, n, H_q, D]; k, v: [B, n, H_kv, D]; window: [H_kv] integer windows.
    Rows are processed in blocks of ``row_block`` to bound memory; each block
    is the plain masked product S -> A -> O of Eq. 1.
    """
    q, k, v = _as64(q), _as64(k), _as64(v)
    bsz, n, hq, d = q.shape
    hkv = k.shape[2]
    group = hq // hkv
    sc = _scale(d, scale)
    out = np.zeros((bsz, n, hq, d), dtype=np.float64)
    for b in range(bsz):
        for h in range(hq):
            g = h // group
            kg = k[b, :, g, :]
            vg = v[b, :, g, :]
            for r0 in range(0, n, row_block):
                r1 = min(n, r0 + row_block)
                s_rows = (q[b, r0:r1, h, :] @ kg[:r1].T) * sc          # S = Q K^T
                mask = visible_mask(r1 - r0, r1, int(window[g]), num_sink, r0, block)
                a = masked_softmax_rows(s_rows, mask)                  # softmax(S + M)
                out[b, r0:r1, h, :] = a @ vg[:r1]                      # O = A V
    return out


def attention_rows_ref(q, k, v, window: Sequence[int], num_sink: int, b: int, h: int,
                       rows: Sequence[int], scale: Optional[float] = None, block: int = 0) -> np.ndarray:
    """Selected prefill output rows O[b, rows, h, :] in float64 ([len(rows), D]).

    Each row i is softmax over its visible set J_i only, so large workloads can
    be checked on sampled rows.
    """
    d = q.shape[-1]
    hq, hkv = q.shape[2], k.shape[2]
    g = h // (hq // hkv)
    w = int(window[g])
    sc = _scale(d, scale)
    out = np.zeros((len(rows), d), dtype=np.float64)
    for r, i in enumerate(rows):
        i = int(i)
        js = visible_set(i, w, num_sink, block)
        qi = _as64(q[b, i, h, :])
        kj = _as64(k[b, js, g, :])
        vj = _as64(v[b, js, g, :])
        srow = (kj @ qi) * sc
        e = np.exp(srow - srow.max())
        out[r] = (e / e.sum()) @ vj
    return out


def visible_set(i: int, w: int, s: int, block: int = 0) -> np.ndarray:
    """J_i = {j <= i : j < s or j in the band of i} as sorted int64 indices.

    The band starts at i - w + 1 (tokens) or at the first token of block
    i // block - ceil(w / block) + 1 (blocks)."""
    sinks = np.arange(0, min(s, i + 1), dtype=np.int64)
    if block:
        start = (i // block - band_blocks(w, block) + 1) * block
    else:
        start = i - w + 1
    band = np.arange(max(0, start), i + 1, dtype=np.int64)
    return np.union1d(sinks, band)


def probabilities_ref(q, k, window: Sequence[int], num_sink: int, b: int, h: int,
                      scale: Optional[float] = None, block: int = 0) -> np.ndarray:
    """Full attention-probability matrix A [n, n] of one (batch, query head)."""
    q, k = _as64(q), _as64(k)
    n, d = q.shape[1], q.shape[3]
    g = h // (q.shape[2] // k.shape[2])
    s_all = (q[b, :, h, :] @ k[b, :, g, :].T) * _scale(d, scale)
    return masked_softmax_rows(s_all, visible_mask(n, n, int(window[g]), num_sink, 0, block))


def decode_ref(q_t, k_hist, v_hist, window: Sequence[int], num_sink: int,
               scale: Optional[float] = None) -> np.ndarray:
    """Decode output [B, H_q, D] for the newest token t = len(history) - 1.

    q_t: [B, H_q, D]; k_hist, v_hist: [B, t + 1, H_kv, D] (the full history,
    including the new token).  This is row t of the prefill computation.
    """
    q_t, k_hist, v_hist = _as64(q_t), _as64(k_hist), _as64(v_hist)
    bsz, hq, d = q_t.shape
    t = k_hist.shape[1] - 1
    hkv = k_hist.shape[2]
    group = hq // hkv
    sc = _scale(d, scale)
    out = np.zeros((bsz, hq, d), dtype=np.float64)
    for b in range(bsz):
        for h in range(hq):
            g = h // group
            js = visible_set(t, int(window[g]), num_sink)
            srow = (k_hist[b, js, g, :] @ q_t[b, h, :]) * sc
            e = np.exp(srow - srow.max())
            out[b, h] = (e / e.sum()) @ v_hist[b, js, g, :]
    return out


# ----------------------------------------------------------------------------
# Static per-head KV cache with in-place replacement (Appendix, efficiency setup)
# ----------------------------------------------------------------------------

class CacheModel:
    """Sequential simulation of one KV head's static cache.

    Slots are filled in arrival order until the cache holds s + w tokens.
    After that each new token overwrites, in place, the slot of the oldest
    non-sink token; sink tokens (positions < s) are never replaced.
    ``slots[k]`` is the position held in slot k, or -1.
    """

    def __init__(self, window: int, num_sink: int):
        self.w = int(window)
        self.s = int(num_sink)
        self.capacity = self.w + self.s
        self.slots: List[int] = [-1] * self.capacity
        self.next_pos = 0

    def append(self, p: int) -> int:
        if p != self.next_pos:
            raise ValueError("appends must be contiguous")
        self.next_pos += 1
        free = [k for k, x in enumerate(self.slots) if x < 0]
        if free:
            slot = free[0]
        else:
            non_sink = [(x, k) for k, x in enumerate(self.slots) if x >= self.s]
            slot = min(non_sink)[1]              # oldest non-sink entry
        self.slots[slot] = p
        return slot

    def positions(self) -> List[int]:
        return sorted(x for x in self.slots if x >= 0)


def cache_ref(window: Sequence[int], num_sink: int, total: int) -> np.ndarray:
    """Expected slot -> position table [sum_g (s + w_g)] after appending 0..total-1."""
    table: List[int] = []
    for w in window:
        cm = CacheModel(int(w), num_sink)
        for p in range(total):
            cm.append(p)
        table.extend(cm.slots)
    return np.array(table, dtype=np.int32)


def cache_contents_ref(k_hist, v_hist, window: Sequence[int], num_sink: int):
    """Expected (pos, K cache, V cache) for a batch after appending the history.

    k_hist, v_hist: [B, T, H_kv, D] (any dtype; values are copied bit for bit).
    Returns pos [B, sum C] int32 and K/V [B, sum C, D] in the input dtype,
    empty slots zero.
    """
    import torch

    bsz, total, hkv, d = k_hist.shape
    table = cache_ref(window, num_sink, total)
    caps = [int(w) + num_sink for w in window]
    kc = torch.zeros((bsz, len(table), d), dtype=k_hist.dtype)
    vc = torch.zeros((bsz, len(table), d), dtype=v_hist.dtype)
    row = 0
    for g, c in enumerate(caps):
        for slot in range(c):
            p = int(table[row + slot])
            if p >= 0:
                kc[:, row + slot, :] = k_hist[:, p, g, :]
                vc[:, row + slot, :] = v_hist[:, p, g, :]
        row += c
    pos = np.broadcast_to(table, (bsz, len(table))).copy()
    return pos, kc, vc
