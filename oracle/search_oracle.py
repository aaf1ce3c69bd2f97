"""Plain fp64 CPU oracle for the MoA rule search (rule-loss table and selection).

TEST INFRASTRUCTURE ONLY.  Only the test-suite may import this module.  It
shares no code with the library.

What it computes, in the paper's terms:

* Candidate rules (Appendix "Main Setup"): 6 values of alpha uniformly
  spaced over [-2048, 8192] and 9 values of beta uniformly spaced over
  [0, 1], 54 (alpha, beta) pairs per head.
* Rule loss (Sec. 3.3, Eq. 4): the accuracy loss of giving head h rule r at
  length N is the sum of the head's average attention influence over the
  positions the rule masks, Delta L_{h,r} = sum_ij M_{r,ij} E_bar_{h,ij}.
  E_bar is block-averaged, so every token (i, j) of a block carries the
  block's value.  M_r marks the causal pairs (j <= i) that the rule's mask
  hides: the rule's window (and sinks, block band) from the plan's reading.
* Density of a rule at length N (Sec. 4 "Setups": the average in-memory
  KV-cache length divided by the sequence length during decoding): the
  number of tokens the rule's cache holds once N tokens have been seen,
  divided by N.  The cache then holds exactly the keys the newest token sees
  (the token-exact visible set of query N - 1: the sinks and the last w
  tokens), so the density is |J_{N-1}| / N.  The block band changes only the
  prefill mask, not the cache, so it does not enter the density.
* Single-length selection (Appendix "Optimizing at Single Length"): choose
  one rule per head minimising the mean loss subject to the mean density
  not exceeding the budget; optionally at most K distinct rules per layer.
  Solved here by enumerating every assignment (tiny head counts only).
* Multi-length search (Sec. 3.4, Appendix "Optimizing at Multiple Lengths"):
  the Pareto front of the per-length mean losses over all assignments that
  meet every length's density budget, by enumeration.

Parity status: pinned by the CPU tests (a hand-worked masked sum and
density, the masked-pair count under a unit profile, the density against a
simulated cache, hand-worked selection and Pareto examples, enumeration
checked against a library MILP solver); nothing is unpinned.
"""
from __future__ import annotations

import itertools
from typing import Optional, Sequence

import numpy as np

from .moa_oracle import visible_mask, visible_set, window_ref


def candidate_rules(n_alpha: int = 6, n_beta: int = 9):
    """The (alpha, beta) grid: alpha uniform over [-2048, 8192], beta over [0, 1]."""
    alphas = np.linspace(-2048.0, 8192.0, n_alpha)
    betas = np.linspace(0.0, 1.0, n_beta)
    pairs = [(float(a), float(b)) for a in alphas for b in betas]
    return np.array([p[0] for p in pairs]), np.array([p[1] for p in pairs])


def masked_pairs(n: int, w: int, s: int, block: int = 0) -> np.ndarray:
    """Boolean [n, n]: causal pairs hidden by the mask of window w, sinks s."""
    causal = np.tril(np.ones((n, n), dtype=bool))
    return causal & ~visible_mask(n, n, w, s, 0, block)


def rule_loss_ref(ebar: np.ndarray, n: int, num_sink: int, alpha: Sequence[float], beta: Sequence[float],
                  span_includes_sinks: bool = False, block: int = 0, profile_block: int = 64):
    """(Delta L [H, R], density [R]) of every rule for every head at length n.

    ebar: [H, nb, nb] block-averaged influence (profile_block x profile_block
    blocks); each token pair takes its block's value (Eq. 4 summed token by
    token).  density[r] = |cache of rule r after n tokens| / n (Sec. 4
    "Setups"), see density_ref."""
    ebar = np.asarray(ebar, dtype=np.float64)
    h = ebar.shape[0]
    tok = np.repeat(np.repeat(ebar, profile_block, axis=1), profile_block, axis=2)[:, :n, :n]
    dl = np.zeros((h, len(alpha)), dtype=np.float64)
    dens = np.zeros(len(alpha), dtype=np.float64)
    for r, (a, b) in enumerate(zip(alpha, beta)):
        w = window_ref(a, b, n, num_sink, span_includes_sinks)
        m = masked_pairs(n, w, num_sink, block)
        dl[:, r] = (tok * m[None]).sum(axis=(1, 2))
        dens[r] = density_ref(n, w, num_sink)
    return dl, dens


def density_ref(n: int, w: int, s: int) -> float:
    """Density of a head with window w and s sinks at sequence length n
    (Sec. 4 "Setups": in-memory KV-cache length / sequence length, during
    decoding).  After n tokens the cache holds the token-exact visible set of
    the newest token, J_{n-1} (the sinks and the last w tokens)."""
    return len(visible_set(n - 1, w, s)) / n


def select_bruteforce(dl: np.ndarray, density: np.ndarray, budget: float,
                      layer_of: Optional[Sequence[int]] = None, max_rules_per_layer: int = 0):
    """Exhaustive single-length selection: argmin mean_h dl[h, r_h] subject to
    mean_h density[r_h] <= budget (and at most max_rules_per_layer distinct
    rules among the heads of a layer when given).  Returns (rules, loss) or
    (None, inf) when no assignment fits."""
    h, r = dl.shape
    best, best_rules = np.inf, None
    for combo in itertools.product(range(r), repeat=h):
        if np.mean(density[list(combo)]) > budget + 1e-12:
            continue
        if max_rules_per_layer and layer_of is not None:
            per_layer = {}
            for hh, rr in enumerate(combo):
                per_layer.setdefault(layer_of[hh], set()).add(rr)
            if any(len(v) > max_rules_per_layer for v in per_layer.values()):
                continue
        loss = float(np.mean([dl[hh, rr] for hh, rr in enumerate(combo)]))
        if loss < best:
            best, best_rules = loss, list(combo)
    return best_rules, best


def dominates(p, q) -> bool:
    """p is no worse than q at every length and better at one."""
    p, q = np.asarray(p), np.asarray(q)
    return bool(np.all(p <= q) and np.any(p < q))


def pareto_front_bruteforce(dls, densities, budgets):
    """All non-dominated per-length loss vectors over the feasible assignments
    (each a tuple of mean losses, one per length), by enumeration."""
    dls = [np.asarray(d, dtype=np.float64) for d in dls]
    h, r = dls[0].shape
    points = set()
    for combo in itertools.product(range(r), repeat=h):
        ok = all(np.mean(np.asarray(densities[i])[list(combo)]) <= budgets[i] + 1e-12
                 for i in range(len(dls)) if budgets[i] is not None)
        if ok:
            points.add(tuple(float(np.mean([d[hh, rr] for hh, rr in enumerate(combo)])) for d in dls))
    return sorted(p for p in points if not any(dominates(q, p) for q in points))

