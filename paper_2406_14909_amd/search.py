"""Rule search on the host: the candidate-rule grid, the single-length
selection and the multi-length Pareto search (paper Sec. 3.4 "Automatic
Optimization"; Appendix "Optimizing at Single Length", "Optimizing at
Multiple Lengths" and "Main Setup").

The GPU produces the profile (moa_influence) and the loss table of every
candidate rule for every head (moa_rule_loss); choosing one rule per head is a
small mixed-integer program over that table.  The paper solves it with Gurobi;
here it goes to the HiGHS solver that scipy ships, with the relative gap set to
zero so the result is the exact optimum:

    minimise  (1/H) sum_h sum_r dl[h, r] x[h, r]
    s.t.      sum_r x[h, r] = 1                      for every head h
              (1/H) sum_h sum_r density[r] x[h, r] <= budget
              x[h, r] <= y[l, r], sum_r y[l, r] <= K  (optional: at most K
                                                      distinct rules per layer l)
              x, y binary.
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np


def candidate_rules(n_alpha: int = 6, n_beta: int = 9) -> Tuple[np.ndarray, np.ndarray]:
    """(alpha, beta) of the candidate grid: n_alpha values spaced uniformly over
    [-2048, 8192] times n_beta values over [0, 1] (54 rules by default)."""
    alphas = -2048.0 + (8192.0 + 2048.0) * np.arange(n_alpha) / (n_alpha - 1)
    betas = np.arange(n_beta) / (n_beta - 1)
    return np.repeat(alphas, n_beta), np.tile(betas, n_alpha)


def select_rules(dl, density, budget: float, layer_of: Optional[Sequence[int]] = None,
                 max_rules_per_layer: int = 0, time_limit: float = 60.0):
    """Exact single-length selection.  dl: [H, R] losses; density: [R] (or
    [H, R]) rule densities (in-memory KV-cache length over sequence length,
    paper Sec. 4 "Setups", as moa_rule_loss returns them).  Returns
    (rules [H] ints, mean loss), or
    (None, inf) when no assignment meets the budget."""
    return _solve(dl, [(density, -np.inf, budget)], layer_of, max_rules_per_layer, time_limit)


def _solve(dl, mean_bounds, layer_of=None, max_rules_per_layer: int = 0, time_limit: float = 60.0):
    """min mean_h dl[h, r_h] over one rule per head, subject to
    lo <= mean_h table[h, r_h] <= hi for every (table, lo, hi) in mean_bounds
    (a table is [R] or [H, R])."""
    from scipy.optimize import Bounds, LinearConstraint, milp
    from scipy.sparse import csr_matrix

    dl = np.asarray(dl, dtype=np.float64)
    h, r = dl.shape
    nx = h * r
    use_layers = bool(max_rules_per_layer) and layer_of is not None
    layers = sorted(set(layer_of)) if use_layers else []
    ny = len(layers) * r
    c = np.concatenate([dl.reshape(-1) / h, np.zeros(ny)])

    rows = np.repeat(np.arange(h), r)
    one_per_head = csr_matrix((np.ones(nx), (rows, np.arange(nx))), shape=(h, nx + ny))
    cons = [LinearConstraint(one_per_head, 1.0, 1.0)]
    for table, lo, hi in mean_bounds:
        t = np.broadcast_to(np.asarray(table, dtype=np.float64), (h, r))
        row = csr_matrix(np.concatenate([t.reshape(-1) / h, np.zeros(ny)])[None, :])
        cons.append(LinearConstraint(row, float(lo), float(hi)))
    if use_layers:
        lidx = {l: i for i, l in enumerate(layers)}
        # x[h, r] - y[layer(h), r] <= 0
        xi = np.arange(nx)
        yi = np.array([nx + lidx[layer_of[hh]] * r + rr for hh in range(h) for rr in range(r)])
        link = csr_matrix((np.concatenate([np.ones(nx), -np.ones(nx)]),
                           (np.concatenate([xi, xi]), np.concatenate([xi, yi]))), shape=(nx, nx + ny))
        cons.append(LinearConstraint(link, -np.inf, 0.0))
        cap = csr_matrix((np.ones(ny), (np.repeat(np.arange(len(layers)), r), nx + np.arange(ny))),
                         shape=(len(layers), nx + ny))
        cons.append(LinearConstraint(cap, -np.inf, float(max_rules_per_layer)))
    res = milp(c, constraints=cons, integrality=np.ones(nx + ny), bounds=Bounds(0.0, 1.0),
               options={"mip_rel_gap": 0.0, "time_limit": time_limit})
    if res.x is None or res.status not in (0,):
        return None, np.inf
    x = np.round(res.x[:nx]).reshape(h, r)
    rules = [int(np.argmax(x[hh])) for hh in range(h)]
    loss = float(np.mean([dl[hh, rr] for hh, rr in enumerate(rules)]))
    return rules, loss


def pareto_filter(points):
    """Indices of the points (loss vectors) that no other point dominates
    (no worse at every length, better at one); duplicates keep the first."""
    pts = np.asarray(points, dtype=np.float64)
    keep = []
    for i, p in enumerate(pts):
        dominated = any(np.all(q <= p) and np.any(q < p) for j, q in enumerate(pts) if j != i)
        duplicate = any(np.array_equal(pts[k], p) for k in keep)
        if not dominated and not duplicate:
            keep.append(i)
    return keep


def select_multi_length(dls, densities, budgets, intervals: int = 5, val_dl=None,
                        layer_of: Optional[Sequence[int]] = None, max_rules_per_layer: int = 0,
                        time_limit: float = 60.0):
    """Pareto search over several profiled lengths by the epsilon-constraint
    method (paper Appendix "Optimizing at Multiple Lengths").

    dls: per profiled length, the [H, R] loss table; densities: per length,
    the [R] rule densities; budgets: per length, the mean-density budget (None:
    no constraint at that length).  First each length's loss is minimised
    alone, recording the other lengths' losses, which gives each length a loss
    range; then, for each length, its loss is minimised again with every other
    length's loss held inside one of `intervals` equal parts of its range, for
    every combination of parts.  Returns (front, best): front is a list of
    (rules, loss vector) that no other found solution dominates; best is the
    member with the least loss on val_dl (an [H, R] table at a length not
    profiled) or None when val_dl is not given."""
    dls = [np.asarray(d, dtype=np.float64) for d in dls]
    k = len(dls)
    h = dls[0].shape[0]
    dens_bounds = [(densities[i], -np.inf, budgets[i]) for i in range(k) if budgets[i] is not None]

    def losses(rules):
        return np.array([float(np.mean(d[np.arange(h), rules])) for d in dls])

    found = []
    for i in range(k):
        rules, _ = _solve(dls[i], dens_bounds, layer_of, max_rules_per_layer, time_limit)
        if rules is not None:
            found.append((rules, losses(rules)))
    if not found:
        return [], None
    pts = np.array([f[1] for f in found])
    lo, hi = pts.min(axis=0), pts.max(axis=0)
    import itertools
    for i in range(k):
        others = [j for j in range(k) if j != i]
        for parts in itertools.product(range(intervals), repeat=len(others)):
            bounds = list(dens_bounds)
            for j, part in zip(others, parts):
                width = (hi[j] - lo[j]) / intervals
                a = lo[j] + part * width
                b = hi[j] if part == intervals - 1 else lo[j] + (part + 1) * width
                bounds.append((dls[j], a - 1e-12, b + 1e-12))
            rules, _ = _solve(dls[i], bounds, layer_of, max_rules_per_layer, time_limit)
            if rules is not None:
                found.append((rules, losses(rules)))
    keep = pareto_filter([f[1] for f in found])
    front = [found[i] for i in keep]
    best = None
    if val_dl is not None:
        val = np.asarray(val_dl, dtype=np.float64)
        best = min(front, key=lambda f: float(np.mean(val[np.arange(h), f[0]])))
    return front, best

