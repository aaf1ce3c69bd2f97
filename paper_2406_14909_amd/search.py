"""Rule search on the host: the candidate-rule grid and the single-length
selection (paper Sec. 3.4 "Automatic Optimization"; Appendix "Optimizing at
Single Length" and "Main Setup").

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
    [H, R]) kept fractions.  Returns (rules [H] ints, mean loss), or
    (None, inf) when no assignment meets the budget."""
    from scipy.optimize import Bounds, LinearConstraint, milp
    from scipy.sparse import csr_matrix

    dl = np.asarray(dl, dtype=np.float64)
    h, r = dl.shape
    dens = np.broadcast_to(np.asarray(density, dtype=np.float64), (h, r))
    nx = h * r
    use_layers = bool(max_rules_per_layer) and layer_of is not None
    layers = sorted(set(layer_of)) if use_layers else []
    ny = len(layers) * r
    c = np.concatenate([dl.reshape(-1) / h, np.zeros(ny)])

    rows = np.repeat(np.arange(h), r)
    one_per_head = csr_matrix((np.ones(nx), (rows, np.arange(nx))), shape=(h, nx + ny))
    budget_row = csr_matrix(np.concatenate([dens.reshape(-1) / h, np.zeros(ny)])[None, :])
    cons = [LinearConstraint(one_per_head, 1.0, 1.0), LinearConstraint(budget_row, -np.inf, float(budget))]
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
