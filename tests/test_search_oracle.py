"""Pins of the rule-search oracle (paper Sec. 3.3, Eq. 4; Appendix "Main
Setup" and "Optimizing at Single Length")."""
import numpy as np
import pytest
from scipy.optimize import Bounds, LinearConstraint, milp

from conftest import read_golden
from oracle import search_oracle as so


def test_golden_rule_loss():
    ((ws, dl, dens),) = read_golden("rule_loss_n8.txt")
    w, s = (int(x) for x in ws.split())
    ebar = np.array([[[1.0, 0.0], [2.0, 3.0]]])
    # alpha = w, beta = 0 gives window w at any N (default reading)
    out, d = so.rule_loss_ref(ebar, 8, s, [float(w)], [0.0], profile_block=4)
    assert out[0, 0] == float(dl)
    num, den = dens.split("/")
    assert d[0] == int(num) / int(den)


def test_candidate_rule_grid():
    a, b = so.candidate_rules()
    assert len(a) == 54
    assert sorted(set(a)) == [-2048.0, 0.0, 2048.0, 4096.0, 6144.0, 8192.0]
    assert sorted(set(b)) == [k / 8 for k in range(9)]


def _masked_count(n, w, s, block):
    """Causal pairs hidden by window w and s sinks, by brute force over (i, j)."""
    nbw = -(-w // block) if block else 0
    count = 0
    for i in range(n):
        for j in range(i + 1):
            if j < s:
                continue
            in_band = (i // block - j // block < nbw) if block else (i - j < w)
            count += not in_band
    return count


@pytest.mark.parametrize("block", [0, 4])
def test_unit_profile_counts_masked_pairs(block):
    # With E_bar = 1 on and below the diagonal blocks, Delta L is the number of
    # masked causal pairs.
    n = 21
    nb = -(-n // 4)
    ebar = np.tril(np.ones((nb, nb)))[None]
    a, b = so.candidate_rules()
    a = a / 512.0   # small windows at this length
    dl, dens = so.rule_loss_ref(ebar, n, 2, a, b, span_includes_sinks=True, block=block, profile_block=4)
    for r in range(len(a)):
        w = so.window_ref(a[r], b[r], n, 2, True)
        assert dl[0, r] == _masked_count(n, w, 2, block)
    assert np.all((dens > 0) & (dens <= 1))


@pytest.mark.parametrize("n, s", [(1, 0), (7, 0), (7, 3), (20, 4), (33, 40)])
def test_density_is_cache_length_over_n(n, s):
    # Density (Sec. 4 "Setups"): in-memory KV-cache length / sequence length
    # during decoding.  Simulate the cache (fill in arrival order, then replace
    # the oldest non-sink entry) over n tokens and count what it holds; the
    # block band leaves the cache token-exact, so it does not change density.
    from oracle.moa_oracle import CacheModel
    for w in range(1, n + 1):
        cm = CacheModel(w, s)
        for p in range(n):
            cm.append(p)
        held = len(cm.positions())
        assert so.density_ref(n, w, s) == held / n
        assert held == min(n, s + w)
        for block in (0, 4):
            _, d = so.rule_loss_ref(np.zeros((1, 9, 9)), n, s, [float(w)], [0.0], block=block, profile_block=4)
            assert d[0] == held / n


def test_density_half_band_rule():
    # A plain band w = N/2 with no sinks keeps half the sequence in memory:
    # density 0.5 (the kept share of the causal pairs would be about 3/4).
    n = 64
    _, d = so.rule_loss_ref(np.zeros((1, 1, 1)), n, 0, [32.0], [0.0])
    assert d[0] == 0.5


def test_selection_hand_example():
    dl = np.array([[0.0, 5.0], [0.0, 1.0]])
    dens = np.array([1.0, 0.5])
    rules, loss = so.select_bruteforce(dl, dens, 0.75)
    assert rules == [0, 1] and loss == 0.5
    assert so.select_bruteforce(dl, dens, 0.4) == (None, np.inf)


def _milp(dl, dens, budget):
    h, r = dl.shape
    c = dl.reshape(-1) / h
    rows = [np.kron(np.eye(h)[i], np.ones(r)) for i in range(h)]
    cons = [LinearConstraint(np.array(rows), 1, 1), LinearConstraint(np.tile(dens, h)[None] / h, -np.inf, budget)]
    res = milp(c, constraints=cons, integrality=np.ones(h * r), bounds=Bounds(0, 1))
    return res.fun if res.success else np.inf


@pytest.mark.parametrize("seed", range(5))
def test_selection_bruteforce_matches_library_milp(seed):
    rng = np.random.default_rng(seed)
    h, r = 3, 6
    dl = rng.normal(size=(h, r))
    dens = rng.uniform(0.1, 1.0, r)
    budget = float(rng.uniform(dens.min(), dens.max()))
    rules, loss = so.select_bruteforce(dl, dens, budget)
    assert loss == pytest.approx(_milp(dl, dens, budget), abs=1e-9)
    if rules is not None:
        assert np.mean(dens[rules]) <= budget + 1e-12


def test_selection_layer_limit():
    # Two layers of two heads; the best unconstrained choice uses two rules in
    # layer 0; with at most one rule per layer the layer must share one.
    dl = np.array([[0.0, 3.0, 9.0], [9.0, 3.0, 0.0], [0.0, 9.0, 9.0], [0.0, 9.0, 9.0]])
    dens = np.array([0.5, 0.5, 0.5])
    rules, loss = so.select_bruteforce(dl, dens, 1.0)
    assert rules == [0, 2, 0, 0] and loss == 0.0
    rules, loss = so.select_bruteforce(dl, dens, 1.0, layer_of=[0, 0, 1, 1], max_rules_per_layer=1)
    assert rules == [1, 1, 0, 0] and loss == 1.5


def test_pareto_front_hand_example():
    # One head, four rules; per-length losses (length A, length B):
    # r0 (1, 3), r1 (2, 2), r2 (3, 1), r3 (2, 3) -- r3 is dominated by r1.
    dls = [np.array([[1.0, 2.0, 3.0, 2.0]]), np.array([[3.0, 2.0, 1.0, 3.0]])]
    dens = [np.array([0.5, 0.5, 0.5, 0.5])] * 2
    assert so.pareto_front_bruteforce(dls, dens, [1.0, None]) == [(1.0, 3.0), (2.0, 2.0), (3.0, 1.0)]
    # a budget that only r0 and r3 meet
    dens_b = [np.array([0.5, 0.9, 0.9, 0.5])] * 2
    assert so.pareto_front_bruteforce(dls, dens_b, [0.6, None]) == [(1.0, 3.0)]
    assert so.dominates((1, 2), (1, 3)) and not so.dominates((1, 3), (1, 3)) and not so.dominates((0, 4), (1, 3))

