"""Host-side rule selection (paper Appendix "Optimizing at Single Length")
against exhaustive enumeration by the oracle, on oracle-computed loss tables."""
import numpy as np
import pytest

import oracle
from paper_2406_14909_amd import search


def test_candidate_grid_matches_oracle():
    a, b = search.candidate_rules()
    oa, ob = oracle.candidate_rules()
    assert np.array_equal(a, oa) and np.array_equal(b, ob)


def _table(seed, h=3, n=300, flags=(True, 64)):
    rng = np.random.default_rng(seed)
    nb = -(-n // 64)
    ebar = np.tril(rng.normal(size=(h, nb, nb))) * 1e-3
    a, b = oracle.candidate_rules()
    return oracle.rule_loss_ref(ebar, n, 64, a, b, span_includes_sinks=flags[0], block=flags[1])


@pytest.mark.parametrize("seed", range(4))
def test_selection_matches_exhaustive_search(seed):
    dl, dens = _table(seed)
    for budget in (float(dens.min()), 0.3, 0.6, 1.0):
        rules, loss = search.select_rules(dl, dens, budget)
        ref_rules, ref_loss = oracle.select_bruteforce(dl, dens, budget)
        if ref_rules is None:
            assert rules is None
            continue
        assert loss == pytest.approx(ref_loss, abs=1e-12)       # the optimum is unique; ties in rules are not
        assert np.mean(dens[rules]) <= budget + 1e-12


def test_selection_with_layer_limit_matches_exhaustive_search():
    rng = np.random.default_rng(9)
    dl = rng.normal(size=(4, 6))
    dens = rng.uniform(0.2, 1.0, 6)
    layer_of = [0, 0, 1, 1]
    for k in (1, 2):
        rules, loss = search.select_rules(dl, dens, 0.7, layer_of=layer_of, max_rules_per_layer=k)
        _, ref_loss = oracle.select_bruteforce(dl, dens, 0.7, layer_of=layer_of, max_rules_per_layer=k)
        assert loss == pytest.approx(ref_loss, abs=1e-12)
        for layer in (0, 1):
            assert len({rules[h] for h in range(4) if layer_of[h] == layer}) <= k


def test_infeasible_budget():
    dl, dens = _table(1)
    assert search.select_rules(dl, dens, float(dens.min()) - 1e-3) == (None, np.inf)


@pytest.mark.parametrize("seed", range(3))
def test_multi_length_front_lies_on_the_exact_front(seed):
    rng = np.random.default_rng(20 + seed)
    h, r = 3, 6
    dls = [rng.normal(size=(h, r)) for _ in range(2)]
    dens = [rng.uniform(0.2, 1.0, r), rng.uniform(0.2, 1.0, r)]
    budgets = [0.7, 0.8]
    val = rng.normal(size=(h, r))
    front, best = search.select_multi_length(dls, dens, budgets, intervals=5, val_dl=val)
    exact = oracle.pareto_front_bruteforce(dls, dens, budgets)
    assert front
    for rules, vec in front:
        assert any(np.allclose(vec, p, atol=1e-12) for p in exact)          # every member is Pareto-optimal
        for i in range(2):
            assert np.mean(dens[i][rules]) <= budgets[i] + 1e-12
    for i in range(2):                                                      # both extreme points are found
        assert min(v[i] for _, v in front) == pytest.approx(min(p[i] for p in exact), abs=1e-12)
    assert best is not None and float(np.mean(val[np.arange(h), best[0]])) == pytest.approx(
        min(float(np.mean(val[np.arange(h), f[0]])) for f in front), abs=1e-12)

