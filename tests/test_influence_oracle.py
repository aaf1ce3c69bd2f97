"""Pins of the attention-influence oracle (paper Sec. 3.3, Eq. 3; Appendix
"Derivation of Attention Influence"), independent of its own formula."""
import math

import numpy as np
import pytest
import torch

from conftest import read_golden
from oracle import influence_oracle as io
from oracle import moa_oracle as om


def _frac(t):
    a, b = t.split("/")
    return int(a) / int(b)


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _softmax_rows(s):
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def test_golden_hand_worked_row():
    ((a, g, e),) = read_golden("influence_row.txt")
    a = np.array([[_frac(x) for x in a.split()]])
    g = np.array([[float(x) for x in g.split()]])
    e = np.array([[_frac(x) for x in e.split()]])
    np.testing.assert_allclose(io.influence_ref(a, g), e, rtol=0, atol=1e-15)


def _exact_masking_change(a, c):
    """For L(A) = sum C * A: the exact change of L when A[i, j] is masked and
    row i renormalised, by recomputing the masked row."""
    n_rows, n_cols = a.shape
    out = np.zeros_like(a)
    base = (c * a).sum(axis=-1)
    for i in range(n_rows):
        for j in range(n_cols):
            if a[i, j] == 0.0 or a[i, j] == 1.0:
                continue
            row = a[i].copy()
            row[j] = 0.0
            row /= row.sum()
            out[i, j] = (c[i] * row).sum() - base[i]
    return out


@pytest.mark.parametrize("seed", range(3))
def test_exact_masking_identity_for_linear_loss(seed):
    # Causal softmax rows of random scores (row 0 has a single weight 1).
    n = 9
    s = _rand((n, n), seed) * 2.0
    s = np.where(np.tril(np.ones((n, n), dtype=bool)), s, -np.inf)
    a = _softmax_rows(s)
    c = _rand((n, n), 100 + seed)
    e = io.influence_ref(a, c)
    np.testing.assert_allclose(e, _exact_masking_change(a, c), rtol=0, atol=1e-12)
    assert np.all(e[np.triu_indices(n, 1)] == 0.0) and e[0, 0] == 0.0


def test_grad_wrt_probabilities_matches_autograd():
    bsz, n, hq, hkv, d = 2, 7, 4, 2, 5
    q, k, v, do = (_rand(sh, 10 + i) for i, sh in enumerate([(bsz, n, hq, d), (bsz, n, hkv, d),
                                                              (bsz, n, hkv, d), (bsz, n, hq, d)]))
    a = io.causal_probabilities(q, k)
    at = torch.tensor(a, requires_grad=True)
    vt = torch.tensor(v).repeat_interleave(hq // hkv, dim=2).permute(0, 2, 1, 3)   # [B, Hq, n, d]
    o = at @ vt
    loss = (o * torch.tensor(do).permute(0, 2, 1, 3)).sum()
    loss.backward()
    np.testing.assert_allclose(io.grad_wrt_probabilities(v, do, hq), at.grad.numpy(), rtol=0, atol=1e-12)
    # A itself: the full-window, no-sink MoA probabilities (already pinned) are dense causal attention
    for b in range(bsz):
        for h in range(hq):
            np.testing.assert_allclose(a[b, h], om.probabilities_ref(q, k, [n] * hkv, 0, b, h), rtol=0, atol=1e-14)


def test_influence_through_the_output_is_exact():
    # A loss L = sum W * O with O = A V is linear in A, so the influence computed
    # from dL/dA = W V^T equals the exact change of L when (i, j) is masked.
    n, d = 12, 4
    q, k, v, w = (_rand((1, n, 1, d), 20 + i) for i in range(4))
    a = io.causal_probabilities(q * 0.3, k)[0, 0]
    g = io.grad_wrt_probabilities(v, w, 1)[0, 0]
    e = io.influence_ref(a, g)
    loss = lambda aa: float(((aa @ v[0, :, 0, :]) * w[0, :, 0, :]).sum())
    for i, j in ((5, 2), (11, 0), (7, 7), (3, 1)):
        row = a[i].copy()
        row[j] = 0.0
        row /= row.sum()
        a2 = a.copy()
        a2[i] = row
        assert abs((loss(a2) - loss(a)) - e[i, j]) <= 1e-12


def test_constant_gradient_rows_have_no_influence():
    a = _softmax_rows(_rand((6, 6), 3))
    g = np.repeat(_rand((6, 1), 4), 6, axis=1)
    assert np.abs(io.influence_ref(a, g)).max() < 1e-15


def test_block_average_equals_torch_pooling():
    e = _rand((3, 2, 256, 256), 5)
    pooled = torch.nn.functional.avg_pool2d(torch.tensor(e), 64).mean(dim=0).numpy()
    np.testing.assert_allclose(io.block_average_ref(e, 64), pooled, rtol=0, atol=1e-14)
    # partial edge tiles average over the entries that exist
    e2 = np.ones((1, 1, 70, 70))
    e2[0, 0, 64:, :] = 3.0
    out = io.block_average_ref(e2, 64)
    assert out.shape == (1, 2, 2) and out[0, 1, 0] == 3.0 and out[0, 0, 1] == 1.0


def test_profile_composes_the_steps():
    bsz, n, hq, hkv, d = 2, 130, 2, 1, 8
    q, k, v, do = (_rand(sh, 40 + i) for i, sh in enumerate([(bsz, n, hq, d), (bsz, n, hkv, d),
                                                              (bsz, n, hkv, d), (bsz, n, hq, d)]))
    prof = io.influence_profile_ref(q, k, v, do)
    a = io.causal_probabilities(q, k)
    g = io.grad_wrt_probabilities(v, do, hq)
    e = io.influence_ref(a, g)
    assert prof.shape == (hq, 3, 3)
    assert prof[1, 2, 1] == pytest.approx(e[:, 1, 128:, 64:128].sum() / (bsz * 2 * 64), abs=1e-15)
    assert np.all(prof[:, 0, 1:] == 0.0) and prof[0, 1, 2] == 0.0   # above the diagonal blocks


def test_planted_influence_mistakes_are_caught():
    n = 8
    s = np.where(np.tril(np.ones((n, n), dtype=bool)), _rand((n, n), 50), -np.inf)
    a = _softmax_rows(s)
    c = _rand((n, n), 51)
    exact = _exact_masking_change(a, c)

    def ok(fn):
        return np.allclose(fn(a, c), exact, atol=1e-10)

    assert ok(io.influence_ref)
    d = lambda aa, gg: (gg * aa).sum(axis=-1, keepdims=True)
    inside = lambda aa: (aa > 0) & (aa < 1)
    mutants = [
        # the printed matrix form without the minus sign
        lambda aa, gg: np.where(inside(aa), aa / np.where(inside(aa), 1 - aa, 1) * (gg - d(aa, gg)), 0.0),
        # direct effect only (no renormalisation of the row)
        lambda aa, gg: np.where(inside(aa), -aa * gg, 0.0),
        # column sums in place of row sums
        lambda aa, gg: np.where(inside(aa), -aa / np.where(inside(aa), 1 - aa, 1)
                                * (gg - (gg * aa).sum(axis=0, keepdims=True)), 0.0),
        # 1/A in place of 1/(1 - A)
        lambda aa, gg: np.where(inside(aa), -(1 - aa) / np.where(inside(aa), aa, 1) * (gg - d(aa, gg)), 0.0),
    ]
    for m in mutants:
        assert not ok(m)


def test_sampled_rows_equal_the_full_oracle():
    bsz, n, hq, hkv, d = 2, 70, 4, 2, 8
    q, k, v, do = (_rand(sh, 60 + i) for i, sh in enumerate([(bsz, n, hq, d), (bsz, n, hkv, d),
                                                              (bsz, n, hkv, d), (bsz, n, hq, d)]))
    full = io.influence_ref(io.causal_probabilities(q, k), io.grad_wrt_probabilities(v, do, hq))
    rows = [0, 1, 33, 64, 69]
    for b, h in ((0, 0), (1, 3)):
        np.testing.assert_allclose(io.influence_rows_ref(q, k, v, do, b, h, rows), full[b, h, rows],
                                   rtol=0, atol=1e-13)

