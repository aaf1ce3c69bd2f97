"""Pins of the fp64 oracle against facts fixed outside the oracle itself.

Each pin is independent of the oracle's own code: hand-derived worked examples
(tests/golden), a pure-Python brute force written from the definition, a
library routine (torch scaled_dot_product_attention) for the full-window
special case, closed forms, and invariants.  The last test plants plausible
mistakes into copies of the oracle and checks that some pin catches each.
"""
import itertools
import math

import numpy as np
import pytest
import torch

from conftest import read_golden
import oracle
from oracle import moa_oracle as om

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# ---------------------------------------------------------------------------
# independent brute force, written from the definition (pure Python loops)
# ---------------------------------------------------------------------------

def brute_attention(q, k, v, windows, s, scale):
    """Pure-Python loops: O[b][i][h][d] with explicit visibility test."""
    bsz, n, hq, d = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    hkv = len(k[0][0])
    grp = hq // hkv
    out = [[[[0.0] * d for _ in range(hq)] for _ in range(n)] for _ in range(bsz)]
    for b in range(bsz):
        for h in range(hq):
            g = h // grp
            w = windows[g]
            for i in range(n):
                keys = [j for j in range(n) if j <= i and (j < s or i - j < w)]
                sc = [scale * sum(q[b][i][h][x] * k[b][j][g][x] for x in range(d)) for j in keys]
                mx = max(sc)
                ex = [math.exp(z - mx) for z in sc]
                tot = sum(ex)
                for x in range(d):
                    out[b][i][h][x] = sum(ex[t] * v[b][keys[t]][g][x] for t in range(len(keys))) / tot
    return np.array(out)


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------

def test_golden_uniform_attention():
    rows = read_golden("uniform_n8_s2_w3.txt")
    n, s, w = 8, 2, 3
    q = np.zeros((1, n, 1, 1))
    k = _rand((1, n, 1, 1), 0)
    v = np.arange(n, dtype=np.float64).reshape(1, n, 1, 1)
    out = om.attention_ref(q, k, v, [w], s)
    for i, (ii, js, mean) in enumerate(rows):
        assert int(ii) == i
        expect_set = [int(x) for x in js.split()]
        assert list(om.visible_set(i, w, s)) == expect_set
        assert out[0, i, 0, 0] == pytest.approx(float(mean), abs=1e-14)
        # decode at position i over the history 0..i gives the same row
        dec = om.decode_ref(q[:, i], k[:, : i + 1], v[:, : i + 1], [w], s)
        assert dec[0, 0, 0] == pytest.approx(float(mean), abs=1e-14)


def test_golden_cache_trace():
    (row,) = read_golden("cache_s2_w3_t10.txt")
    expect = [int(x) for x in row[0].split()]
    assert list(om.cache_ref([3], 2, 10)) == expect


def test_golden_rule_windows():
    for lhs, rhs in read_golden("rule_windows.txt"):
        a, b, n = lhs.split()
        assert om.window_ref(float(a), float(b), int(n)) == int(rhs)
    p = om.plan_ref([-2048.0, 64.0], [0.5, 0.25], 1000, 64)
    assert list(p["window"]) == [1, 314]
    assert list(p["capacity"]) == [65, 378]
    assert list(p["offset"]) == [0, 65, 443]


@pytest.mark.parametrize("hq,hkv", [(1, 1), (4, 2)])
def test_brute_force_all_windows_and_sinks(hq, hkv):
    n, d = 7, 3
    q = _rand((1, n, hq, d), 1)
    k = _rand((1, n, hkv, d), 2)
    v = _rand((1, n, hkv, d), 3)
    scale = 1.0 / math.sqrt(d)
    for w0, w1, s in itertools.product(range(1, n + 1), (1, 3, n), range(0, n + 1)):
        windows = [w0, w1][:hkv] if hkv == 2 else [w0]
        ref = om.attention_ref(q, k, v, windows, s)
        bf = brute_attention(q.tolist(), k.tolist(), v.tolist(), windows, s, scale)
        np.testing.assert_allclose(ref, bf, rtol=0, atol=1e-12)


def test_full_window_equals_library_causal_attention():
    bsz, n, h, d = 2, 37, 3, 16
    q = _rand((bsz, n, h, d), 4)
    k = _rand((bsz, n, h, d), 5)
    v = _rand((bsz, n, h, d), 6)
    tq = torch.from_numpy(q).permute(0, 2, 1, 3)
    tk = torch.from_numpy(k).permute(0, 2, 1, 3)
    tv = torch.from_numpy(v).permute(0, 2, 1, 3)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    ref = ref.permute(0, 2, 1, 3).numpy()
    for windows, s in (([n] * h, 0), ([n + 5, n, 10 ** 6], 3), ([1, 2, 3], n), ([4, 4, 4], n + 9)):
        out = om.attention_ref(q, k, v, windows, s)
        np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_window_one_no_sink_returns_v():
    q = _rand((2, 19, 4, 8), 7) * 30.0
    k = _rand((2, 19, 2, 8), 8)
    v = _rand((2, 19, 2, 8), 9)
    out = om.attention_ref(q, k, v, [1, 1], 0)
    expect = np.repeat(v, 2, axis=2)
    assert np.array_equal(out, expect)


def test_probability_rows_sum_to_one_and_vanish_outside_mask():
    n, d = 50, 8
    q = _rand((1, n, 2, d), 10)
    k = _rand((1, n, 1, d), 11)
    a = om.probabilities_ref(q, k, [7], 5, 0, 1)
    mask = np.array([[om.visible(i, j, 7, 5) for j in range(n)] for i in range(n)])
    np.testing.assert_allclose(a.sum(-1), 1.0, atol=1e-12)
    assert np.all(a[~mask] == 0.0)
    assert np.all(a[mask] > 0.0)


def test_gqa_equals_repeated_mha():
    n, d = 40, 8
    q = _rand((2, n, 8, d), 12)
    k = _rand((2, n, 2, d), 13)
    v = _rand((2, n, 2, d), 14)
    w = [5, 17]
    out = om.attention_ref(q, k, v, w, 3)
    out_mha = om.attention_ref(q, np.repeat(k, 4, 2), np.repeat(v, 4, 2), [5] * 4 + [17] * 4, 3)
    np.testing.assert_allclose(out, out_mha, atol=1e-13, rtol=0)


def test_dominant_key_selects_its_value():
    # One visible key whose score dwarfs the rest: A -> one-hot, O_i -> v_j.
    n, d = 12, 4
    rng = np.random.default_rng(15)
    q = rng.standard_normal((1, n, 1, d))
    k = rng.standard_normal((1, n, 1, d)) * 1e-3
    v = rng.standard_normal((1, n, 1, d))
    i, j, w, s = 9, 1, 3, 2          # j is a sink, outside the band of i
    k[0, j, 0] = 1e3 * q[0, i, 0]
    out = om.attention_ref(q, k, v, [w], s)
    np.testing.assert_allclose(out[0, i, 0], v[0, j, 0], atol=1e-12)
    # the same key is invisible to row i once it is no longer a sink
    out2 = om.attention_ref(q, k, v, [w], 1)
    assert np.abs(out2[0, i, 0] - v[0, j, 0]).max() > 1e-3


def test_attention_rows_and_decode_match_prefill():
    n, d = 45, 8
    q = _rand((2, n, 4, d), 16)
    k = _rand((2, n, 2, d), 17)
    v = _rand((2, n, 2, d), 18)
    w, s = [6, 30], 4
    full = om.attention_ref(q, k, v, w, s, row_block=16)
    rows = [0, 3, 4, 5, 29, 30, 44]
    for b in range(2):
        for h in range(4):
            part = om.attention_rows_ref(q, k, v, w, s, b, h, rows)
            np.testing.assert_allclose(part, full[b, rows, h], atol=1e-13, rtol=0)
    for t in (0, 5, 31, 44):
        dec = om.decode_ref(q[:, t], k[:, : t + 1], v[:, : t + 1], w, s)
        np.testing.assert_allclose(dec, full[:, t], atol=1e-13, rtol=0)


@pytest.mark.parametrize("w,s", [(1, 0), (1, 3), (4, 0), (4, 2), (9, 9), (2, 30)])
def test_cache_closed_form(w, s):
    for total in range(0, 25):
        cm = om.CacheModel(w, s)
        for p in range(total):
            cm.append(p)
        expect = sorted(set(range(min(s, total))) | set(range(max(s, total - w), total)))
        assert cm.positions() == expect
        # the cached set is exactly the visible set of the newest token
        if total:
            assert expect == list(om.visible_set(total - 1, w, s))


def test_cache_contents_bits():
    bsz, total, hkv, d = 2, 23, 2, 4
    k = torch.randn(bsz, total, hkv, d).to(torch.bfloat16)
    v = torch.randn(bsz, total, hkv, d).to(torch.bfloat16)
    pos, kc, vc = om.cache_contents_ref(k, v, [5, 40], 3)
    assert pos.shape == (bsz, 8 + 43)
    for b in range(bsz):
        for slot, p in enumerate(pos[b]):
            g = 0 if slot < 8 else 1
            if p >= 0:
                assert torch.equal(kc[b, slot], k[b, p, g])
                assert torch.equal(vc[b, slot], v[b, p, g])
            else:
                assert g == 1 and p == -1


# ---------------------------------------------------------------------------
# planted mistakes: each mutated oracle must fail at least one pin
# ---------------------------------------------------------------------------

def _golden_ok(mask_fn):
    rows = read_golden("uniform_n8_s2_w3.txt")
    n, s, w = 8, 2, 3
    for i, (_, _, mean) in enumerate(rows):
        keys = [j for j in range(n) if mask_fn(i, j, w, s)]
        if not keys or abs(sum(keys) / len(keys) - float(mean)) > 1e-12:
            return False
    return True


def test_planted_mask_mistakes_are_caught():
    assert _golden_ok(om.visible)
    mutants = [
        lambda i, j, w, s: j <= i and (j < s or i - j <= w),      # band one too wide
        lambda i, j, w, s: j <= i and (j < s or i - j < w - 1),   # band one too narrow
        lambda i, j, w, s: j < s or (j <= i and i - j < w),       # sinks ignore causality
        lambda i, j, w, s: j <= i and (j <= s or i - j < w),      # one sink too many
        lambda i, j, w, s: j <= i and i - j < w,                  # sinks dropped
        lambda i, j, w, s: j < i and (j < s or i - j < w),        # diagonal dropped
    ]
    for m in mutants:
        assert not _golden_ok(m)


def test_planted_arithmetic_mistakes_are_caught(monkeypatch):
    bsz, n, h, d = 1, 9, 2, 4
    q = _rand((bsz, n, h, d), 20)
    k = _rand((bsz, n, h, d), 21)
    v = _rand((bsz, n, h, d), 22)
    tq, tk, tv = (torch.from_numpy(x).permute(0, 2, 1, 3) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    ref = ref.permute(0, 2, 1, 3).numpy()

    def caught(fn):
        try:
            out = fn(q, k, v, [n, n], 0)
        except Exception:
            return True
        return not np.allclose(out, ref, atol=1e-9)

    assert not caught(om.attention_ref)
    # missing 1/sqrt(D) scale
    monkeypatch.setattr(om, "_scale", lambda d, s: 1.0)
    assert caught(om.attention_ref)
    monkeypatch.undo()
    # transposed score matrix (K Q^T in place of Q K^T)
    def transposed(q, k, v, window, s):
        q64, k64, v64 = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
        out = np.zeros_like(q64)
        for hh in range(h):
            sc = (k64[0, :, hh] @ q64[0, :, hh].T) / math.sqrt(d)
            a = om.masked_softmax_rows(sc, om.visible_mask(n, n, window[hh], s))
            out[0, :, hh] = a @ v64[0, :, hh]
        return out
    assert caught(transposed)
    # softmax normalised over the wrong axis
    monkeypatch.setattr(om, "masked_softmax_rows",
                        lambda s_rows, m: np.exp(np.where(m, s_rows, -np.inf))
                        / np.exp(np.where(m, s_rows, -np.inf)).sum(0, keepdims=True))
    assert caught(om.attention_ref)


# ---------------------------------------------------------------------------
# block-granular band and "span includes sinks" plan mode
# ---------------------------------------------------------------------------

def _frac(text):
    num, den = text.split("/")
    return int(num) / int(den)


def test_golden_block_band_uniform_attention():
    rows = read_golden("block_n16_b4_s2_w6.txt")
    n, s, w, blk = 16, 2, 6, 4
    q = np.zeros((1, n, 1, 1))
    k = _rand((1, n, 1, 1), 30)
    v = np.arange(n, dtype=np.float64).reshape(1, n, 1, 1)
    out = om.attention_ref(q, k, v, [w], s, block=blk)
    mask = om.visible_mask(n, n, w, s, block=blk)
    for i, (ii, js, mean) in enumerate(rows):
        assert int(ii) == i
        expect_set = [int(x) for x in js.split()]
        assert list(om.visible_set(i, w, s, blk)) == expect_set
        assert [j for j in range(n) if om.visible(i, j, w, s, blk)] == expect_set
        assert list(np.nonzero(mask[i])[0]) == expect_set
        assert out[0, i, 0, 0] == pytest.approx(_frac(mean), abs=1e-14)
        rows_out = om.attention_rows_ref(q, k, v, [w], s, 0, 0, [i], block=blk)
        assert rows_out[0, 0] == pytest.approx(_frac(mean), abs=1e-14)


def test_golden_span_includes_sinks_rule():
    for lhs, span, rhs in read_golden("rule_windows_span_sinks.txt"):
        a, b, n, s = lhs.split()
        w = om.window_ref(float(a), float(b), int(n), int(s), span_includes_sinks=True)
        assert w == int(rhs)
        assert w + int(s) == max(int(span), int(s) + 1)
    p = om.plan_ref([100.0, 5000.0], [0.0, 0.0], 1000, 64, span_includes_sinks=True)
    assert list(p["window"]) == [36, 936]
    assert list(p["capacity"]) == [100, 1000]


def test_block_band_against_token_band():
    # The block band of row i starts at a block boundary: on the last row of a
    # block it covers the token band (equal to it when w is a multiple of the
    # block), on the first row it is covered by it, and the counts differ by
    # less than one block everywhere.
    n, blk = 300, 64
    ends, starts = np.arange(blk - 1, n, blk), np.arange(0, n, blk)
    for w in (1, 5, 63, 64, 65, 128, 200, 256, 299):
        for s in (0, 3, 64):
            tok = om.visible_mask(n, n, w, s)
            blm = om.visible_mask(n, n, w, s, block=blk)
            assert not np.any(tok[ends] & ~blm[ends])
            assert not np.any(blm[starts] & ~tok[starts])
            assert np.abs(blm.sum(axis=1) - tok.sum(axis=1)).max() <= blk - 1
            if w % blk == 0:
                assert np.array_equal(tok[ends], blm[ends])


def test_block_band_wide_enough_equals_causal_attention():
    bsz, n, h, d = 1, 70, 2, 8
    q = _rand((bsz, n, h, d), 31)
    k = _rand((bsz, n, h, d), 32)
    v = _rand((bsz, n, h, d), 33)
    tq, tk, tv = (torch.from_numpy(x).permute(0, 2, 1, 3) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True).permute(0, 2, 1, 3).numpy()
    # 65 tokens round up to 2 blocks of 64: every key of a 70-token prompt is in the band
    np.testing.assert_allclose(om.attention_ref(q, k, v, [65, 128], 0, block=64), ref, rtol=0, atol=1e-12)


def test_block_band_brute_force():
    # Mask rebuilt from explicit lists of allowed blocks; softmax by Python loops.
    n, d, blk = 11, 3, 3
    q = _rand((1, n, 1, d), 34)
    k = _rand((1, n, 1, d), 35)
    v = _rand((1, n, 1, d), 36)
    for w in range(1, n + 2):
        nb = (w + blk - 1) // blk
        for s in (0, 1, 3, 5):
            ref = om.attention_ref(q, k, v, [w], s, block=blk)
            for i in range(n):
                blocks = [bb for bb in range(i // blk + 1) if bb > i // blk - nb]
                keys = sorted({j for bb in blocks for j in range(bb * blk, min(bb * blk + blk, i + 1))}
                              | set(range(min(s, i + 1))))
                sc = [sum(q[0, i, 0, x] * k[0, j, 0, x] for x in range(d)) / math.sqrt(d) for j in keys]
                mx = max(sc)
                ex = [math.exp(z - mx) for z in sc]
                for x in range(d):
                    val = sum(e * v[0, j, 0, x] for e, j in zip(ex, keys)) / sum(ex)
                    assert abs(val - ref[0, i, 0, x]) < 1e-12


def _golden_block_ok(mask_fn):
    rows = read_golden("block_n16_b4_s2_w6.txt")
    n, s, w, blk = 16, 2, 6, 4
    for i, (_, _, mean) in enumerate(rows):
        keys = [j for j in range(n) if mask_fn(i, j, w, s, blk)]
        if not keys or abs(sum(keys) / len(keys) - _frac(mean)) > 1e-12:
            return False
    return True


def test_planted_block_mask_mistakes_are_caught():
    assert _golden_block_ok(om.visible)
    mutants = [
        lambda i, j, w, s, b: j <= i and (j < s or i // b - j // b < w // b),             # floor, not ceil
        lambda i, j, w, s, b: j <= i and (j < s or i // b - j // b <= -(-w // b)),        # one block too many
        lambda i, j, w, s, b: j <= i and (j < s or i // b - (j + 1) // b < -(-w // b)),   # key block shifted
        lambda i, j, w, s, b: j <= i and (j < s or i - j < w),                            # token band
        lambda i, j, w, s, b: j < s or (j <= i and i // b - j // b < -(-w // b)),         # sinks ignore causality
        lambda i, j, w, s, b: j // b <= i // b and (j < s or i // b - j // b < -(-w // b)),  # no causality inside the block
    ]
    for m in mutants:
        assert not _golden_block_ok(m)


def test_decode_over_the_cache_slots_in_any_order():
    # Softmax over a set does not depend on its order: attending over the cache
    # model's filled slots (ring order, then shuffled) gives the decode row
    # computed from the full history.
    n, hq, hkv, d, s = 40, 4, 2, 8, 3
    windows = [5, 17]
    q = _rand((1, n, hq, d), 70)
    k = _rand((1, n, hkv, d), 71)
    v = _rand((1, n, hkv, d), 72)
    ref = om.decode_ref(q[:, n - 1], k, v, windows, s)
    pos, kc, vc = om.cache_contents_ref(torch.from_numpy(k), torch.from_numpy(v), windows, s)
    offsets = np.cumsum([0] + [w + s for w in windows])
    rng = np.random.default_rng(5)
    for h in range(hq):
        g = h // (hq // hkv)
        slots = [i for i in range(offsets[g], offsets[g + 1]) if pos[0, i] >= 0]
        for order in (slots, list(rng.permutation(slots))):
            ks = kc[0, order].numpy()
            vs = vc[0, order].numpy()
            sc = ks @ q[0, n - 1, h] / math.sqrt(d)
            e = np.exp(sc - sc.max())
            np.testing.assert_allclose((e / e.sum()) @ vs, ref[0, h], rtol=0, atol=1e-12)
