"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Small and medium shapes that the oracle finishes in seconds; they span several
tiles and ragged tails.  The full workload shapes are in test_gpu_workloads.py.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from helpers import BF16_ATOL, F32_ATOL, assert_close, bits, guard_intact, guarded_empty, oracle_windows
from paper_2406_14909_amd import moa as M

pytestmark = pytest.mark.gpu

DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _say(*args):
    print("[case]", *args, flush=True)


def _inputs(bsz, n, hq, hkv, d, dtype, seed):
    q = workloads.randn((bsz, n, hq, d), seed, dtype, "cuda")
    k = workloads.randn((bsz, n, hkv, d), seed + 1, dtype, "cuda")
    v = workloads.randn((bsz, n, hkv, d), seed + 2, dtype, "cuda")
    return q, k, v


def _plan(hq, hkv, d, s, n, dtype, windows, flags=0):
    """Plan with rule alpha = w, beta = 0 per head, and the oracle's windows
    for the same rule (what every oracle call below is given)."""
    alpha, beta = [float(w) for w in windows], [0.0] * len(windows)
    plan = M.moa_plan(hq, hkv, d, s, n, dtype, alpha, beta, flags=flags)
    return plan, oracle_windows(plan, alpha, beta, bool(flags & M.MOA_SPAN_INCLUDES_SINKS))


# ---------------------------------------------------------------------------
# prefill
# ---------------------------------------------------------------------------

PREFILL_CASES = [
    # dtype, B, n, Hq, Hkv, D, sinks, windows
    ("f32", 1, 512, 4, 4, 64, 4, [64, 128, 256, 512]),          # the small workload shape
    ("f32", 2, 300, 4, 2, 128, 3, [1, 77]),
    ("bf16", 1, 512, 4, 4, 64, 4, [64, 128, 256, 512]),
    ("bf16", 2, 333, 8, 2, 128, 16, [5, 200]),
    ("bf16", 1, 700, 8, 1, 128, 64, [129]),
    ("bf16", 1, 257, 4, 4, 128, 0, [1, 2, 64, 1000]),
    ("bf16", 3, 130, 2, 2, 64, 200, [3, 7]),                    # sinks cover everything
    ("bf16", 1, 1, 8, 8, 128, 4, [1, 1, 1, 1, 5, 5, 5, 5]),     # single token
    ("bf16", 1, 1100, 16, 2, 128, 64, [96, 640]),
]


@pytest.mark.parametrize("case", PREFILL_CASES, ids=lambda c: f"{c[0]}-B{c[1]}-n{c[2]}-hq{c[3]}-hkv{c[4]}-d{c[5]}-s{c[6]}")
def test_prefill_matches_oracle(case):
    dt, bsz, n, hq, hkv, d, s, windows = case
    _say("prefill", case)
    dtype = DT[dt]
    plan, rw = _plan(hq, hkv, d, s, n, dt, windows)
    q, k, v = _inputs(bsz, n, hq, hkv, d, dtype, 100 + n)
    o, buf = guarded_empty(q.shape, dtype)
    M.moa_prefill(plan, q, k, v, o)
    torch.cuda.synchronize()
    assert guard_intact(buf, q.shape), "write past the output"
    ref = oracle.attention_ref(q, k, v, rw, s)
    assert_close(o, ref, dtype, with_rounding=True, what=f"prefill {case}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_prefill_window_one_no_sink_is_identity(dt):
    _say("prefill w=1 s=0", dt)
    dtype = DT[dt]
    bsz, n, hq, hkv, d = 2, 389, 8, 4, 128
    plan, _ = _plan(hq, hkv, d, 0, n, dt, [1] * hkv)
    q, k, v = _inputs(bsz, n, hq, hkv, d, dtype, 7)
    o = M.moa_prefill(plan, q, k, v)
    torch.cuda.synchronize()
    expect = v.repeat_interleave(hq // hkv, dim=2)
    assert torch.equal(bits(o), bits(expect))


def test_prefill_full_window_equals_causal_attention():
    _say("prefill full window")
    bsz, n, h, d = 1, 600, 4, 128
    plan, _ = _plan(h, h, d, 0, n, "f32", [n] * h)
    q, k, v = _inputs(bsz, n, h, h, d, torch.float32, 9)
    o = M.moa_prefill(plan, q, k, v)
    tq, tk, tv = (x.double().cpu().permute(0, 2, 1, 3) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    assert_close(o, ref.permute(0, 2, 1, 3).numpy(), torch.float32, what="full window")


def test_prefill_is_deterministic():
    _say("prefill determinism")
    plan, _ = _plan(8, 2, 128, 16, 800, "bf16", [33, 400])
    q, k, v = _inputs(1, 800, 8, 2, 128, torch.bfloat16, 11)
    o1 = M.moa_prefill(plan, q, k, v)
    o2 = M.moa_prefill(plan, q, k, v)
    torch.cuda.synchronize()
    assert torch.equal(bits(o1), bits(o2))


BLOCK_CASES = [
    # dtype, B, n, Hq, Hkv, D, sinks, windows (band counted in 64-token blocks)
    ("bf16", 1, 700, 8, 2, 128, 64, [1, 200]),
    ("bf16", 2, 333, 4, 4, 64, 64, [63, 64, 65, 128]),
    ("f32", 1, 300, 4, 2, 128, 3, [5, 130]),
    ("bf16", 1, 1100, 16, 2, 128, 64, [96, 640]),
    ("bf16", 1, 129, 2, 2, 128, 0, [64, 1000]),
    ("bf16", 3, 520, 8, 8, 128, 10, [1, 64, 127, 128, 129, 256, 300, 520]),
]


@pytest.mark.parametrize("case", BLOCK_CASES, ids=lambda c: f"{c[0]}-B{c[1]}-n{c[2]}-hq{c[3]}-hkv{c[4]}-d{c[5]}-s{c[6]}")
def test_prefill_block_band_matches_oracle(case):
    dt, bsz, n, hq, hkv, d, s, windows = case
    _say("prefill block band", case)
    dtype = DT[dt]
    plan, rw = _plan(hq, hkv, d, s, n, dt, windows, flags=M.MOA_BLOCK_BAND)
    assert rw == [min(w, n) for w in windows]
    q, k, v = _inputs(bsz, n, hq, hkv, d, dtype, 200 + n)
    o, buf = guarded_empty(q.shape, dtype)
    M.moa_prefill(plan, q, k, v, o)
    torch.cuda.synchronize()
    assert guard_intact(buf, q.shape), "write past the output"
    ref = oracle.attention_ref(q, k, v, rw, s, block=64)
    assert_close(o, ref, dtype, with_rounding=True, what=f"block prefill {case}")


def test_span_includes_sinks_prefill_and_decode():
    _say("span includes sinks")
    alpha, beta, n, s = [100.0, 10.0, 5000.0, 300.5], [0.0, 0.0, 0.0, 0.1], 900, 64
    plan = M.moa_plan(8, 4, 128, s, n, "bf16", alpha, beta, flags=M.MOA_SPAN_INCLUDES_SINKS)
    windows = oracle_windows(plan, alpha, beta, span_includes_sinks=True)
    assert windows == [36, 1, 836, 326]
    q, k, v = _inputs(2, n + 1, 8, 4, 128, torch.bfloat16, 77)
    o = M.moa_prefill(plan, q[:, :n].contiguous(), k[:, :n].contiguous(), v[:, :n].contiguous())
    kc, vc, pos = M.new_cache(plan, 2)
    ws = M.new_workspace(plan, 2)
    M.moa_kv_append(plan, kc, vc, pos, k[:, :n].contiguous(), v[:, :n].contiguous(), 0)
    M.moa_kv_append(plan, kc, vc, pos, k[:, n:].contiguous(), v[:, n:].contiguous(), n)
    od = M.moa_decode(plan, q[:, n].contiguous(), kc, vc, n, ws)
    torch.cuda.synchronize()
    assert_close(o, oracle.attention_ref(q[:, :n], k[:, :n], v[:, :n], windows, s), torch.bfloat16,
                 with_rounding=True, what="span prefill")
    assert_close(od, oracle.decode_ref(q[:, n], k, v, windows, s), torch.bfloat16, with_rounding=True,
                 what="span decode")


def test_block_band_leaves_decode_token_exact():
    _say("block band decode")
    n, s, windows = 300, 4, [70, 129]
    plan, rw = _plan(4, 2, 128, s, n, "bf16", windows, flags=M.MOA_BLOCK_BAND)
    assert rw == windows
    q, k, v = _inputs(1, n, 4, 2, 128, torch.bfloat16, 78)
    kc, vc, pos = M.new_cache(plan, 1)
    ws = M.new_workspace(plan, 1)
    M.moa_kv_append(plan, kc, vc, pos, k.contiguous(), v.contiguous(), 0)
    od = M.moa_decode(plan, q[:, n - 1].contiguous(), kc, vc, n - 1, ws)
    torch.cuda.synchronize()
    assert_close(od, oracle.decode_ref(q[:, n - 1], k, v, windows, s), torch.bfloat16, with_rounding=True,
                 what="block-band plan decode")


# ---------------------------------------------------------------------------
# KV append / evict (bit-exact)
# ---------------------------------------------------------------------------

APPEND_CASES = [
    ("bf16", 2, 4, 128, 3, [1, 5, 17, 64]),
    ("f32", 3, 2, 64, 0, [1, 9]),
    ("bf16", 1, 3, 64, 8, [2, 8, 100]),
    ("f32", 2, 1, 128, 5, [40]),
]


@pytest.mark.parametrize("case", APPEND_CASES, ids=lambda c: f"{c[0]}-B{c[1]}-hkv{c[2]}-d{c[3]}-s{c[4]}")
def test_kv_append_bulk_then_single_bit_exact(case):
    dt, bsz, hkv, d, s, windows = case
    _say("append", case)
    dtype = DT[dt]
    total, n0 = 150, 90
    plan, rw = _plan(hkv, hkv, d, s, n0, dt, windows)
    k = workloads.randn((bsz, total, hkv, d), 21, dtype, "cuda")
    v = workloads.randn((bsz, total, hkv, d), 22, dtype, "cuda")
    kc, vc, pos = M.new_cache(plan, bsz)
    M.moa_kv_append(plan, kc, vc, pos, k[:, :n0].contiguous(), v[:, :n0].contiguous(), 0)
    for t in range(n0, total):
        M.moa_kv_append(plan, kc, vc, pos, k[:, t:t + 1].contiguous(), v[:, t:t + 1].contiguous(), t)
        if t in (n0, n0 + 1, total - 1):
            torch.cuda.synchronize()
            epos, ek, ev = oracle.cache_contents_ref(k[:, : t + 1].cpu(), v[:, : t + 1].cpu(), rw, s)
            assert np.array_equal(pos.cpu().numpy(), epos), f"pos table after {t}"
            assert torch.equal(bits(kc), bits(ek)), f"K cache after {t}"
            assert torch.equal(bits(vc), bits(ev)), f"V cache after {t}"


def test_kv_append_chunked_equals_single():
    _say("append chunked")
    bsz, hkv, d, s = 2, 3, 128, 4
    plan, _ = _plan(hkv, hkv, d, s, 64, "bf16", [1, 13, 64])
    total = 200
    k = workloads.randn((bsz, total, hkv, d), 31, torch.bfloat16, "cuda")
    v = workloads.randn((bsz, total, hkv, d), 32, torch.bfloat16, "cuda")
    c1 = M.new_cache(plan, bsz)
    c2 = M.new_cache(plan, bsz)
    for t in range(total):
        M.moa_kv_append(plan, *c1, k[:, t:t + 1].contiguous(), v[:, t:t + 1].contiguous(), t)
    cuts = [0, 3, 4, 50, 51, 120, 200]
    for a, b in zip(cuts[:-1], cuts[1:]):
        M.moa_kv_append(plan, *c2, k[:, a:b].contiguous(), v[:, a:b].contiguous(), a)
    torch.cuda.synchronize()
    for x, y in zip(c1, c2):
        assert torch.equal(bits(x), bits(y))


# ---------------------------------------------------------------------------
# decode (split-K over ragged per-head caches)
# ---------------------------------------------------------------------------

def _decode_run(dt, bsz, hq, hkv, d, s, windows, n0, steps, seed, poison=False):
    dtype = DT[dt]
    total = n0 + steps
    plan, rw = _plan(hq, hkv, d, s, max(n0, max(windows)), dt, windows)
    q = workloads.randn((bsz, total, hq, d), seed, dtype, "cuda")
    k = workloads.randn((bsz, total, hkv, d), seed + 1, dtype, "cuda")
    v = workloads.randn((bsz, total, hkv, d), seed + 2, dtype, "cuda")
    kc, vc, pos = M.new_cache(plan, bsz)
    ws = M.new_workspace(plan, bsz)
    if poison:   # partials must never be read before being written (0xFF.. = NaN)
        ws.fill_(0xFF)
    M.moa_kv_append(plan, kc, vc, pos, k[:, :n0].contiguous(), v[:, :n0].contiguous(), 0)
    outs = []
    for t in range(n0, total):
        M.moa_kv_append(plan, kc, vc, pos, k[:, t:t + 1].contiguous(), v[:, t:t + 1].contiguous(), t)
        o, buf = guarded_empty((bsz, hq, d), dtype)
        M.moa_decode(plan, q[:, t].contiguous(), kc, vc, t, ws, o)
        outs.append((t, o, buf))
    torch.cuda.synchronize()
    for t, o, buf in outs:
        assert guard_intact(buf, (bsz, hq, d)), f"write past decode output at {t}"
        ref = oracle.decode_ref(q[:, t], k[:, : t + 1], v[:, : t + 1], rw, s)
        assert_close(o, ref, dtype, with_rounding=True, what=f"decode t={t}")
    return plan, q, k, v


def test_decode_small_workload_f32():
    wl = workloads.workload(0)
    _say("decode small workload", wl.name)
    _decode_run("f32", 1, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.num_sink,
                [64, 128, 256, 512], wl.n, wl.decode_steps, 40)


DECODE_CASES = [
    # dtype, B, Hq, Hkv, D, s, windows, n0, steps
    ("bf16", 2, 4, 4, 128, 4, [1, 30, 700, 1500], 1400, 4),   # several chunks, growing head
    ("bf16", 3, 8, 1, 128, 64, [2000], 2100, 3),               # G = 8
    ("bf16", 2, 16, 4, 128, 16, [100, 1025, 513, 512], 1100, 3),  # G = 4, chunk edges
    ("bf16", 2, 4, 2, 64, 0, [1, 3], 10, 5),                   # tiny caches, no sinks
    ("f32", 2, 8, 4, 128, 8, [600, 5, 1, 1200], 1300, 3),      # G = 2 fp32
    ("f32", 1, 4, 4, 64, 2, [1, 2, 3, 4], 1, 6),               # first positions
    ("bf16", 1, 8, 1, 128, 64, [140000], 140000, 2),          # one cache over ~550 workers
    ("bf16", 2, 16, 8, 128, 64, [1, 63, 64, 65, 200, 1000, 2500, 40], 2600, 2),  # G = 2 matrix cores
    ("bf16", 2, 8, 2, 64, 4, [300, 1900], 2000, 3),           # G = 4, head_dim 64
    ("bf16", 1, 64, 8, 128, 64, [5000, 1, 3000, 64, 700, 4999, 128, 2048], 5100, 2),  # G = 8
    ("bf16", 4, 16, 2, 64, 3, [1, 2], 5, 4),                  # G = 8, one worker for the batch
    ("bf16", 8, 8, 8, 128, 64, [3000, 17, 900, 2999, 1, 1500, 333, 2000], 3000, 2),  # many workers
    ("bf16", 1, 16, 4, 64, 16, [30000, 5, 70000, 1], 70000, 2),  # G = 4, one cache over > 32 workers
    # every other (dtype, head_dim, group) instantiation the plan accepts
    ("bf16", 3, 4, 4, 64, 8, [10, 700, 1300, 64], 1400, 3),   # bf16 G = 1, head_dim 64
    ("f32", 2, 4, 4, 128, 16, [1, 500, 1200, 77], 1300, 3),   # fp32 G = 1, head_dim 128
    ("f32", 2, 8, 4, 64, 0, [1, 900, 64, 1500], 1600, 2),     # fp32 G = 2, head_dim 64
    ("f32", 2, 8, 2, 64, 4, [300, 1900], 2000, 3),            # fp32 G = 4, head_dim 64
    ("f32", 1, 16, 4, 128, 64, [5, 1025, 3000, 64], 3100, 2),  # fp32 G = 4, head_dim 128
    ("f32", 2, 16, 2, 64, 3, [2500, 40], 2600, 2),            # fp32 G = 8, head_dim 64
    ("f32", 1, 64, 8, 128, 64, [5000, 1, 3000, 64, 700, 4999, 128, 2048], 5100, 2),  # fp32 G = 8, head_dim 128
]


@pytest.mark.parametrize("case", DECODE_CASES, ids=lambda c: f"{c[0]}-B{c[1]}-hq{c[2]}-hkv{c[3]}-d{c[4]}")
def test_decode_matches_oracle(case):
    _say("decode", case)
    _decode_run(*case, seed=50, poison=True)


SINGLE_KEY_CASES = [
    # dtype, B, Hq, Hkv, D (one case per decode kernel family and group size)
    ("bf16", 3, 4, 4, 128),     # vector-ALU kernel, G = 1
    ("bf16", 3, 8, 4, 128),     # matrix-core kernel, G = 2
    ("bf16", 2, 16, 4, 64),     # matrix-core kernel, G = 4, head_dim 64
    ("bf16", 64, 64, 8, 128),   # matrix-core kernel, G = 8, 512 slots: two workers
    ("f32", 2, 4, 4, 64),       # fp32, G = 1
    ("f32", 2, 64, 8, 128),     # fp32, G = 8
]


@pytest.mark.parametrize("case", SINGLE_KEY_CASES, ids=lambda c: f"{c[0]}-B{c[1]}-hq{c[2]}-hkv{c[3]}-d{c[4]}")
def test_decode_of_a_single_cached_key_returns_its_value(case):
    """Decode at position 0: every cache holds one key, whose softmax weight is
    exactly 1 (paper Sec. 2.1, Eq. 1 over a one-element set), so each output
    row is the cached value of its KV head, bit for bit in either dtype."""
    dt, bsz, hq, hkv, d = case
    _say("decode single key", case)
    dtype = DT[dt]
    plan, _ = _plan(hq, hkv, d, 4, 64, dt, [1 + 9 * g for g in range(hkv)])
    q, k, v = _inputs(bsz, 1, hq, hkv, d, dtype, 70)
    kc, vc, pos = M.new_cache(plan, bsz)
    ws = M.new_workspace(plan, bsz)
    ws.fill_(0xFF)
    M.moa_kv_append(plan, kc, vc, pos, k, v, 0)
    o, buf = guarded_empty((bsz, hq, d), dtype)
    M.moa_decode(plan, q[:, 0].contiguous(), kc, vc, 0, ws, o)
    torch.cuda.synchronize()
    assert guard_intact(buf, (bsz, hq, d))
    want = v[:, 0].repeat_interleave(hq // hkv, dim=1)      # q head h reads KV head h // G
    assert torch.equal(bits(o), bits(want))


def test_decode_equals_prefill_row():
    _say("decode vs prefill row")
    bsz, hq, hkv, d, s, n = 2, 8, 2, 128, 8, 900
    windows = [50, 700]
    plan, _ = _plan(hq, hkv, d, s, n, "bf16", windows)
    q, k, v = _inputs(bsz, n, hq, hkv, d, torch.bfloat16, 60)
    o_pre = M.moa_prefill(plan, q, k, v)
    kc, vc, pos = M.new_cache(plan, bsz)
    ws = M.new_workspace(plan, bsz)
    M.moa_kv_append(plan, kc, vc, pos, k[:, : n - 1].contiguous(), v[:, : n - 1].contiguous(), 0)
    M.moa_kv_append(plan, kc, vc, pos, k[:, n - 1:].contiguous(), v[:, n - 1:].contiguous(), n - 1)
    o_dec = M.moa_decode(plan, q[:, n - 1].contiguous(), kc, vc, n - 1, ws)
    torch.cuda.synchronize()
    diff = (o_dec.float() - o_pre[:, n - 1].float()).abs().max().item()
    assert diff <= BF16_ATOL, diff


SPLIT_CASES = [
    # dtype, Hq, Hkv, D, sinks, windows, context
    ("bf16", 8, 8, 128, 16, [3000, 700, 1, 2999, 64, 1500, 2000, 10], 3000),   # vector-ALU kernel
    ("bf16", 16, 4, 128, 64, [2500, 90, 1200, 2048], 2600),                     # matrix cores, G = 4
    ("f32", 8, 2, 64, 4, [1900, 333], 2000),                                    # fp32, G = 4
]


@pytest.mark.parametrize("case", SPLIT_CASES, ids=lambda c: f"{c[0]}-hq{c[1]}-hkv{c[2]}-d{c[3]}")
def test_decode_does_not_depend_on_the_work_split(case):
    """A softmax over a set does not depend on how the set is partitioned
    (Eq. 1).  The same sequence's caches are decoded inside a batch of 32 and
    alone: the equal-work split over workers cuts its caches at different
    keys (about 15 workers for the sequence alone, hundreds for the batch), so
    the partial sums and their merge differ; the outputs must agree within the
    floating-point bar, and both must match the oracle."""
    dt, hq, hkv, d, s, windows, n = case
    _say("split invariance", case)
    dtype = DT[dt]
    bsz = 32
    plan, rw = _plan(hq, hkv, d, s, n, dt, windows)
    q, k, v = _inputs(bsz, n + 1, hq, hkv, d, dtype, 90)
    kc, vc, pos = M.new_cache(plan, bsz)
    M.moa_kv_append(plan, kc, vc, pos, k[:, :n].contiguous(), v[:, :n].contiguous(), 0)
    M.moa_kv_append(plan, kc, vc, pos, k[:, n:].contiguous(), v[:, n:].contiguous(), n)
    ws = M.new_workspace(plan, bsz)
    ws.fill_(0xFF)
    o_batch = M.moa_decode(plan, q[:, n].contiguous(), kc, vc, n, ws)
    ws1 = M.new_workspace(plan, 1)
    ws1.fill_(0xFF)
    tol = F32_ATOL if dtype == torch.float32 else BF16_ATOL
    for j in (0, 13, 31):
        o_one = M.moa_decode(plan, q[j:j + 1, n].contiguous(), kc[j:j + 1].clone(), vc[j:j + 1].clone(), n, ws1)
        torch.cuda.synchronize()
        diff = (o_one.double() - o_batch[j:j + 1].double()).abs().max().item()
        assert diff <= tol, f"sequence {j}: batch-of-32 vs alone differ by {diff}"
        ref = oracle.decode_ref(q[j:j + 1, n], k[j:j + 1], v[j:j + 1], rw, s)
        assert_close(o_one, ref, dtype, with_rounding=True, what=f"alone j={j}")
        assert_close(o_batch[j:j + 1], ref, dtype, with_rounding=True, what=f"in batch j={j}")
