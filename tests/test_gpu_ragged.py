"""Per-sequence positions in one batch (one-token append and decode), against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from helpers import assert_close, bits, oracle_windows
from paper_2406_14909_amd import moa as M

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("dt,hq,hkv,d,s,windows,lengths", [
    ("bf16", 8, 2, 128, 16, [40, 900], [5, 60, 1100, 0, 700]),
    ("f32", 4, 4, 64, 4, [1, 7, 600, 1500], [1300, 3, 17, 800]),
])
def test_ragged_append_and_decode(dt, hq, hkv, d, s, windows, lengths):
    _say("ragged", dt, lengths)
    dtype = torch.float32 if dt == "f32" else torch.bfloat16
    bsz, steps = len(lengths), 3
    plan = M.moa_plan(hq, hkv, d, s, max(max(windows), max(lengths)), dt, [float(w) for w in windows],
                      [0.0] * hkv)
    rw = oracle_windows(plan, windows, [0.0] * hkv)
    total = max(lengths) + steps
    q = workloads.randn((bsz, total, hq, d), 70, dtype, "cuda")
    k = workloads.randn((bsz, total, hkv, d), 71, dtype, "cuda")
    v = workloads.randn((bsz, total, hkv, d), 72, dtype, "cuda")
    kc, vc, pos = M.new_cache(plan, bsz)
    ws = M.new_workspace(plan, bsz)
    ws.fill_(0xFF)                                  # partials must never be read before written
    for b, n0 in enumerate(lengths):                # each sequence's own prompt
        if n0:
            M.moa_kv_append(plan, kc[b:b + 1], vc[b:b + 1], pos[b:b + 1], k[b:b + 1, :n0].contiguous(),
                            v[b:b + 1, :n0].contiguous(), 0)
    inactive = 1                                    # this sequence sits out every step
    cur = list(lengths)
    for step in range(steps):
        p = torch.tensor([-1 if b == inactive else cur[b] for b in range(bsz)], dtype=torch.int32,
                         device="cuda")
        kn = torch.stack([k[b, cur[b]] for b in range(bsz)]).unsqueeze(1).contiguous()
        vn = torch.stack([v[b, cur[b]] for b in range(bsz)]).unsqueeze(1).contiguous()
        qn = torch.stack([q[b, cur[b]] for b in range(bsz)]).contiguous()
        o = torch.full((bsz, hq, d), 7.0, dtype=dtype, device="cuda")
        M.moa_kv_append_ragged(plan, kc, vc, pos, kn, vn, p)
        M.moa_decode_ragged(plan, qn, kc, vc, p, ws, o)
        torch.cuda.synchronize()
        for b in range(bsz):
            if b == inactive:
                assert torch.all(o[b] == 7.0), "inactive sequence was written"
                continue
            t = cur[b]
            ref = oracle.decode_ref(q[b:b + 1, t], k[b:b + 1, : t + 1], v[b:b + 1, : t + 1], rw, s)
            assert_close(o[b:b + 1], ref, dtype, with_rounding=True, what=f"ragged b={b} t={t}")
        for b in range(bsz):
            if b != inactive:
                cur[b] += 1
    for b in range(bsz):
        n_done = cur[b]
        epos, ek, ev = oracle.cache_contents_ref(k[b:b + 1, :n_done].cpu(), v[b:b + 1, :n_done].cpu(),
                                                 rw, s)
        assert np.array_equal(pos[b:b + 1].cpu().numpy(), epos), f"pos table of sequence {b}"
        assert torch.equal(bits(kc[b:b + 1]), bits(ek)) and torch.equal(bits(vc[b:b + 1]), bits(ev))


def test_ragged_with_equal_positions_matches_uniform_bit_exactly():
    # With every cache full, both entry points split the same keys the same way.
    _say("ragged == uniform")
    bsz, hq, hkv, d, s, n0 = 3, 16, 4, 128, 64, 2100
    plan = M.moa_plan(hq, hkv, d, s, n0, "bf16", [100.0, 700.0, 1500.0, 2000.0], [0.0] * 4)
    assert n0 >= max(plan.capacity)
    k = workloads.randn((bsz, n0 + 1, hkv, d), 80, torch.bfloat16, "cuda")
    v = workloads.randn((bsz, n0 + 1, hkv, d), 81, torch.bfloat16, "cuda")
    q = workloads.randn((bsz, hq, d), 82, torch.bfloat16, "cuda")
    c1, c2 = M.new_cache(plan, bsz), M.new_cache(plan, bsz)
    for c in (c1, c2):
        M.moa_kv_append(plan, *c, k[:, :n0].contiguous(), v[:, :n0].contiguous(), 0)
    M.moa_kv_append(plan, *c1, k[:, n0:].contiguous(), v[:, n0:].contiguous(), n0)
    p = torch.full((bsz,), n0, dtype=torch.int32, device="cuda")
    M.moa_kv_append_ragged(plan, *c2, k[:, n0:].contiguous(), v[:, n0:].contiguous(), p)
    ws = M.new_workspace(plan, bsz)
    o1 = M.moa_decode(plan, q, c1[0], c1[1], n0, ws)
    o2 = M.moa_decode_ragged(plan, q, c2[0], c2[1], p, ws)
    torch.cuda.synchronize()
    for x, y in zip(c1, c2):
        assert torch.equal(bits(x), bits(y))
    assert torch.equal(bits(o1), bits(o2))


def test_long_context_batch1_decode_sampled():
    """The 128k-context batch-1 Vicuna-7B-shaped decode (mean window N/2)."""
    wl = workloads.workload("vicuna7b-decode-b1-ctx131072")
    _say("decode", wl.name)
    n, steps = wl.n, 2
    plan = M.moa_plan(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.num_sink, n, wl.dtype, wl.alpha, wl.beta)
    rw = oracle_windows(plan, wl.alpha, wl.beta)
    k = workloads.randn((1, n + steps, wl.num_kv_heads, wl.head_dim), 90, torch.bfloat16, "cuda")
    v = workloads.randn((1, n + steps, wl.num_kv_heads, wl.head_dim), 91, torch.bfloat16, "cuda")
    q = workloads.randn((steps, 1, wl.num_q_heads, wl.head_dim), 92, torch.bfloat16, "cuda")
    kc, vc, pos = M.new_cache(plan, 1)
    ws = M.new_workspace(plan, 1)
    M.moa_kv_append(plan, kc, vc, pos, k[:, :n].contiguous(), v[:, :n].contiguous(), 0)
    outs = []
    for i in range(steps):
        t = n + i
        M.moa_kv_append(plan, kc, vc, pos, k[:, t:t + 1].contiguous(), v[:, t:t + 1].contiguous(), t)
        outs.append(M.moa_decode(plan, q[i], kc, vc, t, ws))
    torch.cuda.synchronize()
    for g in range(0, wl.num_kv_heads, 3):
        kb, vb = k[:, :, g:g + 1].cpu(), v[:, :, g:g + 1].cpu()
        for i in range(steps):
            t = n + i
            ref = oracle.decode_ref(q[i, :, g:g + 1].cpu(), kb[:, : t + 1], vb[:, : t + 1],
                                    [rw[g]], wl.num_sink)
            assert_close(outs[i][:, g:g + 1], ref, torch.bfloat16, what=f"128k t={t} h={g}")
