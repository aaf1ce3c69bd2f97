"""moa_decode_noalloc (the decode entry point that allocates nothing and keeps
its split-K partials in the library's own per-GPU array) against moa_decode
with a caller workspace: the same kernels and work split, so the outputs must
be bit-identical, and both must match the oracle.  Two calls in a row, the
second on a smaller input, so leftovers of the first call in the shared array
cannot leak into the second."""
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


def _filled(hq, hkv, d, s, windows, n, bsz, dt, seed):
    dtype = torch.bfloat16 if dt == "bf16" else torch.float32
    alpha, beta = [float(w) for w in windows], [0.0] * hkv
    plan = M.moa_plan(hq, hkv, d, s, n, dt, alpha, beta)
    rw = oracle_windows(plan, alpha, beta)
    q = workloads.randn((bsz, hq, d), seed, dtype, "cuda")
    k = workloads.randn((bsz, n + 1, hkv, d), seed + 1, dtype, "cuda")
    v = workloads.randn((bsz, n + 1, hkv, d), seed + 2, dtype, "cuda")
    kc, vc, pos = M.new_cache(plan, bsz)
    M.moa_kv_append(plan, kc, vc, pos, k[:, :n].contiguous(), v[:, :n].contiguous(), 0)
    M.moa_kv_append(plan, kc, vc, pos, k[:, n:].contiguous(), v[:, n:].contiguous(), n)
    return plan, rw, q, k, v, kc, vc, dtype


CALLS = [
    # (dtype, Hq, Hkv, D, sinks, windows, context, batch): the second is smaller
    [("bf16", 32, 8, 128, 64, [5000, 100, 2500, 1, 4000, 64, 1300, 3000], 5000, 16),
     ("bf16", 8, 2, 128, 4, [300, 40], 350, 2)],
    [("bf16", 32, 32, 128, 64, [3000, 17, 900, 2999, 1, 1500, 333, 2000] * 4, 3000, 8),
     ("f32", 4, 4, 64, 2, [1, 7, 200, 64], 250, 3)],
]


@pytest.mark.parametrize("calls", CALLS, ids=["gqa-then-small", "mha-then-fp32"])
def test_noalloc_decode_matches_workspace_decode(calls):
    for i, (dt, hq, hkv, d, s, windows, n, bsz) in enumerate(calls):
        _say("noalloc call", i, dt, hq, hkv, d, s, n, bsz)
        plan, rw, q, k, v, kc, vc, dtype = _filled(hq, hkv, d, s, windows, n, bsz, dt, 300 + 10 * i)
        assert M.moa_decode_workspace_bytes(plan, bsz) <= M.MOA_DECODE_SCRATCH_BYTES
        ws = M.new_workspace(plan, bsz)
        ws.fill_(0xFF)
        o_ws = M.moa_decode(plan, q, kc, vc, n, ws)
        o_na = torch.full_like(q, 7.0)
        M.moa_decode_noalloc(plan, q, kc, vc, n, o_na)
        torch.cuda.synchronize()
        assert torch.equal(bits(o_na), bits(o_ws)), f"call {i}: noalloc and workspace decode differ"
        sample = sorted({0, bsz - 1})
        ref = oracle.decode_ref(q[sample], k[sample], v[sample], rw, s)
        assert_close(o_na[sample], ref, dtype, with_rounding=True, what=f"noalloc call {i}")


def test_noalloc_rejects_more_than_its_array():
    # group 8, head_dim 128: (8192 + batch * num_kv_heads) * 8 * 132 * 4 bytes
    # fit in 64 MiB only while batch * num_kv_heads <= 7695.
    plan = M.moa_plan(64, 8, 128, 0, 4, "bf16", [1.0] * 8, [0.0] * 8)
    bsz = 1000
    assert M.moa_decode_workspace_bytes(plan, bsz) > M.MOA_DECODE_SCRATCH_BYTES
    q = torch.zeros((bsz, 64, 128), dtype=torch.bfloat16, device="cuda")
    kc, vc, _ = M.new_cache(plan, bsz)
    o = torch.full_like(q, 7.0)
    with pytest.raises(M.MoaError) as e:
        M.moa_decode_noalloc(plan, q, kc, vc, 0, o)
    assert e.value.status == M.MOA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.all(o == 7.0)
