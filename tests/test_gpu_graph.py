"""The serving decode step captured in a HIP graph and replayed as a decode
loop (paper App. B.2: the decode path over per-head caches).

One step is the one-token append at each sequence's own position, the decode
at those positions and the positions' increment on the device, so a single
captured graph serves every step of the loop.  Each replay runs with the
test's own eager copies and a synchronisation around it, and must equal, bit
for bit, the same step run eagerly on a twin cache: the kernels, their
launch shapes and the work split do not depend on the positions."""
import pytest
import torch

import workloads
from paper_2406_14909_amd import moa as M

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("hq,hkv", [(8, 2), (4, 4)])
def test_graph_replays_equal_eager_steps(hq, hkv):
    _say("graph decode loop", hq, hkv)
    bsz, d, s, n0, steps = 3, 128, 4, 64, 6
    windows = [40, 300] if hkv == 2 else [1, 40, 300, 70]
    plan = M.moa_plan(hq, hkv, d, s, 512, "bf16", [float(w) for w in windows], [0.0] * hkv)
    total = n0 + steps
    k = workloads.randn((bsz, total, hkv, d), 71, torch.bfloat16, "cuda")
    v = workloads.randn((bsz, total, hkv, d), 72, torch.bfloat16, "cuda")
    q = workloads.randn((bsz, total, hq, d), 73, torch.bfloat16, "cuda")

    def fresh_cache():
        kc, vc, pos = M.new_cache(plan, bsz)
        M.moa_kv_append(plan, kc, vc, pos, k[:, :n0].contiguous(), v[:, :n0].contiguous(), 0)
        return kc, vc, pos

    # Static buffers the graph reads and writes.
    k_step = torch.empty((bsz, 1, hkv, d), dtype=torch.bfloat16, device="cuda")
    v_step = torch.empty_like(k_step)
    q_step = torch.empty((bsz, hq, d), dtype=torch.bfloat16, device="cuda")

    def load_step(t):
        k_step.copy_(k[:, n0 + t:n0 + t + 1])
        v_step.copy_(v[:, n0 + t:n0 + t + 1])
        q_step.copy_(q[:, n0 + t])

    # Eager reference.
    kc_e, vc_e, pos_e = fresh_cache()
    positions_e = torch.full((bsz,), n0, dtype=torch.int32, device="cuda")
    ws_e = M.new_workspace(plan, bsz)
    o_e = torch.empty((bsz, hq, d), dtype=torch.bfloat16, device="cuda")
    expected = []
    for t in range(steps):
        load_step(t)
        M.moa_kv_append_ragged(plan, kc_e, vc_e, pos_e, k_step, v_step, positions_e)
        M.moa_decode_ragged(plan, q_step, kc_e, vc_e, positions_e, ws_e, o_e)
        positions_e.add_(1)
        expected.append(o_e.clone())
    torch.cuda.synchronize()

    # Captured step.
    kc_g, vc_g, pos_g = fresh_cache()
    positions_g = torch.full((bsz,), n0, dtype=torch.int32, device="cuda")
    ws_g = M.new_workspace(plan, bsz)
    o_g = torch.empty((bsz, hq, d), dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        M.moa_kv_append_ragged(plan, kc_g, vc_g, pos_g, k_step, v_step, positions_g)
        M.moa_decode_ragged(plan, q_step, kc_g, vc_g, positions_g, ws_g, o_g)
        positions_g.add_(1)
    torch.cuda.synchronize()
    # Capture records without running: the state is still the prefilled one.
    assert torch.equal(positions_g, torch.full_like(positions_g, n0))

    for t in range(steps):
        load_step(t)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_g, expected[t]), f"replay {t} differs from the eager step"
    assert torch.equal(positions_g, positions_e)
    assert torch.equal(pos_g, pos_e)
    assert torch.equal(kc_g, kc_e) and torch.equal(vc_g, vc_e)
