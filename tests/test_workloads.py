"""Seeded workload generators: determinism and the rescaled mean window."""
import numpy as np
import torch

import workloads
from oracle import plan_ref


def test_rules_hit_target_mean_window():
    for wl in workloads.workloads()[1:]:
        p = plan_ref(wl.alpha, wl.beta, wl.n, wl.num_sink)
        target = (0.25 if "70b" in wl.name else 0.5) * wl.n
        assert abs(p["window"].mean() - target) <= 1.0, wl.name
        assert p["window"].min() >= 1 and p["window"].max() <= wl.n


def test_rules_and_tensors_are_deterministic():
    a1, b1 = workloads.sample_rules(7, 8, 4096, 2048.0)
    a2, b2 = workloads.sample_rules(7, 8, 4096, 2048.0)
    assert np.array_equal(a1, a2) and np.array_equal(b1, b2)
    x1 = workloads.randn((3, 5), 11, torch.bfloat16)
    x2 = workloads.randn((3, 5), 11, torch.bfloat16)
    assert torch.equal(x1, x2) and x1.dtype == torch.bfloat16


def test_small_workload_shape():
    wl = workloads.workload(0)
    assert (wl.num_q_heads, wl.head_dim, wl.n, wl.num_sink, wl.dtype) == (4, 64, 512, 4, "f32")
    assert list(plan_ref(wl.alpha, wl.beta, wl.n, wl.num_sink)["window"]) == [64, 128, 256, 512]
