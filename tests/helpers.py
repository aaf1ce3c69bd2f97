"""Shared helpers of the GPU parity tests (tolerances, canaries, bit checks)."""
import numpy as np
import torch

# Floating-point bars: fp32 path max-abs 1e-5; bf16 inputs with fp32
# accumulation max-abs 1e-2.  Where a test deliberately produces outputs of
# magnitude > 1 (tiny windows), the bf16 bar adds, for those outputs only, the
# output rounding of the stored result, 2^-8 * |ref| (half an ulp of an 8-bit
# significand); every output of magnitude <= 1 keeps the plain 1e-2.
F32_ATOL = 1e-5
BF16_ATOL = 1e-2
BF16_ROUND_REL = 2.0 ** -8

SENTINEL = 12288.0   # exactly representable in bf16 and fp32


def assert_close(gpu, ref, dtype, with_rounding=False, what=""):
    got = gpu.detach().to("cpu", torch.float64).numpy()
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - ref)
    if dtype == torch.float32:
        bound = np.full_like(ref, F32_ATOL)
    else:
        big = np.abs(ref) > 1.0
        bound = BF16_ATOL + (np.where(big, BF16_ROUND_REL * np.abs(ref), 0.0) if with_rounding else 0.0)
    bad = err > bound
    if bad.any():
        idx = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: max err {err.max():.3e} at {idx} (got {got[idx]}, ref {ref[idx]}, "
                             f"bound {np.broadcast_to(bound, err.shape)[idx]:.3e}); {bad.sum()} bad")
    return float(err.max())


def oracle_windows(plan, alpha, beta, span_includes_sinks=False):
    """The oracle's windows for the plan's rule (oracle.plan_ref on the same
    alpha, beta, N and sinks).  Parity tests hand these, never the library's
    own table, to the oracle, so a wrong plan cannot cancel out of a GPU
    comparison; the library's table must match them exactly."""
    import oracle

    ref = oracle.plan_ref([float(a) for a in alpha], [float(b) for b in beta], int(plan.desc.n),
                          int(plan.num_sink), span_includes_sinks)["window"]
    assert np.array_equal(np.asarray(plan.window), ref), (list(plan.window), list(ref))
    return [int(x) for x in ref]


def guarded_empty(shape, dtype, device="cuda", guard=4096):
    """Tensor of `shape` followed by a sentinel-filled guard region."""
    n = int(np.prod(shape))
    buf = torch.full((n + guard,), SENTINEL, dtype=dtype, device=device)
    return buf[:n].view(*shape), buf


def guard_intact(buf, shape):
    n = int(np.prod(shape))
    tail = buf[n:].cpu()
    return bool(torch.all(tail == torch.tensor(SENTINEL, dtype=buf.dtype)))


def bits(t):
    """Integer view of a tensor for bit-exact comparison."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16)
    if t.dtype == torch.float32:
        return t.view(torch.int32)
    return t
