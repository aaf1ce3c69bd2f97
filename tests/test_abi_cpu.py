"""C-ABI checks that need no GPU: exported symbols, plan tables, error paths.

Only host-side calls are made here (moa_plan and argument validation, which
returns before any launch).
"""
import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT
import oracle
from paper_2406_14909_amd import moa as M

lib = M.load_library()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "moa.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(moa_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert set(names) == set(M.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def test_desc_struct_layout_matches_header():
    assert ctypes.sizeof(M.moa_desc_t) == 40
    assert M.moa_desc_t.n.offset == 16 and M.moa_desc_t.softmax_scale.offset == 28
    assert M.moa_desc_t.flags.offset == 32 and M.moa_desc_t.reserved.offset == 36
    text = open(os.path.join(ROOT, "include", "moa.h")).read()
    for name in ("MOA_SPAN_INCLUDES_SINKS", "MOA_BLOCK_BAND", "MOA_BAND_BLOCK"):
        assert int(re.search(rf"#define {name} (\d+)", text).group(1)) == getattr(M, name)


def _plan(alpha, beta, n, s=64, hq=None, hkv=None, d=128, dtype="bf16"):
    hkv = hkv or len(alpha)
    return M.moa_plan(hq or hkv, hkv, d, s, n, dtype, alpha, beta)


@pytest.mark.parametrize("seed", range(6))
def test_plan_tables_equal_oracle_plan_bit_exact(seed):
    rng = np.random.default_rng(seed)
    hkv = int(rng.integers(1, 65))
    n = int(rng.integers(1, 1 << 20))
    s = int(rng.integers(0, 200))
    alpha = rng.uniform(-2048, 8192, hkv)
    beta = rng.uniform(0, 1, hkv)
    # exact edge values in the sampled domain
    alpha[: min(hkv, 4)] = [-2048.0, 0.0, 8192.0, 64.5][: min(hkv, 4)]
    p = _plan(alpha, beta, n, s)
    ref = oracle.plan_ref(alpha, beta, n, s)
    assert np.array_equal(p.window, ref["window"])
    assert np.array_equal(p.capacity, ref["capacity"])
    assert np.array_equal(p.offset, ref["offset"])
    assert p.cache_rows == int(ref["offset"][-1])


@pytest.mark.parametrize("seed", range(4))
def test_span_includes_sinks_plan_tables_equal_oracle_bit_exact(seed):
    rng = np.random.default_rng(100 + seed)
    hkv = int(rng.integers(1, 65))
    n = int(rng.integers(1, 1 << 20))
    s = int(rng.integers(0, 300))
    alpha = rng.uniform(-2048, 8192, hkv)
    beta = rng.uniform(0, 1, hkv)
    alpha[: min(hkv, 4)] = [-2048.0, 0.0, float(s), float(s) + 0.5][: min(hkv, 4)]
    for flags in (M.MOA_SPAN_INCLUDES_SINKS, M.MOA_SPAN_INCLUDES_SINKS | M.MOA_BLOCK_BAND):
        p = M.moa_plan(hkv, hkv, 128, s, n, "bf16", alpha, beta, flags=flags)
        ref = oracle.plan_ref(alpha, beta, n, s, span_includes_sinks=True)
        assert np.array_equal(p.window, ref["window"])
        assert np.array_equal(p.capacity, ref["capacity"])
        assert np.array_equal(p.offset, ref["offset"])
    # the block band changes only prefill's mask, never the tables
    q = M.moa_plan(hkv, hkv, 128, s, n, "bf16", alpha, beta, flags=M.MOA_BLOCK_BAND)
    assert np.array_equal(q.window, oracle.plan_ref(alpha, beta, n, s)["window"])


def test_plan_rejects_unknown_flags():
    for flags, reserved in ((4, 0), (1 << 31, 0), (0, 1)):
        desc = M.moa_desc_t(4, 4, 128, 4, 512, M.MOA_BF16, 0.0, flags, reserved)
        a = (ctypes.c_double * 4)(*([16.0] * 4))
        out = ctypes.c_void_p(1)
        assert lib.moa_plan(ctypes.byref(desc), a, a, ctypes.byref(out)) == M.MOA_ERR_INVALID_ARG
        assert out.value is None


def test_plan_rounding_edges():
    # values whose floor is sensitive to rounding of alpha + beta * N
    n = 3
    alpha = [0.1, 1.0 - 2 ** -52, 2.0, -0.0, 1e300, -1e300]
    beta = [0.3, 0.0, 1.0 / 3.0, 0.5, 0.0, 1.0]
    p = _plan(alpha, beta, n, 0, d=64, dtype="f32")
    ref = oracle.plan_ref(alpha, beta, n, 0)
    assert np.array_equal(p.window, ref["window"])


def test_workload_plans_match_oracle():
    import workloads
    for wl in workloads.workloads():
        p = M.moa_plan(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.num_sink, wl.n, wl.dtype,
                       wl.alpha, wl.beta)
        ref = oracle.plan_ref(wl.alpha, wl.beta, wl.n, wl.num_sink)
        assert np.array_equal(p.window, ref["window"]), wl.name
        assert np.array_equal(p.offset, ref["offset"]), wl.name


@pytest.mark.parametrize("kw,status", [
    (dict(hkv=0), M.MOA_ERR_INVALID_ARG),
    (dict(hkv=65), M.MOA_ERR_INVALID_ARG),
    (dict(hq=6, hkv=4), M.MOA_ERR_INVALID_ARG),
    (dict(hq=12, hkv=4), M.MOA_ERR_UNSUPPORTED),
    (dict(hq=64, hkv=4), M.MOA_ERR_UNSUPPORTED),
    (dict(d=96), M.MOA_ERR_UNSUPPORTED),
    (dict(s=-1), M.MOA_ERR_INVALID_ARG),
    (dict(n=0), M.MOA_ERR_INVALID_ARG),
    (dict(n=1 << 30), M.MOA_ERR_INVALID_ARG),
    (dict(dtype=7), M.MOA_ERR_INVALID_ARG),
    (dict(scale=-1.0), M.MOA_ERR_INVALID_ARG),
    (dict(scale=float("nan")), M.MOA_ERR_INVALID_ARG),
    (dict(alpha=float("inf")), M.MOA_ERR_INVALID_ARG),
    (dict(beta=float("nan")), M.MOA_ERR_INVALID_ARG),
])
def test_plan_rejects_invalid_descriptors(kw, status):
    hkv = kw.get("hkv", 4)
    desc = M.moa_desc_t(kw.get("hq", hkv), hkv, kw.get("d", 128), kw.get("s", 4), kw.get("n", 512),
                        kw.get("dtype", M.MOA_BF16), kw.get("scale", 0.0))
    m = max(hkv, 1)
    a = (ctypes.c_double * m)(*([kw.get("alpha", 16.0)] * m))
    b = (ctypes.c_double * m)(*([kw.get("beta", 0.5)] * m))
    out = ctypes.c_void_p(1)
    assert lib.moa_plan(ctypes.byref(desc), a, b, ctypes.byref(out)) == status
    assert out.value is None
    assert lib.moa_last_error().decode().startswith("moa_plan")


def test_plan_null_arguments():
    out = ctypes.c_void_p()
    assert lib.moa_plan(None, None, None, ctypes.byref(out)) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_plan_tables(None, None, None, None) == M.MOA_ERR_INVALID_ARG
    lib.moa_plan_free(None)
    assert lib.moa_decode_workspace_bytes(None, 4) == 0


def test_gpu_entry_points_validate_before_launch():
    # Every call below is invalid and must return before touching the GPU.
    p = _plan([100.0, 200.0], [0.0, 0.0], 1024, 4, hq=4, hkv=2)
    h = p.handle
    fake = 1 << 20          # aligned non-null address, never dereferenced
    st = lib.moa_prefill(h, None, fake, fake, fake, 1, 16, None)
    assert st == M.MOA_ERR_INVALID_ARG and "null" in lib.moa_last_error().decode()
    assert lib.moa_prefill(None, fake, fake, fake, fake, 1, 16, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_prefill(h, fake, fake, fake, fake + 1 << 30, 0, 16, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_prefill(h, fake, fake, fake, fake, 1, 0, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_prefill(h, fake + 8, fake, fake, fake, 1, 16, None) == M.MOA_ERR_INVALID_ARG
    st = lib.moa_prefill(h, fake, 2 * fake, 3 * fake, fake + 64, 1, 16, None)
    assert st == M.MOA_ERR_INVALID_ARG and "overlap" in lib.moa_last_error().decode()

    assert lib.moa_kv_append(h, fake, fake, fake, None, fake, 1, 0, 1, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_kv_append(h, fake, fake, fake, fake, fake, 0, 0, 1, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_kv_append(h, fake, fake, fake, fake, fake, 70000, 0, 1, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_kv_append(h, fake, fake, fake, fake, fake, 1, -1, 1, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_kv_append(h, fake, fake, fake, fake, fake, 1, 0, 0, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_kv_append(h, fake, fake, fake, fake, fake, 1, (1 << 31) - 1, 1, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_kv_append(h, fake, fake, fake + 2, fake, fake, 1, 0, 1, None) == M.MOA_ERR_INVALID_ARG

    need = lib.moa_decode_workspace_bytes(h, 2)
    assert need > 0
    assert lib.moa_decode(h, fake, fake, fake, fake, 2, 0, None, need, None) == M.MOA_ERR_WORKSPACE
    assert lib.moa_decode(h, fake, fake, fake, fake, 2, 0, fake, need - 1, None) == M.MOA_ERR_WORKSPACE
    assert lib.moa_decode(h, fake, fake, fake, fake, 2, 0, fake + 16, need, None) == M.MOA_ERR_WORKSPACE
    assert lib.moa_decode(h, fake, fake, fake, fake, 2, -1, fake, need, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_decode(h, fake, fake, fake, fake, 0, 0, fake, need, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_decode(h, None, fake, fake, fake, 2, 0, fake, need, None) == M.MOA_ERR_INVALID_ARG
    # Written buffers (o, workspace) may not overlap anything else.
    q, kc, vc, ws, o = 1 << 20, 1 << 28, 1 << 29, 1 << 30, 3 << 30
    for args in ((q, kc, vc, q + 16, ws), (q, kc, vc, kc + 4096, ws), (q, kc, vc, ws + 256, ws),
                 (q, kc, vc, o, kc + 256), (q, kc, vc, o, q)):
        st = lib.moa_decode(h, *args[:4], 2, 0, args[4], need, None)
        assert st == M.MOA_ERR_INVALID_ARG and "overlap" in lib.moa_last_error().decode(), args


def test_noalloc_decode_validates_before_launch():
    # Invalid calls return before any HIP call; a plan and batch whose partials
    # exceed the library's own array are refused with MOA_ERR_WORKSPACE.
    p = _plan([100.0, 200.0], [0.0, 0.0], 1024, 4, hq=4, hkv=2)
    h = p.handle
    fake = 1 << 20
    assert lib.moa_decode_noalloc(None, fake, fake, fake, fake, 2, 0, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_decode_noalloc(h, None, fake, fake, fake, 2, 0, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_decode_noalloc(h, fake, fake, fake, fake, 0, 0, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_decode_noalloc(h, fake, fake, fake, fake, 2, -1, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_decode_noalloc(h, fake + 8, fake, fake, fake, 2, 0, None) == M.MOA_ERR_INVALID_ARG
    g8 = _plan([1.0] * 8, [0.0] * 8, 4, 0, hq=64, hkv=8)
    assert M.moa_decode_workspace_bytes(g8, 961) <= M.MOA_DECODE_SCRATCH_BYTES    # 961 * 8 = 7688
    assert M.moa_decode_workspace_bytes(g8, 962) > M.MOA_DECODE_SCRATCH_BYTES   # 962 * 8 = 7696
    st = lib.moa_decode_noalloc(g8.handle, fake, 2 * fake, 3 * fake, 4 * fake, 962, 0, None)
    assert st == M.MOA_ERR_WORKSPACE and "moa_decode with a caller-owned workspace" in lib.moa_last_error().decode()
    text = open(os.path.join(ROOT, "include", "moa.h")).read()
    assert int(re.search(r"#define MOA_DECODE_SCRATCH_BYTES \((\d+)u << (\d+)\)", text).group(1)) << 20 == \
        M.MOA_DECODE_SCRATCH_BYTES


def test_decode_workspace_size():
    # Partials for at most 8192 workers plus one per (sequence, KV head), each
    # group x (head_dim + 4) floats; independent of the cache lengths.
    small = _plan([100.0, 200.0], [0.0, 0.0], 1024, 4, hq=4, hkv=2)
    big = _plan([5000.0, 200.0], [0.0, 0.0], 8192, 4, hq=4, hkv=2)
    for p in (small, big):
        for bsz in (1, 2, 8):
            assert M.moa_decode_workspace_bytes(p, bsz) == (8192 + bsz * 2) * 2 * (128 + 4) * 4
    gqa = _plan([float(1 << 27)], [0.0], 1 << 29, 64, hq=8, hkv=1, d=64)
    assert M.moa_decode_workspace_bytes(gqa, 3) == (8192 + 3) * 8 * (64 + 4) * 4


def test_binding_fails_loudly_without_library(tmp_path):
    import importlib
    saved = M._lib
    try:
        M._lib = None
        with pytest.raises(ImportError):
            M.load_library(str(tmp_path / "missing.so"))
    finally:
        M._lib = saved


def test_library_resolves_all_of_its_own_symbols():
    # Every kernel stub and entry point must be defined inside libmoa.so itself.
    import subprocess
    out = subprocess.run(["nm", "-D", "--undefined-only", M.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    own = [line for line in out.splitlines() if "moa" in line]
    assert own == [], own


def test_ragged_entry_points_validate_before_launch():
    p = _plan([100.0, 200.0], [0.0, 0.0], 1024, 4, hq=4, hkv=2)
    h = p.handle
    fake = 1 << 20
    need = lib.moa_decode_workspace_bytes(h, 2)
    assert lib.moa_kv_append_ragged(h, fake, fake, fake, fake, fake, None, 2, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_kv_append_ragged(h, fake, fake, fake, fake, fake, fake + 2, 2, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_kv_append_ragged(h, fake, fake, fake, fake, fake, fake, 0, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_decode_ragged(h, fake, fake, fake, fake, None, 2, fake, need, None) == M.MOA_ERR_INVALID_ARG
    assert lib.moa_decode_ragged(h, fake, fake, fake, fake, fake, 2, fake, need - 1, None) == M.MOA_ERR_WORKSPACE
    assert lib.moa_decode_ragged(h, fake, fake, fake, fake, fake, 0, fake, need, None) == M.MOA_ERR_INVALID_ARG
    q, kc, vc, ws = 1 << 20, 1 << 28, 1 << 29, 1 << 30
    st = lib.moa_decode_ragged(h, q, kc, vc, q + 16, fake, 2, ws, need, None)
    assert st == M.MOA_ERR_INVALID_ARG and "overlap" in lib.moa_last_error().decode()


def test_influence_validates_before_launch():
    fake = 1 << 20
    def call(desc=None, q=fake, ebar=fake, batch=1, n=128):
        d = desc or M.moa_desc_t(4, 2, 128, 0, 0, M.MOA_BF16, 0.0, 0, 0)
        return lib.moa_influence(ctypes.byref(d), q, fake, fake, fake, ebar, batch, n, None)
    assert call(q=None) == M.MOA_ERR_INVALID_ARG
    assert call(desc=M.moa_desc_t(4, 2, 128, 0, 0, M.MOA_F32, 0.0, 0, 0)) == M.MOA_ERR_UNSUPPORTED
    assert call(desc=M.moa_desc_t(4, 2, 96, 0, 0, M.MOA_BF16, 0.0, 0, 0)) == M.MOA_ERR_UNSUPPORTED
    assert call(desc=M.moa_desc_t(5, 2, 128, 0, 0, M.MOA_BF16, 0.0, 0, 0)) == M.MOA_ERR_INVALID_ARG
    assert call(n=65537) == M.MOA_ERR_UNSUPPORTED
    assert call(n=0) == M.MOA_ERR_INVALID_ARG
    assert call(batch=0) == M.MOA_ERR_INVALID_ARG
    assert call(q=fake + 8) == M.MOA_ERR_INVALID_ARG
    assert call(ebar=fake + 2) == M.MOA_ERR_INVALID_ARG
    assert "moa_influence" in lib.moa_last_error().decode()



def test_binding_rejects_tensors_on_different_devices():
    import torch
    a, b = torch.zeros(4), torch.zeros(4, device="meta")
    with pytest.raises(M.MoaError) as e:
        M._one_device(q=a, k=b)
    assert "different devices" in str(e.value)
    assert M._one_device(q=a, k=torch.ones(2)) == a.device
