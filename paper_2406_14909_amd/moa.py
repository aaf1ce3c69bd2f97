"""Thin ctypes binding of libmoa.so with the same names as the C ABI.

Argument marshalling only: shapes and dtypes of torch tensors are checked and
their device pointers, together with torch's current HIP stream, are handed to
the library.  Every step of the computation runs in the library's kernels;
there is no fallback.  If libmoa.so is missing, loading fails with an error.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libmoa.so")

MOA_OK, MOA_ERR_INVALID_ARG, MOA_ERR_UNSUPPORTED, MOA_ERR_WORKSPACE, MOA_ERR_HIP = range(5)
MOA_F32, MOA_BF16 = 0, 1
MOA_MAX_KV_HEADS = 64
MOA_MAX_Q_HEADS = 512

EXPORTED = (
    "moa_plan", "moa_plan_tables", "moa_plan_free", "moa_prefill", "moa_kv_append",
    "moa_decode_workspace_bytes", "moa_decode", "moa_last_error", "moa_kv_append_ragged",
    "moa_decode_ragged", "moa_influence", "moa_rule_loss", "moa_decode_noalloc",
)


class moa_desc_t(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("num_sink", ctypes.c_int32),
        ("n", ctypes.c_int64),
        ("dtype", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("flags", ctypes.c_uint32),
        ("reserved", ctypes.c_uint32),
    ]


MOA_SPAN_INCLUDES_SINKS = 1
MOA_BLOCK_BAND = 2
MOA_BAND_BLOCK = 64


class MoaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[moa status {status}] {message}")
        self.status = status


_lib = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Loads libmoa.so once.  torch is imported first so that the library
    binds to the same HIP runtime instance as torch (same soname)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (shares its HIP runtime with the library)

    path = path or LIB_PATH
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2406_14909_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.moa_plan.argtypes = [ctypes.POINTER(moa_desc_t), ctypes.POINTER(ctypes.c_double),
                             ctypes.POINTER(ctypes.c_double), ctypes.POINTER(vp)]
    lib.moa_plan.restype = ctypes.c_int
    lib.moa_plan_tables.argtypes = [vp, vp, vp, vp]
    lib.moa_plan_tables.restype = ctypes.c_int
    lib.moa_plan_free.argtypes = [vp]
    lib.moa_plan_free.restype = None
    lib.moa_prefill.argtypes = [vp, vp, vp, vp, vp, i32, i64, vp]
    lib.moa_prefill.restype = ctypes.c_int
    lib.moa_kv_append.argtypes = [vp, vp, vp, vp, vp, vp, i32, i64, i64, vp]
    lib.moa_kv_append.restype = ctypes.c_int
    lib.moa_decode_workspace_bytes.argtypes = [vp, i32]
    lib.moa_decode_workspace_bytes.restype = ctypes.c_size_t
    lib.moa_decode.argtypes = [vp, vp, vp, vp, vp, i32, i64, vp, ctypes.c_size_t, vp]
    lib.moa_decode.restype = ctypes.c_int
    lib.moa_kv_append_ragged.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, vp]
    lib.moa_kv_append_ragged.restype = ctypes.c_int
    lib.moa_decode_noalloc.argtypes = [vp, vp, vp, vp, vp, i32, i64, vp]
    lib.moa_decode_noalloc.restype = ctypes.c_int
    lib.moa_decode_ragged.argtypes = [vp, vp, vp, vp, vp, vp, i32, vp, ctypes.c_size_t, vp]
    lib.moa_decode_ragged.restype = ctypes.c_int
    lib.moa_influence.argtypes = [ctypes.POINTER(moa_desc_t), vp, vp, vp, vp, vp, i32, i64, vp]
    lib.moa_influence.restype = ctypes.c_int
    lib.moa_rule_loss.argtypes = [vp, i32, i64, i32, ctypes.c_uint32, ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(ctypes.c_double), i32, vp, vp, vp]
    lib.moa_rule_loss.restype = ctypes.c_int
    lib.moa_last_error.argtypes = []
    lib.moa_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != MOA_OK:
        raise MoaError(status, load_library().moa_last_error().decode())


class Plan:
    """Owns a moa_plan_t* and its host copies of the per-KV-head tables."""

    def __init__(self, handle: int, desc: moa_desc_t):
        self.handle = ctypes.c_void_p(handle)
        self.desc = desc
        hkv = desc.num_kv_heads
        self.window = np.zeros(hkv, dtype=np.int32)
        self.capacity = np.zeros(hkv, dtype=np.int32)
        self.offset = np.zeros(hkv + 1, dtype=np.int64)
        _check(load_library().moa_plan_tables(self.handle, self.window.ctypes.data,
                                              self.capacity.ctypes.data, self.offset.ctypes.data))

    @property
    def num_q_heads(self) -> int:
        return self.desc.num_q_heads

    @property
    def num_kv_heads(self) -> int:
        return self.desc.num_kv_heads

    @property
    def head_dim(self) -> int:
        return self.desc.head_dim

    @property
    def num_sink(self) -> int:
        return self.desc.num_sink

    @property
    def cache_rows(self) -> int:
        return int(self.offset[-1])

    @property
    def torch_dtype(self):
        import torch
        return torch.bfloat16 if self.desc.dtype == MOA_BF16 else torch.float32

    def free(self) -> None:
        if self.handle is not None and self.handle.value:
            load_library().moa_plan_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def moa_plan(num_q_heads: int, num_kv_heads: int, head_dim: int, num_sink: int, n: int,
             dtype: str, alpha: Sequence[float], beta: Sequence[float],
             softmax_scale: float = 0.0, flags: int = 0) -> Plan:
    """Builds the per-KV-head window / capacity / offset tables (host only).

    flags: MOA_SPAN_INCLUDES_SINKS and/or MOA_BLOCK_BAND (see include/moa.h)."""
    lib = load_library()
    desc = moa_desc_t(int(num_q_heads), int(num_kv_heads), int(head_dim), int(num_sink), int(n),
                      MOA_BF16 if dtype in ("bf16", "bfloat16") else MOA_F32, float(softmax_scale),
                      int(flags), 0)
    a = np.ascontiguousarray(alpha, dtype=np.float64)
    b = np.ascontiguousarray(beta, dtype=np.float64)
    if a.shape != (num_kv_heads,) or b.shape != (num_kv_heads,):
        raise MoaError(MOA_ERR_INVALID_ARG, "alpha and beta need num_kv_heads entries")
    out = ctypes.c_void_p()
    _check(lib.moa_plan(ctypes.byref(desc), a.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                        b.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), ctypes.byref(out)))
    return Plan(out.value, desc)


def _stream(t, stream) -> ctypes.c_void_p:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(t.device)
    return ctypes.c_void_p(stream.cuda_stream)


def _one_device(**tensors):
    """The GPU that every tensor of a call lives on; the call runs with it as
    the current device (raises if the tensors are spread over devices)."""
    devs = {t.device for t in tensors.values()}
    if len(devs) != 1:
        raise MoaError(MOA_ERR_INVALID_ARG, "tensors on different devices: " +
                       ", ".join(f"{k} on {t.device}" for k, t in tensors.items()))
    return devs.pop()


def _need(t, shape, dtype, name):
    if tuple(t.shape) != tuple(shape):
        raise MoaError(MOA_ERR_INVALID_ARG, f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if t.dtype != dtype:
        raise MoaError(MOA_ERR_INVALID_ARG, f"{name}: expected dtype {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise MoaError(MOA_ERR_INVALID_ARG, f"{name}: must be contiguous")
    if t.device.type != "cuda":
        raise MoaError(MOA_ERR_INVALID_ARG, f"{name}: must be a GPU tensor")


def moa_prefill(plan: Plan, q, k, v, o=None, stream=None):
    """o[b,i,h,:] = MoA attention of q over k, v ([B, n, H, D] layouts)."""
    import torch
    bsz, n = int(q.shape[0]), int(q.shape[1])
    dt = plan.torch_dtype
    _need(q, (bsz, n, plan.num_q_heads, plan.head_dim), dt, "q")
    _need(k, (bsz, n, plan.num_kv_heads, plan.head_dim), dt, "k")
    _need(v, (bsz, n, plan.num_kv_heads, plan.head_dim), dt, "v")
    if o is None:
        o = torch.empty_like(q)
    _need(o, q.shape, dt, "o")
    with torch.cuda.device(_one_device(q=q, k=k, v=v, o=o)):
        _check(load_library().moa_prefill(plan.handle, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                          o.data_ptr(), bsz, n, _stream(q, stream)))
    return o


def new_cache(plan: Plan, batch: int, device="cuda"):
    """Empty (k_cache, v_cache, pos_cache) for `batch` sequences (pos = -1)."""
    import torch
    shape = (batch, plan.cache_rows, plan.head_dim)
    kc = torch.zeros(shape, dtype=plan.torch_dtype, device=device)
    vc = torch.zeros(shape, dtype=plan.torch_dtype, device=device)
    pos = torch.full((batch, plan.cache_rows), -1, dtype=torch.int32, device=device)
    return kc, vc, pos


def moa_kv_append(plan: Plan, k_cache, v_cache, pos_cache, k_new, v_new, start_pos: int,
                  stream=None) -> None:
    """Appends positions start_pos .. start_pos + n_new - 1 (k_new: [B, n_new, H_kv, D])."""
    import torch
    bsz, n_new = int(k_new.shape[0]), int(k_new.shape[1])
    dt = plan.torch_dtype
    _need(k_new, (bsz, n_new, plan.num_kv_heads, plan.head_dim), dt, "k_new")
    _need(v_new, (bsz, n_new, plan.num_kv_heads, plan.head_dim), dt, "v_new")
    _need(k_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "k_cache")
    _need(v_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "v_cache")
    _need(pos_cache, (bsz, plan.cache_rows), torch.int32, "pos_cache")
    with torch.cuda.device(_one_device(k_cache=k_cache, v_cache=v_cache, pos_cache=pos_cache, k_new=k_new, v_new=v_new)):
        _check(load_library().moa_kv_append(plan.handle, k_cache.data_ptr(), v_cache.data_ptr(),
                                            pos_cache.data_ptr(), k_new.data_ptr(), v_new.data_ptr(),
                                            bsz, int(start_pos), n_new, _stream(k_new, stream)))


def moa_decode_workspace_bytes(plan: Plan, batch: int) -> int:
    return int(load_library().moa_decode_workspace_bytes(plan.handle, int(batch)))


def new_workspace(plan: Plan, batch: int, device="cuda"):
    """Decode workspace of the required size (contents need no initialisation)."""
    import torch
    nbytes = max(256, moa_decode_workspace_bytes(plan, batch))
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def moa_decode(plan: Plan, q, k_cache, v_cache, pos: int, workspace, o=None, stream=None):
    """Decode output for the token at `pos` (q, o: [B, H_q, D])."""
    import torch
    bsz = int(q.shape[0])
    dt = plan.torch_dtype
    _need(q, (bsz, plan.num_q_heads, plan.head_dim), dt, "q")
    _need(k_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "k_cache")
    _need(v_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "v_cache")
    if o is None:
        o = torch.empty_like(q)
    _need(o, q.shape, dt, "o")
    if workspace.device.type != "cuda" or not workspace.is_contiguous():
        raise MoaError(MOA_ERR_WORKSPACE, "workspace must be a contiguous GPU tensor")
    nbytes = workspace.numel() * workspace.element_size()
    with torch.cuda.device(_one_device(q=q, k_cache=k_cache, v_cache=v_cache, o=o, workspace=workspace)):
        _check(load_library().moa_decode(plan.handle, q.data_ptr(), k_cache.data_ptr(),
                                         v_cache.data_ptr(), o.data_ptr(), bsz, int(pos),
                                         workspace.data_ptr(), nbytes, _stream(q, stream)))
    return o


MOA_DECODE_SCRATCH_BYTES = 64 << 20


def moa_decode_noalloc(plan: Plan, q, k_cache, v_cache, pos: int, o, stream=None):
    """moa_decode without a caller workspace: the library keeps the split-K
    partials in its own fixed per-GPU array (MOA_DECODE_SCRATCH_BYTES), so the
    call allocates nothing; o must be given (q, o: [B, H_q, D]).  Calls that
    overlap in time on one GPU share that array and race."""
    bsz = int(q.shape[0])
    dt = plan.torch_dtype
    _need(q, (bsz, plan.num_q_heads, plan.head_dim), dt, "q")
    _need(k_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "k_cache")
    _need(v_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "v_cache")
    _need(o, q.shape, dt, "o")
    import torch
    with torch.cuda.device(_one_device(q=q, k_cache=k_cache, v_cache=v_cache, o=o)):
        _check(load_library().moa_decode_noalloc(plan.handle, q.data_ptr(), k_cache.data_ptr(),
                                                 v_cache.data_ptr(), o.data_ptr(), bsz, int(pos),
                                                 _stream(q, stream)))
    return o


def _positions(positions, bsz):
    import torch
    if positions.dtype != torch.int32 or tuple(positions.shape) != (bsz,) or positions.device.type != "cuda":
        raise MoaError(MOA_ERR_INVALID_ARG, f"positions: expected a GPU int32 tensor of shape ({bsz},)")
    if not positions.is_contiguous():
        raise MoaError(MOA_ERR_INVALID_ARG, "positions: must be contiguous")


def moa_kv_append_ragged(plan: Plan, k_cache, v_cache, pos_cache, k_new, v_new, positions,
                         stream=None) -> None:
    """One token per sequence at its own position (k_new: [B, 1, H_kv, D]; positions: int32[B])."""
    import torch
    bsz = int(k_new.shape[0])
    dt = plan.torch_dtype
    _need(k_new, (bsz, 1, plan.num_kv_heads, plan.head_dim), dt, "k_new")
    _need(v_new, (bsz, 1, plan.num_kv_heads, plan.head_dim), dt, "v_new")
    _need(k_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "k_cache")
    _need(v_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "v_cache")
    _need(pos_cache, (bsz, plan.cache_rows), torch.int32, "pos_cache")
    _positions(positions, bsz)
    with torch.cuda.device(_one_device(k_cache=k_cache, v_cache=v_cache, pos_cache=pos_cache, k_new=k_new, v_new=v_new, positions=positions)):
        _check(load_library().moa_kv_append_ragged(plan.handle, k_cache.data_ptr(), v_cache.data_ptr(),
                                                   pos_cache.data_ptr(), k_new.data_ptr(), v_new.data_ptr(),
                                                   positions.data_ptr(), bsz, _stream(k_new, stream)))


def moa_decode_ragged(plan: Plan, q, k_cache, v_cache, positions, workspace, o=None, stream=None):
    """Decode with sequence b at position positions[b] (q, o: [B, H_q, D])."""
    import torch
    bsz = int(q.shape[0])
    dt = plan.torch_dtype
    _need(q, (bsz, plan.num_q_heads, plan.head_dim), dt, "q")
    _need(k_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "k_cache")
    _need(v_cache, (bsz, plan.cache_rows, plan.head_dim), dt, "v_cache")
    _positions(positions, bsz)
    if o is None:
        o = torch.empty_like(q)
    _need(o, q.shape, dt, "o")
    if workspace.device.type != "cuda" or not workspace.is_contiguous():
        raise MoaError(MOA_ERR_WORKSPACE, "workspace must be a contiguous GPU tensor")
    nbytes = workspace.numel() * workspace.element_size()
    with torch.cuda.device(_one_device(q=q, k_cache=k_cache, v_cache=v_cache, o=o, positions=positions, workspace=workspace)):
        _check(load_library().moa_decode_ragged(plan.handle, q.data_ptr(), k_cache.data_ptr(),
                                                v_cache.data_ptr(), o.data_ptr(), positions.data_ptr(), bsz,
                                                workspace.data_ptr(), nbytes, _stream(q, stream)))
    return o


def moa_influence(q, k, v, dout, ebar=None, softmax_scale: float = 0.0, stream=None):
    """Block-averaged attention influence [H_q, nb, nb] (fp32) of dense causal
    attention over a batch of calibration items (paper Sec. 3.3, Eq. 3).

    q, dout: [B, n, H_q, D] bf16; k, v: [B, n, H_kv, D] bf16 (GPU, contiguous)."""
    import torch
    bsz, n, hq, d = (int(x) for x in q.shape)
    hkv = int(k.shape[2])
    for t, name, shape in ((q, "q", (bsz, n, hq, d)), (k, "k", (bsz, n, hkv, d)), (v, "v", (bsz, n, hkv, d)),
                           (dout, "dout", (bsz, n, hq, d))):
        _need(t, shape, torch.bfloat16, name)
    nb = -(-n // 64)
    if ebar is None:
        ebar = torch.empty((hq, nb, nb), dtype=torch.float32, device=q.device)
    _need(ebar, (hq, nb, nb), torch.float32, "ebar")
    desc = moa_desc_t(hq, hkv, d, 0, n, MOA_BF16, float(softmax_scale), 0, 0)
    with torch.cuda.device(_one_device(q=q, k=k, v=v, dout=dout, ebar=ebar)):
        _check(load_library().moa_influence(ctypes.byref(desc), q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                            dout.data_ptr(), ebar.data_ptr(), bsz, n, _stream(q, stream)))
    return ebar


def moa_rule_loss(ebar, n: int, num_sink: int, alpha, beta, flags: int = 0, stream=None):
    """(dl [H, R] fp64, density [R] fp64) on the GPU: the loss of every candidate
    rule for every head at length n (paper Sec. 3.3, Eq. 4) from the
    block-averaged influence ebar [H, nb, nb] (fp32, GPU)."""
    import torch
    h = int(ebar.shape[0])
    nb = -(-int(n) // 64)
    _need(ebar, (h, nb, nb), torch.float32, "ebar")
    a = np.ascontiguousarray(alpha, dtype=np.float64)
    b = np.ascontiguousarray(beta, dtype=np.float64)
    if a.shape != b.shape or a.ndim != 1:
        raise MoaError(MOA_ERR_INVALID_ARG, "alpha and beta must be 1-D arrays of the same length")
    r = int(a.shape[0])
    dl = torch.empty((h, r), dtype=torch.float64, device=ebar.device)
    dens = torch.empty((r,), dtype=torch.float64, device=ebar.device)
    with torch.cuda.device(_one_device(ebar=ebar, dl=dl, density=dens)):
        _check(load_library().moa_rule_loss(ebar.data_ptr(), h, int(n), int(num_sink), int(flags),
                                            a.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                            b.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), r,
                                            dl.data_ptr(), dens.data_ptr(), _stream(ebar, stream)))
    return dl, dens

