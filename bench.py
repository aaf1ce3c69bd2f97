#!/usr/bin/env python3
"""Benchmark of the MoA hot path on one MI355X.

One step = one pass of the whole path over one batch of the Vicuna-7B-shaped
layer (32 MHA heads, head_dim 128, bf16, batch 32, context N = 8192, per-head
elastic windows with mean N/2, 64 sinks):

    moa_plan (host) -> moa_prefill (B x N tokens) -> moa_kv_append (bulk fill)
    -> 256 x [moa_kv_append (one token) -> moa_decode]

`value` = decoded tokens / wall time of the whole step (prefill included).
The JSON line also carries the decode-only rate, the prefill rate, and the
roofline of the dominant kernel (decode, HBM-bound) and of prefill (MFMA).
All inputs are synthetic (seeded N(0,1)) and resident in HBM before timing.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, TFLOP/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class TimingEvents:
    """Pairs of HIP events that only time launches on a stream.

    They are created with hipEventDisableSystemFence.  A default HIP event
    performs a system-scope release when it is recorded (an L2 write-back and
    invalidation); between the decode loop's kernels each such record left
    about 5 us of idle GPU time, which is measurement cost and not work.
    Elapsed times are read only after a full device synchronisation, so the
    missing fence never matters to the reading.  The events come from the HIP
    runtime torch has loaded, so they live on torch's streams."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, pairs: int):
        import ctypes

        self._c = ctypes
        self._hip = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD | os.RTLD_LAZY)
        self._hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self._hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = []
        for _ in range(pairs):
            pair = (ctypes.c_void_p(), ctypes.c_void_p())
            for e in pair:
                self._check(self._hip.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE),
                            "hipEventCreateWithFlags")
            self.ev.append(pair)

    @staticmethod
    def _check(rc: int, what: str) -> None:
        if rc != 0:
            raise RuntimeError(f"{what} failed with HIP error {rc}")

    def record(self, i: int, end: int, stream) -> None:
        """Records the start (end=0) or end (end=1) event of pair i on a torch stream."""
        self._check(self._hip.hipEventRecord(self.ev[i][end], self._c.c_void_p(stream.cuda_stream)),
                    "hipEventRecord")

    def ms(self, i: int) -> float:
        """Milliseconds between pair i's events (call after torch.cuda.synchronize())."""
        out = self._c.c_float()
        self._check(self._hip.hipEventElapsedTime(self._c.byref(out), self.ev[i][0], self.ev[i][1]),
                    "hipEventElapsedTime")
        return float(out.value)

    def close(self) -> None:
        for pair in self.ev:
            for e in pair:
                self._hip.hipEventDestroy(e)
        self.ev = []


ROOT = os.path.dirname(os.path.abspath(__file__))


def measured_traffic(profile: str):
    """HBM bytes per launch recorded in profiles/<profile> by rocprofv3
    FETCH_SIZE / WRITE_SIZE passes (scaled by the copy-kernel calibration), or
    None when the kernel sources changed since the counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", profile)
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        key, sep, val = line.partition(":")
        if sep and key.strip() in ("traffic_bytes_per_launch", "source_files", "source_sha256"):
            fields[key.strip()] = val.strip()
    if len(fields) != 3:
        return None
    h = hashlib.sha256()
    for f in fields["source_files"].split():
        src = os.path.join(ROOT, "paper_2406_14909_amd", "csrc", f)
        if not os.path.exists(src):
            return None
        h.update(open(src, "rb").read())
    if h.hexdigest() != fields["source_sha256"]:
        return None
    return int(float(fields["traffic_bytes_per_launch"]))


def executed_wave_tiles(n: int, w: int, s: int, block: int = 0) -> int:
    """(32-row wave, 64-key tile) products the prefill kernel runs for one
    query head.  Each 128-row work-group visits the sink tiles [0, ta) and
    the band tiles [tb, tl] of its rows; each of its 32-row waves multiplies
    a visited tile when the tile holds a visible pair of one of its rows
    (the masked entries inside such a tile are computed too).  With block
    (64) the band counts whole 64-token blocks, ceil(w / 64) of them."""
    sh, W = (6, -(-w // 64)) if block else (0, w)

    def band_start(i):
        return ((i >> sh) - W + 1) << sh

    def inter(lo1, hi1, lo2, hi2):          # |[lo1, hi1) & [lo2, hi2)|
        return np.maximum(0, np.minimum(hi1, hi2) - np.maximum(lo1, lo2))

    r0 = np.arange(0, n, 32, dtype=np.int64)          # each wave's first row
    r1 = np.minimum(n, r0 + 32)
    i0 = (r0 // 128) * 128                            # its work-group's rows
    i1 = np.minimum(n, i0 + 128)
    ta = (np.minimum(s, i1) + 63) // 64
    tl = (i1 - 1) // 64
    tb = np.maximum(ta, np.maximum(0, band_start(i0)) // 64)
    tmax = (r1 - 1) // 64                             # causal: tile starts at or before the last row
    t_sink = (s + 63) // 64                           # tiles starting below s
    t_band = band_start(r0) // 64                     # tiles reaching the first row's band
    far = np.int64(1) << 40
    total = 0
    for lo, hi in ((np.zeros_like(ta), ta), (tb, tl + 1)):
        hi = np.minimum(hi, tmax + 1)
        total += int((inter(lo, hi, 0, t_sink) + inter(lo, hi, t_band, far)
                      - inter(np.maximum(lo, t_band), hi, 0, t_sink)).sum())
    return total


def visible_pairs(n: int, w: int, s: int, block: int = 0) -> int:
    """sum_{i<n} |{j <= i : j < s or j in the band of i}| (closed form).

    Token band: i - j < w.  Block band (block > 0): the band of row i starts
    at bs = max(0, (i // block - ceil(w / block) + 1) * block), so row i sees
    (i + 1 - bs) band keys plus min(s, bs) sinks before the band; bs is
    constant over a block of rows."""
    if block:
        nb = -(-w // block)
        total = 0
        for first in range(0, n, block):
            last = min(n, first + block)                 # rows [first, last)
            bs = max(0, (first // block - nb + 1) * block)
            total += (last * (last + 1) - first * (first + 1)) // 2 - (last - first) * bs
            total += (last - first) * min(s, bs)
        return total
    total = 0
    # rows i < w: all i+1 keys visible
    a = min(n, w)
    total += a * (a + 1) // 2
    if n > w:
        rows = n - w
        total += rows * w
        # sinks outside the band: for row i >= w, keys j < min(s, i - w + 1)
        # sum_{i=w}^{n-1} min(s, i - w + 1) = sum_{r=1}^{rows} min(s, r)
        m = min(s, rows)
        total += m * (m + 1) // 2 + (rows - m) * s
    return total


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--decode-steps", type=int, default=None)
    ap.add_argument("--workload", default="vicuna7b-decode-b32-ctx8192")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layers", type=int, default=1,
                    help="independent cache sets decoded in rotation (keeps small caches out of the "
                         "256 MB last-level cache between steps); each set has its own timeline")
    ap.add_argument("--block-band", action="store_true",
                    help="prefill band in 64-token blocks (the paper's kernel setting)")
    ap.add_argument("--span-includes-sinks", action="store_true",
                    help="the elastic rule gives the whole span, sinks included")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds per oracle leg")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-configuration prefill / decode measurements of the other workloads")
    ap.add_argument("--configs-reps", type=int, default=32,
                    help="timed decode calls per configuration (prefill: a quarter of it, at least 5)")
    ap.add_argument("--profile-kernel", choices=["decode", "prefill", "append", "copy"], default=None,
                    help="launch only this kernel --reps times on the bench workload (hardware-counter runs)")
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--influence", action="store_true",
                    help="time the attention-influence profile (moa_influence) on the workload's layer shape")
    ap.add_argument("--influence-n", type=int, default=8192, help="profiled length for --influence")
    ap.add_argument("--influence-items", type=int, default=4, help="calibration items for --influence")
    ap.add_argument("--rule-loss", action="store_true",
                    help="time the rule-loss table (moa_rule_loss): 54 rules x 1024 heads at --influence-n")
    ap.add_argument("--power", choices=["prefill", "decode", "influence", "mfma"], default=None,
                    help="run one kernel of the workload (or the MFMA-only calibration loop) for --power-seconds "
                         "while sampling the board's socket power and shader clock with amd-smi")
    ap.add_argument("--power-seconds", type=float, default=12.0)
    ap.add_argument("--peaks", action="store_true",
                    help="measure practical ceilings: hipBLASLt bf16 GEMM TFLOP/s and streaming-read GB/s")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the MoA path is built and measured on a single "
              "MI355X (run with --gpus 1).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    if args.peaks:
        print(json.dumps(measure_peaks()), flush=True)
        return 0
    if args.power:
        print(json.dumps(measure_power(args)), flush=True)
        return 0
    if args.influence:
        print(json.dumps(measure_influence(args)), flush=True)
        return 0
    if args.rule_loss:
        print(json.dumps(measure_rule_loss(args)), flush=True)
        return 0

    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import workloads
    from paper_2406_14909_amd import moa as M

    wl = workloads.workload(args.workload)
    B, Hq, Hkv, D, s, N = wl.decode_batch, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.num_sink, wl.n
    steps_dec = args.decode_steps if args.decode_steps is not None else wl.decode_steps
    dtype = wl.torch_dtype()
    esz = 2 if wl.dtype == "bf16" else 4
    dev = "cuda"
    torch.cuda.init()
    log(f"[bench] workload {wl.name}: B={B} Hq={Hq} Hkv={Hkv} D={D} s={s} N={N} decode_steps={steps_dec}")

    # ---- inputs resident in HBM -------------------------------------------
    q_pre = workloads.randn((B, N, Hq, D), wl.seed * 10 + 1, dtype, dev)
    k_pre = workloads.randn((B, N, Hkv, D), wl.seed * 10 + 2, dtype, dev)
    v_pre = workloads.randn((B, N, Hkv, D), wl.seed * 10 + 3, dtype, dev)
    q_dec = workloads.randn((steps_dec, B, Hq, D), wl.seed * 10 + 4, dtype, dev)
    k_dec = workloads.randn((steps_dec, B, 1, Hkv, D), wl.seed * 10 + 5, dtype, dev)
    v_dec = workloads.randn((steps_dec, B, 1, Hkv, D), wl.seed * 10 + 6, dtype, dev)
    o_pre = torch.empty_like(q_pre)
    o_dec = torch.empty((B, Hq, D), dtype=dtype, device=dev)

    flags = (M.MOA_BLOCK_BAND if args.block_band else 0) | (M.MOA_SPAN_INCLUDES_SINKS if args.span_includes_sinks else 0)
    block = M.MOA_BAND_BLOCK if args.block_band else 0
    plan = M.moa_plan(Hq, Hkv, D, s, N, wl.dtype, wl.alpha, wl.beta, flags=flags)
    R = max(1, args.layers)
    sets = [M.new_cache(plan, B) for _ in range(R)]
    kc, vc, pos = sets[0]
    ws = M.new_workspace(plan, B)
    windows = [int(x) for x in plan.window]
    caps = [int(x) for x in plan.capacity]
    log(f"[bench] windows mean {np.mean(windows):.1f} (min {min(windows)}, max {max(windows)}); "
        f"cache {kc.numel() * esz * 2 / 1e9:.2f} GB")

    # ---- algorithmic work -------------------------------------------------
    group = Hq // Hkv
    prefill_flops = 4.0 * D * B * group * sum(visible_pairs(N, w, s, block) for w in windows)
    # matrix-core work the kernel runs, masked entries of edge tiles included
    prefill_exec_flops = 4.0 * D * B * group * 32 * 64 * sum(executed_wave_tiles(N, w, s, block) for w in windows)
    dec_bytes = []
    for i in range(steps_dec):
        t = N + i // R                                  # decode step i runs on cache set i % R
        fills = sum(min(t + 1, c) for c in caps)
        dec_bytes.append(B * fills * D * 2 * esz + 2 * B * Hq * D * esz)

    if args.profile_kernel:
        return profile_kernel(args, M, plan, q_pre, k_pre, v_pre, o_pre, q_dec, k_dec, v_dec, o_dec,
                              kc, vc, pos, ws, N, prefill_flops, dec_bytes[0])

    stream = torch.cuda.current_stream()
    # Events time an even sample of at most 16 decode calls per step: each
    # record between two kernels still leaves the GPU idle for about 4 us, so
    # bracketing all 256 calls would slow the step it measures.  The sample
    # takes the middle call of each stride, so it does not give the first
    # call after the bulk cache fill (slower by up to a quarter) 16 times its
    # share of the average.
    stride = max(1, steps_dec // 16)
    timed = list(range(stride // 2, steps_dec, stride))
    slot = {i: k + 1 for k, i in enumerate(timed)}     # event pair 0 is the prefill
    ev = TimingEvents(len(timed) + 1)

    def step(record: bool):
        p = M.moa_plan(Hq, Hkv, D, s, N, wl.dtype, wl.alpha, wl.beta, flags=flags)
        if record:
            ev.record(0, 0, stream)
        M.moa_prefill(p, q_pre, k_pre, v_pre, o_pre)
        if record:
            ev.record(0, 1, stream)
        for kc_r, vc_r, pos_r in sets:
            M.moa_kv_append(p, kc_r, vc_r, pos_r, k_pre, v_pre, 0)
        for i in range(steps_dec):
            t = N + i // R
            kc_r, vc_r, pos_r = sets[i % R]
            M.moa_kv_append(p, kc_r, vc_r, pos_r, k_dec[i], v_dec[i], t)
            if record and i in slot:
                ev.record(slot[i], 0, stream)
            M.moa_decode(p, q_dec[i], kc_r, vc_r, t, ws, o_dec)
            if record and i in slot:
                ev.record(slot[i], 1, stream)
        return p

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()

    prefill_ms, decode_ms, wall = [], [], []
    for _ in range(args.steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        step(True)
        torch.cuda.synchronize()
        wall.append(time.perf_counter() - t0)
        prefill_ms.append(ev.ms(0))
        decode_ms.append(sum(ev.ms(k) for k in range(1, len(timed) + 1)))
        log(f"[bench] step {len(wall)}: {wall[-1] * 1e3:.2f} ms (prefill {prefill_ms[-1]:.3f} ms, "
            f"{len(timed)} timed decode calls {decode_ms[-1]:.3f} ms)")
    ev.close()
    ms_per_step = 1e3 * float(np.mean(wall))
    pre_ms = float(np.mean(prefill_ms))
    dec_ms = float(np.mean(decode_ms))              # the timed calls of one step
    timed_bytes = float(sum(dec_bytes[i] for i in timed))
    tokens = B * steps_dec
    value = tokens / (ms_per_step / 1e3)
    dec_gbs = timed_bytes / (dec_ms / 1e3) / 1e9
    pre_tflops = prefill_flops / (pre_ms / 1e3) / 1e12
    dec_launch_us = 1e3 * dec_ms / len(timed)

    dname = "bf16" if wl.dtype == "bf16" else "float"
    dec_kernel = (f"decode_mma_kernel<{D},{group}>" if wl.dtype == "bf16" and group >= 2
                  else f"decode_valu_kernel<{dname},{D},{group}>")
    layers = (("vicuna7b", "Vicuna-7B-shaped attention layer"), ("llama3-8b", "Llama-3-8B-shaped attention layer"),
              ("llama3-70b", "Llama-3-70B-shaped attention layer"))
    layer = next((text for prefix, text in layers if wl.name.startswith(prefix)), "small attention layer")
    mean_frac = float(np.mean(windows)) / N
    result = {
        "metric": "decode tokens/s (whole step: plan + prefill + cache fill + decode loop)",
        "value": round(value, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": f"synthetic: q,k,v ~ N(0,1) seeded; per-KV-head elastic windows (mean {mean_frac:.2f} N)",
        "config": {
            "workload": wl.name,
            "layer": layer,
            "batch": B, "context": N, "decode_steps": steps_dec,
            "num_q_heads": Hq, "num_kv_heads": Hkv, "head_dim": D, "num_sink": s,
            "mean_window": float(np.mean(windows)),
            "density": float(np.mean([min(c, N) for c in caps])) / N,
            "parallelism": "single GPU",
            "cache_sets": R,
            "plan_flags": [name for name, on in (("block_band", args.block_band),
                                                  ("span_includes_sinks", args.span_includes_sinks)) if on],
        },
        "decode_only_tokens_per_s": round(B / (dec_launch_us / 1e6), 2),
        "decode_kernel_avg_us": round(dec_launch_us, 3),
        "decode_calls_timed_per_step": len(timed),
        "decode_hbm_gbs": round(dec_gbs, 1),
        "prefill_ms": round(pre_ms, 4),
        "prefill_inband_tflops": round(pre_tflops, 2),
        "prefill_tile_efficiency": round(prefill_flops / prefill_exec_flops, 4),
        "prefill_executed_tflops": round(prefill_exec_flops / (pre_ms / 1e3) / 1e12, 2),
        "roofline": {
            "kernel": f"moa_decode ({dec_kernel} + decode_combine_kernel), per call",
            "bound": "hbm",
            "achieved": round(dec_gbs, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(f"hbm_traffic__decode_kernel__{wl.name}.md"),
            "traffic_kernel": f"{dec_kernel} (bytes per launch)",
            "bytes_per_launch": round(timed_bytes / len(timed)),
        },
        "roofline_prefill": {
            "kernel": "prefill_kernel<bf16,128>, per call",
            "bound": "mfma",
            "achieved": round(pre_tflops, 2),
            "peak": BF16_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(pre_tflops / BF16_MFMA_PEAK_TFLOPS, 4),
            "traffic": measured_traffic(f"hbm_traffic__prefill_kernel__{wl.name}.md"),
            "flops_per_launch": prefill_flops,
        },
    }

    if not args.no_configs:
        result["configs"] = measure_configs(M, workloads, args.configs_reps)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, plan, block, q_pre, k_pre, v_pre, q_dec, k_dec, v_dec,
                                              steps_dec, args.cpu_budget)
    print(json.dumps(result), flush=True)
    return 0


class CallTimer:
    """Times individual launches on torch's current stream with fence-free
    event pairs; median milliseconds per call."""

    def __init__(self, calls: int):
        import torch

        self.stream = torch.cuda.current_stream()
        self.ev = TimingEvents(calls)
        self.n = 0

    def __call__(self, fn):
        i = self.n
        self.ev.record(i, 0, self.stream)
        fn()
        self.ev.record(i, 1, self.stream)
        self.n += 1

    def median_ms(self) -> float:
        import torch

        torch.cuda.synchronize()
        ms = sorted(self.ev.ms(i) for i in range(self.n))
        self.ev.close()
        return float(ms[len(ms) // 2])


def measure_configs(M, workloads, reps: int):
    """Prefill and decode of the other workload shapes, each in the launch
    configuration the paper's efficiency setup describes (one layer; decode
    after a full-context prefill, appending one token per step).

    prefill: moa_prefill of the workload's prefill batch at N tokens, median
      of max(5, reps // 4) calls after 3 warm-ups; in-band TFLOP/s = 4 * D *
      visible pairs / time (masked entries of executed tiles not counted).
    decode: moa_decode at the workload's decode batch over 4 independent
      cache sets decoded in rotation (each call reads data the 256 MB
      last-level cache does not hold: the sets are 0.27-0.54 GB each), one
      append per call, positions advancing; median of `reps` calls after 8
      warm-ups; GB/s = filled-slot K/V bytes + q + o per call / time."""
    import torch

    out = {}
    for name, do_prefill, do_decode in (("vicuna7b-prefill-n4096", True, False),
                                        ("llama3-8b-gqa-n16384", True, True),
                                        ("llama3-70b-gqa-n32768", True, True)):
        wl = workloads.workload(name)
        N, Hq, Hkv, D, s = wl.n, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.num_sink
        esz = 2
        group = Hq // Hkv
        plan = M.moa_plan(Hq, Hkv, D, s, N, wl.dtype, wl.alpha, wl.beta)
        windows = [int(x) for x in plan.window]
        caps = [int(x) for x in plan.capacity]
        entry = {"num_q_heads": Hq, "num_kv_heads": Hkv, "head_dim": D, "num_sink": s, "context": N,
                 "mean_window": float(np.mean(windows)), "density": float(np.mean([min(c, N) for c in caps])) / N}
        log(f"[bench] config {name}")
        if do_prefill:
            B = wl.prefill_batch
            q = workloads.randn((B, N, Hq, D), wl.seed * 10 + 7, torch.bfloat16, "cuda")
            k = workloads.randn((B, N, Hkv, D), wl.seed * 10 + 8, torch.bfloat16, "cuda")
            v = workloads.randn((B, N, Hkv, D), wl.seed * 10 + 9, torch.bfloat16, "cuda")
            o = torch.empty_like(q)
            for _ in range(3):
                M.moa_prefill(plan, q, k, v, o)
            n_calls = max(5, reps // 4)
            timer = CallTimer(n_calls)
            for _ in range(n_calls):
                timer(lambda: M.moa_prefill(plan, q, k, v, o))
            ms = timer.median_ms()
            flops = 4.0 * D * B * group * sum(visible_pairs(N, w, s) for w in windows)
            tf = flops / (ms / 1e3) / 1e12
            entry["prefill"] = {"batch": B, "ms": round(ms, 4), "inband_tflops": round(tf, 2),
                                "peak": BF16_MFMA_PEAK_TFLOPS, "frac": round(tf / BF16_MFMA_PEAK_TFLOPS, 4),
                                "flops_per_launch": flops, "kernel": f"prefill_kernel<bf16,{D}>",
                                "calls_timed": n_calls}
            del q, k, v, o
        if do_decode:
            B, sets_n = wl.decode_batch, 4
            k = workloads.randn((B, N, Hkv, D), wl.seed * 10 + 5, torch.bfloat16, "cuda")
            v = workloads.randn((B, N, Hkv, D), wl.seed * 10 + 6, torch.bfloat16, "cuda")
            total_calls = 8 + reps
            steps = -(-total_calls // sets_n)
            kn = workloads.randn((steps, B, 1, Hkv, D), wl.seed * 10 + 10, torch.bfloat16, "cuda")
            vn = workloads.randn((steps, B, 1, Hkv, D), wl.seed * 10 + 11, torch.bfloat16, "cuda")
            qn = workloads.randn((sets_n, B, Hq, D), wl.seed * 10 + 12, torch.bfloat16, "cuda")
            sets = [M.new_cache(plan, B) for _ in range(sets_n)]
            for c in sets:
                M.moa_kv_append(plan, *c, k, v, 0)
            del k, v
            ws = M.new_workspace(plan, B)
            o = torch.empty((B, Hq, D), dtype=torch.bfloat16, device="cuda")
            timer = CallTimer(reps)
            nbytes = []
            for i in range(total_calls):
                r, t = i % sets_n, N + i // sets_n
                M.moa_kv_append(plan, *sets[r], kn[i // sets_n], vn[i // sets_n], t)
                call = (lambda r=r, t=t: M.moa_decode(plan, qn[r], sets[r][0], sets[r][1], t, ws, o))
                if i < 8:
                    call()
                else:
                    timer(call)
                    nbytes.append(B * sum(min(t + 1, c) for c in caps) * D * 2 * esz + 2 * B * Hq * D * esz)
            ms = timer.median_ms()
            gbs = float(np.mean(nbytes)) / (ms / 1e3) / 1e9
            kern = f"decode_mma_kernel<{D},{group}>" if group >= 2 else f"decode_valu_kernel<bf16,{D},1>"
            entry["decode"] = {"batch": B, "us_per_call": round(ms * 1e3, 2), "hbm_gbs": round(gbs, 1),
                               "peak": HBM_PEAK_GBS, "frac": round(gbs / HBM_PEAK_GBS, 4),
                               "tokens_per_s": round(B / (ms / 1e3), 1),
                               "bytes_per_call": round(float(np.mean(nbytes))), "cache_sets": sets_n,
                               "traffic": measured_traffic(f"hbm_traffic__decode_kernel__{name}.md"),
                               "kernel": f"moa_decode ({kern} + decode_combine_kernel)", "calls_timed": reps}
            del sets, kn, vn, qn, ws, o
        torch.cuda.empty_cache()
        out[name] = entry
    return out


def sample_power(stop, out, delay=4.0, period=0.5):
    """Appends (socket W, mean shader MHz, min, max) from `amd-smi metric` every
    `period` seconds, after `delay` seconds of warm-up, until stop is set."""
    import subprocess

    if stop.wait(delay):
        return
    while not stop.is_set():
        try:
            r = subprocess.run(["amd-smi", "metric", "--power", "--clock", "--json"], capture_output=True,
                               text=True, timeout=10)
            for g in json.loads(r.stdout).get("gpu_data", [])[:1]:
                clks = [v["clk"]["value"] for k, v in g["clock"].items() if k.startswith("gfx_")]
                out.append((float(g["power"]["socket_power"]["value"]), sum(clks) / len(clks), min(clks), max(clks)))
        except Exception as e:                                    # no amd-smi, or a format it does not know
            log(f"[bench] power sample failed: {e}")
            return
        stop.wait(period)


def measure_power(args):
    """Board power and shader clock while one kernel runs back to back.

    The hot path is bound by the board's power limit when the matrix cores
    and vector ALUs work together: the clock then drops below what a pure
    matrix-core load keeps.  prefill / decode: the workload's moa_prefill /
    moa_decode (one cache set) repeated for --power-seconds; mfma: the
    MFMA-only calibration loop held for the same time.  Rate: in-band
    TFLOP/s, HBM GB/s or the loop's TFLOP/s; energy per unit = power / rate."""
    import threading

    import torch

    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    samples, stop = [], threading.Event()
    sampler = threading.Thread(target=sample_power, args=(stop, samples), daemon=True)
    res = {"kernel": args.power, "workload": args.workload}
    if args.power == "mfma":
        import subprocess

        probe = os.path.join(ROOT, "paper_2406_14909_amd", "_build", "mfma_loop")
        sampler.start()
        out = subprocess.run([probe, str(args.power_seconds)], capture_output=True, text=True, timeout=300).stdout
        stop.set()
        rate = float([l.split()[1] for l in out.splitlines() if l.startswith("hold ")][0])
        res.update({"rate": rate, "unit": "TFLOP/s"})
    else:
        import workloads
        from paper_2406_14909_amd import moa as M

        wl = workloads.workload(args.workload)
        B, N = wl.decode_batch, wl.n
        plan = M.moa_plan(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.num_sink, N, wl.dtype, wl.alpha, wl.beta)
        dt = wl.torch_dtype()
        if args.power == "influence":
            n, items = args.influence_n, args.influence_items
            q = workloads.randn((items, n, wl.num_q_heads, wl.head_dim), 11, torch.bfloat16, "cuda")
            k = workloads.randn((items, n, wl.num_kv_heads, wl.head_dim), 12, torch.bfloat16, "cuda")
            v = workloads.randn((items, n, wl.num_kv_heads, wl.head_dim), 13, torch.bfloat16, "cuda")
            do = workloads.randn((items, n, wl.num_q_heads, wl.head_dim), 14, torch.bfloat16, "cuda")
            ebar = M.moa_influence(q, k, v, do)
            call = lambda: M.moa_influence(q, k, v, do, ebar)
            work = 8.0 * wl.head_dim * (n * (n + 1) // 2) * wl.num_q_heads * items / 1e12
            unit = "TFLOP/s"
        elif args.power == "prefill":
            q = workloads.randn((B, N, wl.num_q_heads, wl.head_dim), 1, dt, "cuda")
            k = workloads.randn((B, N, wl.num_kv_heads, wl.head_dim), 2, dt, "cuda")
            v = workloads.randn((B, N, wl.num_kv_heads, wl.head_dim), 3, dt, "cuda")
            o = torch.empty_like(q)
            call = lambda: M.moa_prefill(plan, q, k, v, o)
            group = wl.num_q_heads // wl.num_kv_heads
            work = 4.0 * wl.head_dim * B * group * sum(visible_pairs(N, int(w), wl.num_sink) for w in plan.window) / 1e12
            unit = "TFLOP/s"
        else:
            k = workloads.randn((B, N + 1, wl.num_kv_heads, wl.head_dim), 5, dt, "cuda")
            v = workloads.randn((B, N + 1, wl.num_kv_heads, wl.head_dim), 6, dt, "cuda")
            q = workloads.randn((B, wl.num_q_heads, wl.head_dim), 7, dt, "cuda")
            kc, vc, pos = M.new_cache(plan, B)
            M.moa_kv_append(plan, kc, vc, pos, k, v, 0)
            del k, v
            ws = M.new_workspace(plan, B)
            o = torch.empty_like(q)
            call = lambda: M.moa_decode(plan, q, kc, vc, N, ws, o)
            esz = 2 if wl.dtype == "bf16" else 4
            work = B * sum(min(N + 1, int(c)) for c in plan.capacity) * wl.head_dim * 2 * esz / 1e9
            unit = "GB/s"
        call()
        torch.cuda.synchronize()
        sampler.start()
        t0, calls = time.perf_counter(), 0
        while time.perf_counter() - t0 < args.power_seconds:
            for _ in range(10):
                call()
            torch.cuda.synchronize()
            calls += 10
        elapsed = time.perf_counter() - t0
        stop.set()
        res.update({"rate": round(work * calls / elapsed, 1), "unit": unit, "calls": calls})
    sampler.join(timeout=15)
    if samples:
        pw = sum(s[0] for s in samples) / len(samples)
        res.update({"socket_power_w": round(pw, 1), "shader_clock_mhz": round(sum(s[1] for s in samples) / len(samples)),
                    "shader_clock_min_mhz": min(s[2] for s in samples), "shader_clock_max_mhz": max(s[3] for s in samples),
                    "samples": len(samples),
                    "energy_per_unit": round(pw / res["rate"], 4),
                    "energy_unit": "pJ/FLOP" if res["unit"] == "TFLOP/s" else "J/GB"})
    return res


def measure_influence(args):
    """Times moa_influence (dense causal attention of the workload's layer shape,
    bf16) over a batch of calibration items, after at least 3 untimed calls
    (the first calls run before the clocks have settled).  Algorithmic work:
    two passes of two products (Q K^T and dO V^T), 8 * head_dim flops per
    causal (query, key) pair per item and query head."""
    import torch

    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import workloads
    from paper_2406_14909_amd import moa as M

    wl = workloads.workload(args.workload)
    n, items, hq, hkv, d = args.influence_n, args.influence_items, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    q = workloads.randn((items, n, hq, d), 11, torch.bfloat16, "cuda")
    k = workloads.randn((items, n, hkv, d), 12, torch.bfloat16, "cuda")
    v = workloads.randn((items, n, hkv, d), 13, torch.bfloat16, "cuda")
    do = workloads.randn((items, n, hq, d), 14, torch.bfloat16, "cuda")
    ebar = M.moa_influence(q, k, v, do)
    for _ in range(max(3, args.warmup)):
        M.moa_influence(q, k, v, do, ebar)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        M.moa_influence(q, k, v, do, ebar)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    flops = 8.0 * d * (n * (n + 1) // 2) * hq * items
    return {
        "metric": "attention-influence profile throughput", "unit": "TFLOP/s",
        "value": round(flops / (ms / 1e3) / 1e12, 2), "ms_per_call": round(ms, 3),
        "config": {"workload": wl.name, "n": n, "items": items, "num_q_heads": hq, "num_kv_heads": hkv,
                   "head_dim": d},
        "roofline": {"kernel": f"influence_kernel<{d}>", "bound": "mfma",
                     "achieved": round(flops / (ms / 1e3) / 1e12, 2), "peak": BF16_MFMA_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(flops / (ms / 1e3) / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
                     "flops_per_launch": flops},
    }


def measure_rule_loss(args):
    """Times moa_rule_loss for a 32-layer x 32-head model (1024 profiles) at the
    profiled length, over the paper's 54-rule grid (block band, span includes
    sinks).  Algorithmic bytes: the causal half of the fp32 profile read once
    plus the fp64 table written."""
    import torch

    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    from paper_2406_14909_amd import moa as M
    from paper_2406_14909_amd import search

    heads, n = 1024, args.influence_n
    nb = -(-n // 64)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(21)
    ebar = torch.randn((heads, nb, nb), generator=gen, device="cuda").tril_()
    a, b = search.candidate_rules()
    flags = M.MOA_BLOCK_BAND | M.MOA_SPAN_INCLUDES_SINKS
    for _ in range(max(3, args.warmup)):
        M.moa_rule_loss(ebar, n, 64, a, b, flags)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        M.moa_rule_loss(ebar, n, 64, a, b, flags)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    nbytes = heads * (nb * (nb + 1) // 2) * 4 + heads * len(a) * 8
    return {
        "metric": "rule-loss table time", "unit": "ms", "value": round(ms, 4), "higher_is_better": False,
        "config": {"heads": heads, "n": n, "rules": len(a), "flags": "block_band|span_includes_sinks"},
        "roofline": {"kernel": "rule_loss_kernel", "bound": "hbm", "achieved": round(nbytes / (ms / 1e3) / 1e9, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                     "bytes_per_launch": nbytes},
    }


def measure_peaks():
    """Practical ceilings on this GPU, measured with library kernels.

    HBM read: the package's streaming-read calibration program (16-byte loads
    over 2 GiB, a sweep of grid sizes and loads in flight), best rate;
    MFMA: a 16384^3 bf16 GEMM (torch.matmul -> hipBLASLt), best of 5.
    HBM read: torch.sum over 8 GiB of bf16 (a streaming reduction), best of 5;
    HBM copy: a 4 GiB device-to-device copy (read + write), best of 5.
    """
    import torch

    def best_ms(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1))
        return best

    n = 16384
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    gemm_ms = best_ms(lambda: torch.matmul(a, b))
    del a, b
    big = torch.ones((8 << 30) // 2, device="cuda", dtype=torch.bfloat16)
    read_ms = best_ms(lambda: big.sum(dtype=torch.float32))
    del big
    src = torch.ones((4 << 30) // 2, device="cuda", dtype=torch.bfloat16)
    dst = torch.empty_like(src)
    copy_ms = best_ms(lambda: dst.copy_(src))
    def calibration(name):
        """Runs a calibration program of the package (built by build()); its "best" figure."""
        probe = os.path.join(ROOT, "paper_2406_14909_amd", "_build", name)
        if not os.path.exists(probe):
            return None
        import subprocess
        out = subprocess.run([probe], capture_output=True, text=True, timeout=120).stdout
        log(out.strip())
        best = [line.split()[1] for line in out.splitlines() if line.startswith("best ")]
        return float(best[0]) if best else None

    stream_best = calibration("stream_read")
    mfma_best = calibration("mfma_loop")
    return {
        "hip_stream_read_gbs": stream_best,
        "hip_mfma_loop_bf16_tflops": mfma_best,
        "gemm_bf16_16384_tflops": round(2.0 * n ** 3 / (gemm_ms / 1e3) / 1e12, 1),
        "stream_read_gbs": round((8 << 30) / (read_ms / 1e3) / 1e9, 1),
        "copy_read_plus_write_gbs": round(2 * (4 << 30) / (copy_ms / 1e3) / 1e9, 1),
    }


def profile_kernel(args, M, plan, q_pre, k_pre, v_pre, o_pre, q_dec, k_dec, v_dec, o_dec, kc, vc, pos,
                   ws, N, prefill_flops, dec_bytes):
    """Launches one kernel of the workload --reps times (for rocprofv3 --pmc runs).

    decode: moa_decode at position N over the caches filled from the prompt;
    prefill: moa_prefill of the prompt; append: one-token moa_kv_append;
    copy: a plain 1 GiB device copy (calibrates FETCH_SIZE / WRITE_SIZE).
    Prints one JSON line with the algorithmic work per launch.
    """
    import torch

    info = {"kernel": args.profile_kernel, "reps": args.reps}
    if args.profile_kernel in ("decode", "append"):
        M.moa_kv_append(plan, kc, vc, pos, k_pre, v_pre, 0)
        M.moa_kv_append(plan, kc, vc, pos, k_dec[0], v_dec[0], N)
    torch.cuda.synchronize()
    for _ in range(args.reps):
        if args.profile_kernel == "decode":
            M.moa_decode(plan, q_dec[0], kc, vc, N, ws, o_dec)
        elif args.profile_kernel == "prefill":
            M.moa_prefill(plan, q_pre, k_pre, v_pre, o_pre)
        elif args.profile_kernel == "append":
            M.moa_kv_append(plan, kc, vc, pos, k_dec[0], v_dec[0], N)
    if args.profile_kernel == "copy":
        nbytes = 1 << 30
        src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.reps):
            dst.copy_(src)
        info["bytes_read_per_launch"] = nbytes
        info["bytes_written_per_launch"] = nbytes
    elif args.profile_kernel == "decode":
        info["algorithmic_bytes_per_launch"] = dec_bytes
    elif args.profile_kernel == "prefill":
        info["algorithmic_flops_per_launch"] = prefill_flops
    torch.cuda.synchronize()
    print(json.dumps(info), flush=True)
    return 0


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), or "unknown"."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, plan, block, q_pre, k_pre, v_pre, q_dec, k_dec, v_dec, steps_dec, budget):
    """Times the fp64 oracle on a bounded sample of the same step and scales it.

    Prefill leg: the oracle's row-blocked dense-masked attention (blocks of
    1024 rows x all keys, BLAS products) over whole query heads of sequence 0,
    one head at a time, for about `budget` seconds.  Decode leg: decode tokens
    of sequence 0 (all heads, the first decode position) for about `budget`
    seconds.  The whole-step time is extrapolated by count: B * H_q prefill
    heads + B * steps decode tokens.
    """
    import numpy as np
    import torch
    import oracle

    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1

    B, N, Hq = wl.decode_batch, wl.n, wl.num_q_heads
    group = Hq // wl.num_kv_heads
    log("[bench] timing the CPU oracle on a bounded sample")
    qc, kc, vc = (x[0:1].cpu() for x in (q_pre, k_pre, v_pre))
    heads_done, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < budget or heads_done == 0:
        h = heads_done % Hq
        g = h // group
        oracle.attention_ref(qc[:, :, h:h + 1], kc[:, :, g:g + 1], vc[:, :, g:g + 1], [int(plan.window[g])],
                             wl.num_sink, block=block)
        heads_done += 1
    t_head = (time.perf_counter() - t0) / heads_done          # one head, all N rows
    t = N
    k_hist = torch.cat([kc, k_dec[0, 0:1].cpu()], dim=1)
    v_hist = torch.cat([vc, v_dec[0, 0:1].cpu()], dim=1)
    qt = q_dec[0, 0:1].cpu()
    dec_done, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < budget or dec_done == 0:
        oracle.decode_ref(qt, k_hist, v_hist, plan.window, wl.num_sink)
        dec_done += 1
    t_tok = (time.perf_counter() - t0) / dec_done            # one token, all heads
    step_s = B * Hq * t_head + B * steps_dec * t_tok
    return {
        "value": round(B * steps_dec / step_s, 4),
        "unit": "tokens/s",
        "cores": int(cores),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": (f"fp64 oracle on sequence 0: {heads_done} whole prefill heads ({N} rows each, row-blocked "
                   f"1024 x {N} BLAS products) and {dec_done} decode tokens x {Hq} heads at context {t}; "
                   f"extrapolated by count to the whole step ({B}x{Hq} prefill heads + {B}x{steps_dec} "
                   f"decode tokens)"),
        "seconds_per_prefill_head": t_head,
        "seconds_per_decode_token": t_tok,
        "extrapolated_step_s": step_s,
    }


if __name__ == "__main__":
    sys.exit(main())
