"""bench.py end to end on the small fp32 workload: one JSON line with every
field of the benchmark contract, rooflines and the oracle's CPU baseline."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line_carries_the_contract():
    print("[case] bench.py small-mha4-d64-n512-f32", flush=True)
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "small-mha4-d64-n512-f32",
           "--steps", "2", "--warmup", "1", "--cpu-budget", "0.5", "--configs-reps", "8"]
    r = subprocess.run(cmd, cwd=ROOT, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    for key, typ in (("metric", str), ("value", float), ("unit", str), ("n_gpus", int), ("steps", int),
                     ("warmup", int), ("ms_per_step", float), ("higher_is_better", bool), ("scaling", str),
                     ("dtype", str), ("data", str), ("config", dict)):
        assert isinstance(d[key], typ), key
    assert "vs_baseline" in d and d["vs_baseline"] is None
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1 and d["value"] > 0
    assert d["dtype"] == "f32" and d["config"]["workload"] == "small-mha4-d64-n512-f32"
    roof = d["roofline"]
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert roof["achieved"] > 0 and abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    assert "traffic" in roof
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1 and cpu["sample"]
    assert cpu["cpu_model"]
    # the other workload shapes: prefill of three, decode of the two GQA layers
    cfg = d["configs"]
    assert set(cfg) == {"vicuna7b-prefill-n4096", "llama3-8b-gqa-n16384", "llama3-70b-gqa-n32768"}
    for name, entry in cfg.items():
        pre = entry["prefill"]
        assert pre["inband_tflops"] > 0 and abs(pre["frac"] - pre["inband_tflops"] / pre["peak"]) < 1e-3
        if name != "vicuna7b-prefill-n4096":
            dec = entry["decode"]
            assert dec["cache_sets"] >= 4 and dec["hbm_gbs"] > 0
            assert abs(dec["frac"] - dec["hbm_gbs"] / dec["peak"]) < 1e-3
