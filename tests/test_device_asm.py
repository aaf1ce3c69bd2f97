"""Checks on the gfx950 assembly of every kernel source, compiled here with the
library's own flags (no GPU needed).

* Each buffer-to-LDS DMA issued from inline asm follows an ``s_nop 4``: the
  compiler adds no hazard wait states around inline asm, and such a load may
  read descriptor SGPRs that a vector-ALU instruction (``v_readlane``) wrote
  just before, which this GPU family only allows after 5 wait states.
* Each lane swap (``v_permlane16_swap`` / ``v_permlane32_swap``, also inline
  asm) follows at least 2 wait states (``s_nop 1`` or longer), the count the
  compiler itself puts between a vector-ALU write and such a swap.
* No packed fp32 VALU forms are emitted (they are kept out of every kernel by
  the build flags).
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2406_14909_amd import build as B

pytestmark = pytest.mark.skipif(shutil.which(B.HIPCC) is None and not os.path.exists(B.HIPCC),
                                reason="hipcc not available")


@pytest.fixture(scope="module")
def device_asm(tmp_path_factory):
    """Assembly of a kernel source, compiled once per module."""
    cache = {}
    tmp = tmp_path_factory.mktemp("asm")

    def get(src: str) -> str:
        if src not in cache:
            out = tmp / (src + ".s")
            cmd = [B.HIPCC, *B.HIP_FLAGS, f"-I{B.INCLUDE}", f"-I{B.CSRC}", "--cuda-device-only", "-S",
                   os.path.join(B.CSRC, src), "-o", str(out)]
            r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
            assert r.returncode == 0, r.stdout.decode(errors="replace")
            cache[src] = out.read_text()
        return cache[src]

    return get


def _instructions(asm: str):
    """Instruction lines of the assembly, comments and directives dropped."""
    for line in asm.splitlines():
        t = line.split(";")[0].strip()
        if t and not t.startswith(".") and not t.endswith(":"):
            yield t


@pytest.mark.parametrize("src", B.HIP_SOURCES)
def test_lds_dma_after_hazard_wait_states(src, device_asm):
    ins = list(_instructions(device_asm(src)))
    dma = [i for i, t in enumerate(ins) if re.match(r"buffer_load_dword\w*\s.*\blds\b", t)]
    for i in dma:
        assert ins[i - 1] == "s_nop 4", f"{src}: DMA without wait states: {ins[i - 1]!r} / {ins[i]!r}"
    if src in ("prefill.hip", "influence.hip"):
        assert dma, f"{src} is expected to stage its tiles with LDS DMA"


@pytest.mark.parametrize("src", B.HIP_SOURCES)
def test_lane_swaps_after_wait_states(src, device_asm):
    ins = list(_instructions(device_asm(src)))
    for i, t in enumerate(ins):
        if re.match(r"v_permlane(16|32)_swap", t):
            m = re.match(r"s_nop (\d+)$", ins[i - 1])
            assert m and int(m.group(1)) >= 1, f"{src}: lane swap without wait states: {ins[i - 1]!r} / {t!r}"


@pytest.mark.parametrize("src", B.HIP_SOURCES)
def test_no_packed_fp32_forms(src, device_asm):
    asm = device_asm(src)
    found = sorted(set(re.findall(r"\bv_pk_(?:add|mul|fma|mov)_f32\b", asm)))
    assert not found, f"{src}: packed fp32 forms {found}"
