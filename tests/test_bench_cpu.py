"""Host-side pieces of bench.py: the in-band pair count used for FLOP accounting and
the count of wave-tiles the prefill kernel multiplies."""
import numpy as np
import pytest

import bench
import oracle


@pytest.mark.parametrize("n,w,s", [(1, 1, 0), (7, 3, 2), (50, 1, 0), (50, 50, 0), (50, 10, 60),
                                   (64, 17, 5), (200, 199, 1), (33, 40, 3)])
def test_visible_pairs_matches_mask_count(n, w, s):
    assert bench.visible_pairs(n, w, s) == int(oracle.visible_mask(n, n, w, s).sum())


@pytest.mark.parametrize("n,w,s", [(1, 1, 0), (7, 3, 2), (200, 1, 0), (200, 64, 64), (200, 65, 3),
                                   (300, 130, 70), (129, 1000, 0), (64, 63, 5)])
def test_block_visible_pairs_matches_mask_count(n, w, s):
    assert bench.visible_pairs(n, w, s, 64) == int(oracle.visible_mask(n, n, w, s, block=64).sum())
    assert bench.visible_pairs(n, w, s, 4) == int(oracle.visible_mask(n, n, w, s, block=4).sum())


def test_gpus_above_one_is_refused(monkeypatch, capsys):
    monkeypatch.setattr("sys.argv", ["bench.py", "--gpus", "2"])
    assert bench.main() == 2
    assert "one GPU" in capsys.readouterr().err


def test_measured_traffic_needs_matching_sources(tmp_path, monkeypatch):
    import os
    prof = tmp_path / "profiles"
    prof.mkdir()
    src = tmp_path / "paper_2406_14909_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "k.hip").write_text("kernel v1")
    import hashlib
    h = hashlib.sha256(b"kernel v1").hexdigest()
    (prof / "t.md").write_text(f"traffic_bytes_per_launch: 1234\nsource_files: k.hip\nsource_sha256: {h}\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("t.md") == 1234
    (src / "k.hip").write_text("kernel v2")
    assert bench.measured_traffic("t.md") is None
    assert bench.measured_traffic("missing.md") is None


def _executed_wave_tiles_loop(n, w, s, block=0):
    """The prefill kernel's tile-visit rule written out as loops."""
    sh, W = (6, -(-w // 64)) if block else (0, w)
    band_start = lambda i: ((i >> sh) - W + 1) << sh
    count = 0
    for i0 in range(0, n, 128):
        i1 = min(n, i0 + 128)
        ta = (min(s, i1) + 63) // 64
        tl = (i1 - 1) // 64
        tb = max(ta, max(0, band_start(i0)) // 64)
        tiles = list(range(ta)) + list(range(tb, tl + 1))
        for iw0 in range(i0, i1, 32):
            iw1 = min(i1, iw0 + 32)
            for t in tiles:
                j0 = 64 * t
                if j0 <= iw1 - 1 and (j0 < s or band_start(iw0) <= j0 + 63):
                    count += 1
    return count


@pytest.mark.parametrize("n,w,s,block", [(1, 1, 0, 0), (100, 1, 0, 0), (300, 50, 4, 0), (1000, 1000, 0, 0),
                                         (1000, 130, 64, 0), (777, 65, 200, 0), (2049, 700, 3, 0),
                                         (1000, 130, 64, 64), (900, 1, 64, 64), (2049, 700, 0, 64)])
def test_executed_wave_tiles_matches_loop(n, w, s, block):
    assert bench.executed_wave_tiles(n, w, s, block) == _executed_wave_tiles_loop(n, w, s, block)


@pytest.mark.parametrize("n,w,s,block", [(300, 50, 4, 0), (1000, 130, 64, 0), (777, 65, 200, 0),
                                         (1000, 130, 64, 64), (257, 1, 0, 0), (700, 2000, 5, 0),
                                         (640, 64, 0, 64)])
def test_executed_wave_tiles_are_the_tiles_holding_visible_pairs(n, w, s, block):
    # The kernel multiplies exactly the (32-row wave, 64-key tile) pairs that
    # hold a visible (row, key) pair: none is skipped, none is extra.
    mask = oracle.visible_mask(n, n, w, s, block=block) if block else oracle.visible_mask(n, n, w, s)
    needed = {(i // 32, j // 64) for i, j in zip(*np.nonzero(mask))}
    assert bench.executed_wave_tiles(n, w, s, block) == len(needed)
