"""Host-side pieces of bench.py: the in-band pair count used for FLOP accounting."""
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
