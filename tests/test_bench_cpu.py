"""Host-side pieces of bench.py: the in-band pair count used for FLOP accounting."""
import numpy as np
import pytest

import bench
import oracle


@pytest.mark.parametrize("n,w,s", [(1, 1, 0), (7, 3, 2), (50, 1, 0), (50, 50, 0), (50, 10, 60),
                                   (64, 17, 5), (200, 199, 1), (33, 40, 3)])
def test_visible_pairs_matches_mask_count(n, w, s):
    assert bench.visible_pairs(n, w, s) == int(oracle.visible_mask(n, n, w, s).sum())


def test_gpus_above_one_is_refused(monkeypatch, capsys):
    monkeypatch.setattr("sys.argv", ["bench.py", "--gpus", "2"])
    assert bench.main() == 2
    assert "one GPU" in capsys.readouterr().err
