"""Host-side arithmetic of bench.py (no GPU): the FLOP counts its rates use."""

import numpy as np

import bench
import oracle
from paper_2609_18077_amd import inputs


def test_na3d_pair_count_matches_window_enumeration():
    """The separable product count equals enumerating every query's window."""
    for border in ("clip", "shift"):
        w = inputs.NaWorkload("count", B=2, H=3, grid=(4, 7, 9), seed=0, window=(3, 5, 11), border=border)
        T, Hp, Wp = w.grid
        n = sum(len(oracle.na3d.window_keys(t, h, x, w.grid, w.window, border))
                for t in range(T) for h in range(Hp) for x in range(Wp))
        assert bench.na3d_pairs(w) == n * w.B * w.H


def test_dense_flops_with_lengths():
    w = inputs.WORKLOADS["cross_text"]
    lv = np.array([100, 600])  # second clamps to Lk = 512
    assert bench.flops(w, lv) == 4 * w.H * w.Lq * w.d * (100 + 512)
    assert bench.flops(inputs.WORKLOADS["wan13b_480p"], None) == 6593848934400.0
