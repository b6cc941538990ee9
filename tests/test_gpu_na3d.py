"""GPU parity of the 3D neighbourhood attention (vidax_na3d_fwd) against the
fp64 oracle, through the C ABI: every output element at small and medium
grids (ragged query blocks in every axis, grids smaller than the window, both
border readings, several windows and scales), sampled rows at the full-size
workload, with the contract of the dense forward (max-abs <= 2e-2, mean-abs
<= 2e-3, rel-RMS <= 1e-2; lse max-abs <= 2e-2)."""

import numpy as np
import pytest

import oracle
import paper_2609_18077_amd as vx
from paper_2609_18077_amd import inputs
from tests.gpu_util import assert_lse, assert_parity, log, to_bits, to_dev

pytestmark = pytest.mark.gpu


def _case(w, scale=None, rows=None):
    import torch

    q, k, v = inputs.make_na_qkv(w)
    scale = w.scale if scale is None else scale
    log(f"case na3d {w.name} B{w.B} H{w.H} grid={w.grid} window={w.window} border={w.border} scale={scale}")
    o, lse = vx.na3d_fwd(to_dev(q), to_dev(k), to_dev(v), w.grid, w.window, w.border, scale=scale, return_lse=True)
    torch.cuda.synchronize()
    ob, lb = to_bits(o), lse.cpu().numpy()
    dec = oracle.bf16_bits_to_f64
    ro, rl = oracle.na3d_ref(dec(q), dec(k), dec(v), scale, w.grid, w.window, w.border, rows=rows, workers=8)
    if rows is not None:
        ob, lb = ob[:, rows], lb[:, :, rows]
    assert_parity(ob, ro, w.name)
    assert_lse(lb, rl, w.name)


NA = [
    inputs.NaWorkload("na_tiny", B=1, H=2, grid=(2, 4, 4), seed=71, window=(3, 3, 3)),
    # ragged blocks in t, h and w; the 11^3 window larger than two axes
    inputs.NaWorkload("na_ragged", B=2, H=2, grid=(5, 9, 13), seed=72),
    inputs.NaWorkload("na_ragged_shift", B=1, H=3, grid=(5, 9, 13), seed=73, border="shift"),
    # interior queries with the full window, both readings
    inputs.NaWorkload("na_interior", B=1, H=2, grid=(13, 14, 15), seed=74),
    inputs.NaWorkload("na_interior_shift", B=1, H=2, grid=(13, 14, 15), seed=75, border="shift"),
    # asymmetric windows, a 1-wide window, windows wider than the grid
    inputs.NaWorkload("na_asym", B=1, H=2, grid=(6, 10, 17), seed=76, window=(3, 7, 5)),
    inputs.NaWorkload("na_asym_shift", B=1, H=2, grid=(6, 10, 17), seed=77, window=(5, 1, 9), border="shift"),
    inputs.NaWorkload("na_single_key", B=1, H=1, grid=(3, 5, 6), seed=78, window=(1, 1, 1)),
    inputs.NaWorkload("na_wide", B=1, H=1, grid=(1, 3, 2), seed=79, window=(11, 11, 11), border="shift"),
    inputs.NaWorkload("na_one_token", B=2, H=1, grid=(1, 1, 1), seed=80),
]


@pytest.mark.parametrize("w", NA, ids=lambda w: w.name)
def test_na3d_matches_oracle(w):
    _case(w)


def _random_na_shapes(n=10, seed=2028):
    """Seeded random grids (ragged query blocks in every axis), odd windows of
    1 to 11 per axis, either border reading."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        grid = (int(rng.integers(1, 9)), int(rng.integers(1, 17)), int(rng.integers(1, 25)))
        window = tuple(int(2 * rng.integers(0, 6) + 1) for _ in range(3))
        border = "shift" if rng.random() < 0.5 else "clip"
        cases.append(inputs.NaWorkload(f"na_random{i}", B=int(rng.integers(1, 3)), H=int(rng.integers(1, 3)),
                                       grid=grid, seed=300 + i, window=window, border=border))
    return cases


@pytest.mark.parametrize("w", _random_na_shapes(), ids=lambda w: w.name)
def test_na3d_random_shapes(w):
    _case(w)


@pytest.mark.parametrize("scale", [0.0, -0.2, 0.5])
def test_na3d_scale_values(scale):
    _case(inputs.NaWorkload("na_scale", B=1, H=2, grid=(4, 6, 9), seed=81, window=(3, 5, 7)), scale=scale)


def test_na3d_single_key_is_value_row():
    """A 1 x 1 x 1 window returns each token's own v row, bit for bit."""
    import torch

    w = inputs.NaWorkload("na_single_bits", B=1, H=2, grid=(2, 3, 7), seed=82, window=(1, 1, 1))
    q, k, v = inputs.make_na_qkv(w)
    o = vx.na3d_fwd(to_dev(q), to_dev(k), to_dev(v), w.grid, w.window)
    torch.cuda.synchronize()
    assert np.array_equal(to_bits(o), v)


def test_na3d_empty_calls():
    import torch

    for grid in ((0, 4, 4), (2, 0, 3)):
        x = torch.zeros((1, 0, 2, 128), dtype=torch.bfloat16, device="cuda")
        vx.na3d_fwd(x, x.clone(), x.clone(), grid)
    torch.cuda.synchronize()


def test_na3d_full_size_sampled():
    """The benchmark's workload: sampled query rows, including the corners and
    edges of the grid and the boundaries of the query blocks."""
    w = inputs.NA_WORKLOADS["ltx_vae_na"]
    T, Hp, Wp = w.grid
    rng = np.random.default_rng(9)
    pts = [(t, h, ww) for t in (0, 1, T - 1) for h in (0, 3, 4, Hp - 1) for ww in (0, 3, 4, Wp - 1)]
    rows = np.unique(np.r_[[(t * Hp + h) * Wp + ww for t, h, ww in pts], rng.integers(0, w.L, 96)])
    _case(w, rows=rows)
