"""GPU parity of the Q/K/V projection with the Q/K prologue in its epilogue
(vidax_qkv_proj) against the fp64 oracle, through the C ABI.

Tolerance.  The products of bf16 operands are exact in fp32; the fp32 sum of
the C terms (and the bias) is within C 2^-24 sum_c |x_c w_c| of the exact one
(the worst-case bound of a sum of C terms; it shows only where the terms
cancel), scaled for q and k by the RMS scale and gain; the RMS scale (fp32
reciprocal square root, ~1 ulp), the gain and the rotation (fp32 table) add a
few 2^-24 -- absolute, of the size of the rotary pair's norm, so they show
only where the rotation's two products cancel.  So every output is the
correctly rounded bf16 of the exact value except near a rounding boundary or
a cancellation: each element must be within one bf16 ulp of the reference
plus 2^-20 (1 + |angle|) of its pair's norm (the rotation kernel's bound), and
at least 99 % of them must equal its correctly rounded value."""

import numpy as np
import pytest

import oracle
import paper_2609_18077_amd as vx
from paper_2609_18077_amd import inputs
from tests.gpu_util import log, to_bits

pytestmark = pytest.mark.gpu


def _ulp_bf16(x):
    _, e = np.frexp(np.abs(x))
    return np.ldexp(1.0, np.maximum(e, -125) - 8)


def _dev(a, dtype):
    import torch

    if a is None:
        return None
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _spec(w, mode=0):
    return None if w.grid is None else oracle.RopeSpec(grid=w.grid, dims=w.dims, theta=w.theta, pair_mode=mode)


def _rope(w, mode=0):
    return None if w.grid is None else vx.Rope(w.grid, w.dims, w.theta, pair_mode=mode)


def _run(w, mode=0):
    import torch

    x, wt, bias, gq, gk = inputs.make_proj_inputs(w)
    q, k, v = vx.qkv_proj(_dev(x, "bf16"), _dev(wt, "bf16"), w.B, w.L, w.H, bias=_dev(bias, "f32"),
                          gain_q=_dev(gq, "f32"), gain_k=_dev(gk, "f32"), eps=w.eps, rope=_rope(w, mode))
    torch.cuda.synchronize()
    return (x, wt, bias, gq, gk), (to_bits(q), to_bits(k), to_bits(v))


def _sum_bounds(w, x, wt, bias, gq, gk, rows=None):
    """C 2^-24 sum_c |x_c w_c| (+ |bias|) per output, for q and k times the
    head's RMS scale and |gain| (the accumulated error of the fp32 sums)."""
    dec = oracle.bf16_bits_to_f64
    xs = dec(x) if rows is None else dec(x[rows])
    xw = np.abs(xs) @ np.abs(dec(wt)).T + (0.0 if bias is None else np.abs(bias))
    y = xs @ dec(wt).T + (0.0 if bias is None else bias)
    hd = w.H * w.d
    B, L = (w.B, w.L) if rows is None else (1, len(rows))
    out = []
    for p, g in enumerate((gq, gk, None)):
        t = w.C * 2.0 ** -24 * xw[:, p * hd:(p + 1) * hd].reshape(B, L, w.H, w.d)
        if p < 2:
            yy = y[:, p * hd:(p + 1) * hd].reshape(B, L, w.H, w.d)
            t = t / np.sqrt(np.mean(yy * yy, axis=-1, keepdims=True) + w.eps)
            if g is not None:
                t = t * np.abs(g)
        out.append(t)
    return out


def _check(got_bits, ref, what, extra, spec=None, rows=None):
    from tests.test_gpu_parity import _pair_norm_and_angle

    got = oracle.bf16_bits_to_f64(got_bits)
    err = np.abs(got - ref)
    bound = _ulp_bf16(ref) + extra + 1e-30
    if spec is not None:  # rotated: the pair norm is the same before and after the rotation
        norm, ang = _pair_norm_and_angle(ref, spec, np.arange(ref.shape[1]) if rows is None else rows)
        bound = bound + 2.0 ** -20 * norm * (1.0 + ang)
    exact = float(np.mean(got_bits == oracle.f64_to_bf16_bits(ref)))
    log(f"  {what}: max err/ulp {float((err / bound).max()):.3f} correctly rounded {exact:.5f}")
    assert np.all(np.isfinite(got)), what
    assert np.all(err <= bound), (what, float((err / bound).max()))
    assert exact >= 0.99, (what, exact)


PROJ = [
    # ragged token tile (300 = 256 + 44), rotation over a 2 x 5 x 25 grid + 50 unrotated tokens
    inputs.ProjWorkload("qkv_small", B=1, L=300, H=2, C=128, seed=51, grid=(2, 5, 25)),
    # two sequences (positions restart), odd head count (a half-filled channel tile), 3 stages
    inputs.ProjWorkload("qkv_odd_heads", B=2, L=130, H=3, C=192, seed=52, grid=(2, 5, 13)),
    # no bias, no gains, no rotation
    inputs.ProjWorkload("qkv_plain", B=1, L=257, H=4, C=256, seed=53, bias=False, gains=False),
    # one token, one head
    inputs.ProjWorkload("qkv_one", B=1, L=1, H=1, C=64, seed=54, grid=(1, 1, 1)),
]


def _random_proj_shapes(n=8, seed=2029):
    """Seeded random shapes: token counts off the 256-token tile, head counts
    that half-fill a channel tile, 1 to 6 stages of 64 input channels, a
    rotated prefix or none, with or without bias and gains."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B, L, H = int(rng.integers(1, 3)), int(rng.integers(1, 700)), int(rng.integers(1, 6))
        grid = None
        if rng.random() < 0.6:
            t, h, w = int(rng.integers(1, 3)), int(rng.integers(1, 6)), int(rng.integers(1, 30))
            if t * h * w <= L:
                grid = (t, h, w)
        cases.append(inputs.ProjWorkload(f"qkv_random{i}", B=B, L=L, H=H, C=64 * int(rng.integers(1, 7)),
                                         seed=400 + i, grid=grid, bias=bool(rng.random() < 0.7),
                                         gains=bool(rng.random() < 0.7)))
    return cases


PROJ += _random_proj_shapes()


@pytest.mark.parametrize("w", PROJ, ids=lambda w: w.name)
def test_qkv_proj_matches_oracle(w):
    log(f"case qkv {w.name} B{w.B} L{w.L} H{w.H} C{w.C} grid={w.grid}")
    (x, wt, bias, gq, gk), got = _run(w)
    dec = oracle.bf16_bits_to_f64
    ref = oracle.qkv_proj_ref(dec(x), dec(wt), bias, w.B, w.L, w.H, w.d, gq, gk, w.eps, _spec(w))
    sb = _sum_bounds(w, x, wt, bias, gq, gk)
    for name, g, r, e in zip("qkv", got, ref, sb):
        _check(g, r, name, e, _spec(w) if name != "v" else None)


@pytest.mark.parametrize("w", [PROJ[0], PROJ[1], PROJ[3]], ids=lambda w: w.name)
def test_qkv_proj_half_split_pairs(w):
    """Half-split rotary pairs (channel o_a + j with o_a + j + d_a/2) in the
    epilogue, against the oracle in that convention."""
    log(f"case qkv half split {w.name} B{w.B} L{w.L} H{w.H} C{w.C} grid={w.grid}")
    (x, wt, bias, gq, gk), got = _run(w, mode=1)
    dec = oracle.bf16_bits_to_f64
    ref = oracle.qkv_proj_ref(dec(x), dec(wt), bias, w.B, w.L, w.H, w.d, gq, gk, w.eps, _spec(w, 1))
    sb = _sum_bounds(w, x, wt, bias, gq, gk)
    for name, g, r, e in zip("qkv", got, ref, sb):
        _check(g, r, name, e, _spec(w, 1) if name != "v" else None)


def test_qkv_proj_full_size_sampled():
    """The Wan2.1-1.3B 480p projection: sampled tokens (first, last, tile and
    grid-row boundaries, random) of every head, exact per token."""
    w = inputs.PROJ_WORKLOADS["wan13b_480p_qkv"]
    log(f"case qkv {w.name} B{w.B} L{w.L} H{w.H} C{w.C} grid={w.grid}")
    (x, wt, bias, gq, gk), got = _run(w)
    rng = np.random.default_rng(11)
    rows = np.unique(np.r_[0, 1, 51, 52, 255, 256, 1559, 1560, w.L - 257, w.L - 256, w.L - 1,
                           rng.integers(0, w.L, 200)])
    dec = oracle.bf16_bits_to_f64
    ref = oracle.qkv_proj_ref(dec(x[rows]), dec(wt), bias, 1, len(rows), w.H, w.d, gq, gk, w.eps, _spec(w),
                              token_index=rows)
    sb = _sum_bounds(w, x, wt, bias, gq, gk, rows)
    for name, g, r, e in zip("qkv", got, ref, sb):
        _check(g[:, rows], r, name, e, _spec(w) if name != "v" else None, rows)
