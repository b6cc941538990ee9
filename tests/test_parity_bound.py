"""The per-element parity bound of the GPU tests (tests/gpu_util.py), on the
CPU: an output with the kernels' roundings passes it, and outputs with one
planted, localized mistake -- one channel of one 256-query tile scaled by
1.25, one channel of the ragged last tile 20% low, one row normalised by a wrong sum -- fail it, although each of them
still meets the contract's absolute bounds (max-abs 2e-2, mean-abs 2e-3) and
the relative-RMS guard."""

import numpy as np
import pytest

import oracle
from paper_2609_18077_amd import inputs
from tests.gpu_util import ELEM_ABS_OVER_RMS, MAX_ABS, MEAN_ABS, REL_RMS, element_excess, errors

# many keys, so that outputs are as small as at the benchmark shapes (|o| ~ 1e-2)
B, L, LK, H, D = 1, 600, 16384, 3, 128
SCALE = float(np.float32(1 / np.sqrt(D)))


def _inputs():
    w = inputs.custom("bound", B=B, H=H, Lq=L, Lk=LK, seed=41, grid=None)
    q, k, v, _ = inputs.make_qkv(w)
    return (oracle.bf16_bits_to_f64(x) for x in (q, k, v))


def _kernel_like(q, k, v):
    """The kernels' rounding model: probabilities rounded to bf16 before the
    weighted sum, the row sum over the same rounded weights, the output
    rounded to bf16."""
    out = np.empty_like(q)
    for h in range(H):
        s = SCALE * q[0, :, h] @ k[0, :, h].T
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p = oracle.bf16_bits_to_f64(oracle.f64_to_bf16_bits(p))
        out[0, :, h] = (p @ v[0, :, h]) / p.sum(axis=1, keepdims=True)
    return oracle.f64_to_bf16_bits(out)


@pytest.fixture(scope="module")
def case():
    q, k, v = _inputs()
    ref, _ = oracle.attn_ref(q, k, v, SCALE)
    return ref, _kernel_like(q, k, v)


def _contract_ok(got_bits, ref):
    e = errors(got_bits, ref)
    return e["max_abs"] <= MAX_ABS and e["mean_abs"] <= MEAN_ABS and e["rel_rms"] <= REL_RMS


def test_kernel_rounding_passes_with_margin(case):
    ref, got = case
    ex = element_excess(got, ref)
    assert _contract_ok(got, ref)
    assert ex <= ELEM_ABS_OVER_RMS / 2, ex


def _planted(got, fn):
    bad = got.copy()
    vals = oracle.bf16_bits_to_f64(bad)
    fn(vals)
    return oracle.f64_to_bf16_bits(vals)


@pytest.mark.parametrize("name", ["scaled_channel_in_tile", "low_channel_ragged_tile", "wrong_row_sum"])
def test_planted_mistake_is_caught(case, name):
    ref, got = case

    def scaled(x):  # head 1, query tile 1 (rows 256..511): channel 37 scaled by 1.25
        x[0, 256:512, 1, 37] *= 1.25

    def mixed(x):  # head 2, ragged last tile (rows 512..599): channel 100 20% low
        x[0, 512:, 2, 100] *= 0.8

    def row_sum(x):  # head 0: row 300 divided by a sum 10% too small
        x[0, 300, 0] /= 0.9

    bad = _planted(got, {"scaled_channel_in_tile": scaled, "low_channel_ragged_tile": mixed,
                         "wrong_row_sum": row_sum}[name])
    assert _contract_ok(bad, ref), "the planted mistake should be invisible to the absolute contract"
    assert element_excess(bad, ref) > ELEM_ABS_OVER_RMS
