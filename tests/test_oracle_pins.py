"""The oracle against its pins (closed forms, identities, brute force, torch)."""

import numpy as np
import pytest

import oracle
from oracle import RopeSpec, attn_ref, attn_ref_rows, rope3d_ref
from tests import pins


@pytest.mark.parametrize("check", pins.ALL_ROPE_CHECKS, ids=lambda c: c.__name__)
def test_rope_pins(check):
    check(rope3d_ref, RopeSpec)


def test_attn_brute():
    pins.check_attn_brute(attn_ref, RopeSpec)


def test_attn_torch():
    pins.check_attn_torch(attn_ref)


def test_attn_invariants():
    pins.check_attn_invariants(attn_ref, RopeSpec)


def test_rows_and_threads_agree_with_full():
    rng = np.random.default_rng(1)
    B, L, H, d = 2, 600, 2, 128
    q, k, v = (rng.standard_normal((B, L, H, d)) for _ in range(3))
    spec = RopeSpec(grid=(2, 10, 25), dims=(44, 42, 42))
    lv = [600, 311]
    o, lse = attn_ref(q, k, v, 0.088, kv_valid_len=lv, rope=spec, block=128)
    o4, lse4 = attn_ref(q, k, v, 0.088, kv_valid_len=lv, rope=spec, block=97, workers=4)
    assert np.allclose(o, o4, rtol=1e-13, atol=1e-15) and np.allclose(lse, lse4, rtol=1e-14)
    rows = np.array([0, 1, 255, 256, 499, 500, 599])
    orow, lrow = attn_ref_rows(q, k, v, 0.088, rows, kv_valid_len=lv, rope=spec)
    assert np.allclose(orow, o[:, rows], rtol=1e-13, atol=1e-15)
    assert np.allclose(lrow, lse[:, :, rows], rtol=1e-14)


def test_bf16_codec():
    # exact decode of known bit patterns
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000, 0x8000, 0x7F7F, 0x0001], np.uint16)
    vals = oracle.bf16_bits_to_f64(bits)
    assert vals[0] == 1.0 and vals[1] == -1.0 and vals[2] == 3.140625
    assert vals[3] == 0.0 and vals[5] == 3.3895313892515355e38 and vals[6] == 2.0 ** -133
    # round to nearest even at the halfway point between 1 and the next bfloat16
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -30, -2.5])
    r = oracle.bf16_bits_to_f64(oracle.f64_to_bf16_bits(x))
    assert list(r) == [1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7, -2.5]


@pytest.mark.parametrize("check", pins.ALL_NORM_CHECKS, ids=lambda c: c.__name__)
def test_norm_pins(check):
    check(oracle.qk_norm_ref, oracle.RopeSpec)


@pytest.mark.parametrize("check", pins.ALL_BWD_CHECKS, ids=lambda c: c.__name__)
def test_bwd_pins(check):
    check(oracle.attn_bwd_ref, oracle.attn_ref)


def test_rope_transpose_pin():
    pins.check_rope_transpose(oracle.rope_transpose_ref, oracle.rope3d_ref, oracle.RopeSpec)


def _bwd_rows_all(q, k, v, do, scale, kv_valid_len=None):
    return oracle.attn_bwd_ref_rows(q, k, v, do, scale, np.arange(q.shape[1]), np.arange(k.shape[1]),
                                    kv_valid_len=kv_valid_len)


@pytest.mark.parametrize("check", pins.ALL_BWD_CHECKS[:3], ids=lambda c: c.__name__)
def test_bwd_rows_pins(check):
    """The row-sampled gradient, asked for every row, meets the same pins."""
    check(_bwd_rows_all, oracle.attn_ref)


def test_bwd_rows_subset():
    rng = np.random.default_rng(56)
    q, k, v, do = (rng.standard_normal(s) for s in ((2, 11, 2, 8), (2, 9, 2, 8), (2, 9, 2, 8), (2, 11, 2, 8)))
    lv = np.array([9, 4])
    qr, kr = np.array([10, 0, 3]), np.array([8, 1, 5, 3])
    dq, dk, dv = _bwd_rows_all(q, k, v, do, 0.4, kv_valid_len=lv)
    sq, sk, sv = oracle.attn_bwd_ref_rows(q, k, v, do, 0.4, qr, kr, kv_valid_len=lv)
    assert np.allclose(sq, dq[:, qr], rtol=1e-13, atol=1e-14)
    assert np.allclose(sk, dk[:, kr], rtol=1e-13, atol=1e-14)
    assert np.allclose(sv, dv[:, kr], rtol=1e-13, atol=1e-14)
    assert np.all(sk[1, [0, 2]] == 0) and np.all(sv[1, [0, 2]] == 0)  # keys 8, 5 >= Lv = 4


@pytest.mark.parametrize("check", pins.ALL_NA_CHECKS, ids=lambda c: c.__name__)
def test_na_pins(check):
    check(oracle.na3d_ref, oracle.attn_ref)


@pytest.mark.parametrize("check", pins.ALL_QKV_CHECKS, ids=lambda c: c.__name__)
def test_qkv_pins(check):
    check(oracle.qkv_proj_ref, oracle.RopeSpec)
