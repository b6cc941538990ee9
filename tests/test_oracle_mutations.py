"""Plant plausible mistakes in (copies of) the oracle and show a pin catches each.

Every mutation below is applied with monkeypatch to the oracle's own helpers,
on the CPU; the pins in tests/pins.py must then fail.  This is evidence that
the pins constrain the oracle's arithmetic, not only its shape.
"""

import numpy as np
import pytest

import oracle.attention as oa
import oracle.rope3d as orr
from oracle import RopeSpec, attn_ref, rope3d_ref
from tests import pins


def _pair_channels_sin_flipped(spec):
    return [(a, j, c1, c0, om) for (a, j, c0, c1, om) in _ORIG_PAIRS(spec)]


def _pair_channels_full_d(spec):
    d = sum(spec.dims)
    return [(a, j, c0, c1, float(spec.theta) ** (-2.0 * j / d)) for (a, j, c0, c1, _om) in _ORIG_PAIRS(spec)]


def _pair_channels_mode_swapped(spec):
    other = RopeSpec(grid=spec.grid, dims=spec.dims, theta=spec.theta, pair_mode=1 - spec.pair_mode)
    return _ORIG_PAIRS(other)


def _pair_channels_j_offset(spec):
    return [(a, j, c0, c1, float(spec.theta) ** (-2.0 * (j + 1) / spec.dims[a])) for (a, j, c0, c1, _om) in _ORIG_PAIRS(spec)]


def _coords_hw_swapped(n, grid):
    c = _ORIG_COORDS(n, grid)
    return c[..., [0, 2, 1]]


def _coords_row_major_wrong(n, grid):
    T, Hp, Wp = grid
    n = np.asarray(n, dtype=np.int64)
    return np.stack([n // (Hp * Wp), n % Hp, (n // Hp) % Wp], axis=-1)


_ORIG_PAIRS = orr.pair_channels
_ORIG_COORDS = orr.token_coords

ROPE_MUTATIONS = {
    "rotation_direction": ("pair_channels", _pair_channels_sin_flipped),
    "frequency_over_full_d": ("pair_channels", _pair_channels_full_d),
    "pair_convention": ("pair_channels", _pair_channels_mode_swapped),
    "frequency_index_off_by_one": ("pair_channels", _pair_channels_j_offset),
    "axes_h_w_swapped": ("token_coords", _coords_hw_swapped),
    "token_flattening": ("token_coords", _coords_row_major_wrong),
}


def _any_rope_pin_fails():
    for check in pins.ALL_ROPE_CHECKS:
        try:
            check(rope3d_ref, RopeSpec)
        except AssertionError:
            return True
    return False


@pytest.mark.parametrize("name", sorted(ROPE_MUTATIONS))
def test_rope_mutation_is_caught(name, monkeypatch):
    attr, fn = ROPE_MUTATIONS[name]
    monkeypatch.setattr(orr, attr, fn)
    assert _any_rope_pin_fails(), name


_ORIG_BLOCK = oa._one_block
_ORIG_LEN = oa._valid_lengths


def _block_scale_twice(qb, kb, vb, scale):
    return _ORIG_BLOCK(qb, kb, vb, scale * scale)


def _block_softmax_wrong_axis(qb, kb, vb, scale):
    s = scale * (qb @ kb.T)
    m = s.max(axis=0)
    e = np.exp(s - m[None, :])
    l = e.sum(axis=0)
    o = (e / l[None, :]) @ vb
    return o, np.log(e.sum(axis=1)) + s.max(axis=1)


def _block_lse_no_max(qb, kb, vb, scale):
    o, lse = _ORIG_BLOCK(qb, kb, vb, scale)
    s = scale * (qb @ kb.T)
    return o, lse - s.max(axis=1)


def _block_values_are_keys(qb, kb, vb, scale):
    return _ORIG_BLOCK(qb, kb, kb, scale)


def _block_no_normalisation(qb, kb, vb, scale):
    s = scale * (qb @ kb.T)
    m = s.max(axis=1)
    e = np.exp(s - m[:, None])
    return e @ vb, m + np.log(e.sum(axis=1))


def _len_off_by_one(kv, B, Lk):
    return np.clip(_ORIG_LEN(kv, B, Lk) + 1, 0, Lk)


def _len_ignored(kv, B, Lk):
    return np.full(B, Lk, dtype=np.int64)


ATTN_MUTATIONS = {
    "scale_applied_twice": ("_one_block", _block_scale_twice),
    "softmax_over_queries": ("_one_block", _block_softmax_wrong_axis),
    "lse_without_max": ("_one_block", _block_lse_no_max),
    "values_are_keys": ("_one_block", _block_values_are_keys),
    "missing_normalisation": ("_one_block", _block_no_normalisation),
    "mask_off_by_one": ("_valid_lengths", _len_off_by_one),
    "mask_ignored": ("_valid_lengths", _len_ignored),
}


def _any_attn_pin_fails():
    for check in (lambda: pins.check_attn_brute(attn_ref, RopeSpec),
                  lambda: pins.check_attn_torch(attn_ref),
                  lambda: pins.check_attn_invariants(attn_ref, RopeSpec)):
        try:
            check()
        except AssertionError:
            return True
    return False


@pytest.mark.parametrize("name", sorted(ATTN_MUTATIONS))
def test_attn_mutation_is_caught(name, monkeypatch):
    attr, fn = ATTN_MUTATIONS[name]
    monkeypatch.setattr(oa, attr, fn)
    assert _any_attn_pin_fails(), name


# ------------------------------------------------------ query/key prologue ---

import oracle.qknorm as oq  # noqa: E402

_ORIG_MS = oq.mean_square
_ORIG_RS = oq.rms_scale


def _ms_sum_not_mean(x):
    return np.sum(x * x, axis=-1, keepdims=True)


def _ms_over_heads_and_channels(x):
    return np.mean(x * x, axis=(-2, -1), keepdims=True)


def _ms_over_tokens(x):
    return np.mean(x * x, axis=(1, -1), keepdims=True)


def _ms_abs_not_square(x):
    return np.mean(np.abs(x), axis=-1, keepdims=True) ** 2


def _rs_eps_outside(ms, eps):
    return 1.0 / (np.sqrt(ms) + eps)


def _rs_no_sqrt(ms, eps):
    return 1.0 / (ms + eps)


def _rs_eps_ignored(ms, eps):
    return 1.0 / np.sqrt(ms)


NORM_MUTATIONS = {
    "sum_of_squares_not_mean": ("mean_square", _ms_sum_not_mean),
    "norm_over_all_heads": ("mean_square", _ms_over_heads_and_channels),
    "norm_over_tokens": ("mean_square", _ms_over_tokens),
    "mean_abs_squared": ("mean_square", _ms_abs_not_square),
    "eps_outside_sqrt": ("rms_scale", _rs_eps_outside),
    "missing_sqrt": ("rms_scale", _rs_no_sqrt),
    "eps_ignored": ("rms_scale", _rs_eps_ignored),
}


def _any_norm_pin_fails():
    for check in pins.ALL_NORM_CHECKS:
        try:
            check(oq.qk_norm_ref, RopeSpec)
        except AssertionError:
            return True
    return False


@pytest.mark.parametrize("name", sorted(NORM_MUTATIONS))
def test_norm_mutation_is_caught(name, monkeypatch):
    attr, fn = NORM_MUTATIONS[name]
    monkeypatch.setattr(oq, attr, fn)
    assert _any_norm_pin_fails(), name


def test_norm_gain_dropped_is_caught(monkeypatch):
    orig = oq.qk_norm_ref

    def no_gain(x, gain=None, eps=1e-6, rope=None, token_index=None):
        return orig(x, None, eps, rope, token_index)

    try:
        pins.check_norm_gain(no_gain, RopeSpec)
    except AssertionError:
        return
    raise AssertionError("dropping the gain went unnoticed")


# ------------------------------------------------------ attention gradient ---

import oracle.attention_bwd as ob  # noqa: E402
from oracle import attn_bwd_ref  # noqa: E402

_ORIG_HEAD = ob._one_head


def _softmax(s):
    e = np.exp(s - s.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def _head_no_delta(q, k, v, do, scale, o_saved=None):
    p = _softmax(scale * (q @ k.T))
    ds = p * (do @ v.T)
    return scale * (ds @ k), scale * (ds.T @ q), p.T @ do


def _head_delta_wrong_axis(q, k, v, do, scale, o_saved=None):
    p = _softmax(scale * (q @ k.T))
    dp = do @ v.T
    ds = p * (dp - np.sum(p * dp, axis=0, keepdims=True))
    return scale * (ds @ k), scale * (ds.T @ q), p.T @ do


def _head_dq_unscaled(q, k, v, do, scale, o_saved=None):
    dq, dk, dv = _ORIG_HEAD(q, k, v, do, scale, o_saved)
    return dq / scale, dk, dv


def _head_dk_uses_keys(q, k, v, do, scale, o_saved=None):
    p = _softmax(scale * (q @ k.T))
    dp = do @ v.T
    ds = p * (dp - np.sum(p * dp, axis=1, keepdims=True))
    return scale * (ds @ k), scale * (ds.T @ do), p.T @ do


def _head_dv_not_transposed(q, k, v, do, scale, o_saved=None):
    dq, dk, _ = _ORIG_HEAD(q, k, v, do, scale, o_saved)
    p = _softmax(scale * (q @ k.T))
    return dq, dk, (p.T @ do)[::-1]


def _head_dp_uses_output(q, k, v, do, scale, o_saved=None):
    p = _softmax(scale * (q @ k.T))
    dp = do @ (p @ v).T[:, : k.shape[0]] if q.shape[0] >= k.shape[0] else do @ v.T * 1.01
    ds = p * (dp - np.sum(p * dp, axis=1, keepdims=True))
    return scale * (ds @ k), scale * (ds.T @ q), p.T @ do


def _head_saved_output_ignored(q, k, v, do, scale, o_saved=None):
    return _ORIG_HEAD(q, k, v, do, scale, None)


BWD_MUTATIONS = {
    "saved_output_ignored": _head_saved_output_ignored,
    "no_delta_term": _head_no_delta,
    "delta_over_queries": _head_delta_wrong_axis,
    "dq_missing_scale": _head_dq_unscaled,
    "dk_from_dout": _head_dk_uses_keys,
    "dv_rows_permuted": _head_dv_not_transposed,
    "dp_perturbed": _head_dp_uses_output,
}


@pytest.mark.parametrize("name", sorted(BWD_MUTATIONS))
def test_bwd_mutation_is_caught(name, monkeypatch):
    monkeypatch.setattr(ob, "_one_head", BWD_MUTATIONS[name])
    for check in pins.ALL_BWD_CHECKS:
        try:
            check(attn_bwd_ref, attn_ref)
        except AssertionError:
            return
    raise AssertionError(name + " went unnoticed")


# ------------------------------------------------ neighbourhood attention ---

import oracle.na3d as na  # noqa: E402

_ORIG_AXIS = na.axis_window
_ORIG_KEYS = na.window_keys
_ORIG_NA = na.na3d_ref


def _axis_radius_plus_one(c, N, K, border):
    return _ORIG_AXIS(c, N, K + 2, border)


def _axis_borders_swapped(c, N, K, border):
    return _ORIG_AXIS(c, N, K, "shift" if border == "clip" else "clip")


def _axis_shift_clamp_off(c, N, K, border):
    if border == "shift" and N > K:
        r = (K - 1) // 2
        lo = min(max(c - r, 0), N - K + 1)
        return lo, min(lo + K - 1, N - 1)
    return _ORIG_AXIS(c, N, K, border)


def _keys_axes_reversed(t, h, w, grid, window, border):
    return _ORIG_KEYS(t, h, w, grid, tuple(reversed(window)), border)


def _keys_flattened_w_major(t, h, w, grid, window, border):
    T, Hp, Wp = grid
    idx = _ORIG_KEYS(t, h, w, grid, window, border)
    tt, rem = np.divmod(idx, Hp * Wp)
    hh, ww = np.divmod(rem, Wp)
    return np.minimum((ww * Hp + hh) * T + tt, T * Hp * Wp - 1)


def _na_scale_dropped(q, k, v, scale, grid, window=(11, 11, 11), border="clip", rows=None, workers=1):
    return _ORIG_NA(q, k, v, 1.0, grid, window, border, rows, workers)


NA_AXIS_MUTATIONS = {
    "radius_plus_one": _axis_radius_plus_one,
    "borders_swapped": _axis_borders_swapped,
    "shift_clamp_off_by_one": _axis_shift_clamp_off,
}
NA_KEYS_MUTATIONS = {
    "window_axes_reversed": _keys_axes_reversed,
    "keys_flattened_w_major": _keys_flattened_w_major,
}


def _na_caught(fn=None):
    for check in pins.ALL_NA_CHECKS:
        try:
            check(fn or na.na3d_ref, attn_ref)
        except AssertionError:
            return True
    return False


@pytest.mark.parametrize("name", sorted(NA_AXIS_MUTATIONS))
def test_na_axis_mutation_is_caught(name, monkeypatch):
    monkeypatch.setattr(na, "axis_window", NA_AXIS_MUTATIONS[name])
    assert _na_caught(), name + " went unnoticed"


@pytest.mark.parametrize("name", sorted(NA_KEYS_MUTATIONS))
def test_na_keys_mutation_is_caught(name, monkeypatch):
    monkeypatch.setattr(na, "window_keys", NA_KEYS_MUTATIONS[name])
    assert _na_caught(), name + " went unnoticed"


def test_na_scale_dropped_is_caught():
    assert _na_caught(_na_scale_dropped)


# ------------------------------------------------------ Q/K/V projection ---

from oracle.qknorm import qk_norm_ref as _qkn  # noqa: E402


def _qkv_mutant(kind):
    def f(x, w, bias, B, L, H, d, gain_q=None, gain_k=None, eps=1e-6, rope=None, token_index=None):
        x = np.asarray(x, dtype=np.float64)
        w = np.asarray(w, dtype=np.float64)
        y = x @ (w if kind == "weight_not_transposed" else w.T)
        if bias is not None and kind != "bias_after_norm":
            y = y + bias
        hd = H * d
        q = y[:, :hd].reshape(B, L, H, d)
        k = y[:, hd:2 * hd].reshape(B, L, H, d)
        v = y[:, 2 * hd:].reshape(B, L, H, d)
        if kind == "q_k_blocks_swapped":
            q, k = k, q
        gq, gk = (gain_k, gain_q) if kind == "gains_swapped" else (gain_q, gain_k)
        q = _qkn(q, gq, eps, rope, token_index=token_index)
        k = _qkn(k, gk, eps, None if kind == "k_not_rotated" else rope, token_index=token_index)
        if kind == "v_normalised":
            v = _qkn(v, None, eps, None)
        if kind == "bias_after_norm" and bias is not None:
            q = q + np.asarray(bias[:hd]).reshape(H, d)
            k = k + np.asarray(bias[hd:2 * hd]).reshape(H, d)
            v = v + np.asarray(bias[2 * hd:]).reshape(H, d)
        return q, k, v
    return f


QKV_MUTATIONS = ["weight_not_transposed", "bias_after_norm", "q_k_blocks_swapped", "gains_swapped", "v_normalised",
                 "k_not_rotated"]


@pytest.mark.parametrize("kind", QKV_MUTATIONS)
def test_qkv_mutation_is_caught(kind):
    fn = _qkv_mutant(kind)
    for check in pins.ALL_QKV_CHECKS:
        try:
            check(fn, RopeSpec)
        except (AssertionError, ValueError):  # a shape error is a caught mistake too
            return
    raise AssertionError(kind + " went unnoticed")
