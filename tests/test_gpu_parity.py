"""GPU parity of the HIP path against the fp64 oracle (through the C ABI).

Small and medium cases compare every output element; the full-size workloads
(the launch configuration the benchmark times) compare sampled query rows,
which the oracle computes exactly (rows are independent), and check a
property over every output element: each output is a convex combination of
the valid value rows, so every component lies within their per-channel range.
"""

import numpy as np
import pytest

import oracle
import paper_2609_18077_amd as vx
from paper_2609_18077_amd import inputs
from tests.gpu_util import (assert_lse, assert_parity, errors, lengths_dev, log, rope_of, spec_of, to_bits,
                            to_dev)

pytestmark = pytest.mark.gpu


def _run(w: inputs.Workload, q, k, v, lv, impl=vx.attn_fwd, lse=True):
    import torch

    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    res = impl(qd, kd, vd, scale=w.scale, kv_valid_len=lengths_dev(lv), rope=rope_of(w), return_lse=lse)
    torch.cuda.synchronize()
    if lse:
        o, l = res
        return to_bits(o), l.cpu().numpy()
    return to_bits(res), None


def _oracle_full(w, q, k, v, lv):
    dec = oracle.bf16_bits_to_f64
    return oracle.attn_ref(dec(q), dec(k), dec(v), w.scale, kv_valid_len=lv, rope=spec_of(w), workers=8)


def _full_case(w, impl=vx.attn_fwd, q=None, k=None, v=None, lv="default"):
    if q is None:
        q, k, v, lv0 = inputs.make_qkv(w)
        if lv == "default":
            lv = lv0
    elif lv == "default":
        lv = None
    log(f"case {w.name} B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk} lv={None if lv is None else list(lv)} impl={impl.__name__}")
    ob, lse = _run(w, q, k, v, lv, impl)
    ro, rl = _oracle_full(w, q, k, v, lv)
    assert_parity(ob, ro, w.name)
    assert_lse(lse, rl, w.name)
    return ob


# ---------------------------------------------------------------- rope3d ----

def _ulp_bf16(x):
    m, e = np.frexp(np.abs(x))
    return np.ldexp(1.0, np.maximum(e, -125) - 8)


def _pair_norm_and_angle(x, spec, rows):
    """|(x0, x1)| of the rotary pair each channel belongs to, and that pair's
    angle (0 for unrotated tokens), broadcast to x's [B, R, H, d] shape."""
    from oracle.rope3d import pair_channels

    d = x.shape[-1]
    pairs = pair_channels(spec)
    partner = np.empty(d, np.int64)
    chan_pair = np.empty(d, np.int64)
    for p, (_a, _j, c0, c1, _om) in enumerate(pairs):
        partner[c0], partner[c1] = c1, c0
        chan_pair[c0] = chan_pair[c1] = p
    rows = np.asarray(rows)
    phi = np.zeros((len(rows), len(pairs)))
    rot = rows < spec.n_rot
    if rot.any():
        phi[rot] = oracle.rope_angles(spec, rows[rot])
    ang = phi[:, chan_pair][None, :, None, :]
    return np.sqrt(x * x + x[..., partner] ** 2), np.abs(ang)


def _rope_bound(x, ref, spec, rows):
    """One bf16 ulp of the result plus the fp32 evaluation error of the
    rotation: the angle pos * omega and its sine/cosine carry a relative error
    of a few 2^-24 (absolute ~|phi| 2^-22), and the two products of the pair
    (magnitude <= |pair|) are rounded to 24 bits.  These only show where the
    two products cancel; elsewhere the bf16 rounding dominates."""
    norm, ang = _pair_norm_and_angle(x, spec, rows)
    return _ulp_bf16(ref) + 2.0 ** -20 * norm * (1.0 + ang) + 1e-30


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("inplace", [False, True])
@pytest.mark.parametrize("heads", [3, 6])  # head rows are handled four at a time, then one by one
def test_rope3d_matches_oracle(mode, inplace, heads):
    import torch

    grid = (3, 10, 30)  # 900 video tokens, then 100 unrotated tokens
    x = inputs.bf16_tensor(11, 0, (2, 1000, heads, 128))
    log(f"case rope3d mode={mode} inplace={inplace} heads={heads}")
    xd = to_dev(x)
    r = vx.Rope(grid=grid, dims=(44, 42, 42), theta=10000.0, pair_mode=mode)
    y = vx.rope3d(xd, r, out=xd if inplace else None)
    torch.cuda.synchronize()
    got = oracle.bf16_bits_to_f64(to_bits(y))
    spec = oracle.RopeSpec(grid=grid, pair_mode=mode)
    ref = oracle.rope3d_ref(oracle.bf16_bits_to_f64(x), spec)
    err = np.abs(got - ref)
    bound = _rope_bound(oracle.bf16_bits_to_f64(x), ref, spec, np.arange(x.shape[1]))
    assert np.all(err <= bound), (err.max(), float((err / bound).max()))
    exact = np.mean(to_bits(y) == oracle.f64_to_bf16_bits(ref))
    log(f"  correctly rounded fraction {exact:.5f}")
    assert exact > 0.995
    assert np.array_equal(to_bits(y)[:, 900:], x[:, 900:])


def test_rope3d_full_size_wan13b():
    import torch

    w = inputs.WORKLOADS["wan13b_480p"]
    k = inputs.bf16_tensor(w.seed, inputs.T_K, (w.B, w.Lk, w.H, w.d), rms_norm=True)
    log("case rope3d wan13b_480p K")
    y = vx.rope3d(to_dev(k), rope_of(w))
    torch.cuda.synchronize()
    yb = to_bits(y)
    rows = np.unique(np.r_[0, 1, 51, 52, 1559, 1560, w.Lk - 1, np.random.default_rng(0).integers(0, w.Lk, 300)])
    ref = oracle.rope3d_ref(oracle.bf16_bits_to_f64(k[:, rows]), spec_of(w), token_index=rows)
    got = oracle.bf16_bits_to_f64(yb[:, rows])
    assert np.all(np.abs(got - ref) <= _rope_bound(oracle.bf16_bits_to_f64(k[:, rows]), ref, spec_of(w), rows))


# ------------------------------------------------- query/key prologue ---

def _norm_bound(x, gain, eps, ref, spec, rows):
    """One bf16 ulp of the result, the fp32 normalisation (sum of 128 squares,
    reciprocal square root, two products: relative 2^-16 at most) and, for
    rotated tokens, the rotation's fp32 error as in _rope_bound, all relative
    to the normalised pair's norm."""
    y = oracle.qk_norm_ref(x, gain=gain, eps=eps)
    if spec is None:
        return _ulp_bf16(ref) + 2.0 ** -16 * np.abs(y) + 1e-30
    norm, ang = _pair_norm_and_angle(y, spec, rows)
    return _ulp_bf16(ref) + (2.0 ** -16 + 2.0 ** -20 * (1.0 + ang)) * norm + 1e-30


def _head_scaled(seed, shape, exps):
    """bf16 N(0,1) tensor with head h scaled by 2**exps[h] (exact in bf16)."""
    x = oracle.bf16_bits_to_f64(inputs.bf16_tensor(seed, 0, shape))
    x = x * (2.0 ** np.asarray(exps, np.float64))[None, None, :, None]
    return oracle.f64_to_bf16_bits(x)


@pytest.mark.parametrize("rotate,with_gain,inplace", [(False, False, False), (False, True, False),
                                                     (True, True, False), (True, False, True),
                                                     ("half", True, False), ("half", False, True)])
@pytest.mark.parametrize("heads", [3, 6])  # head rows are handled four at a time, then one by one
def test_qk_norm_rope_matches_oracle(rotate, with_gain, inplace, heads):
    import torch

    grid = (3, 10, 30)  # 900 video tokens, then 100 unrotated tokens
    x = _head_scaled(12, (2, 1000, heads, 128), [-6, 0, 5, 2, -3, 1][:heads])
    g = np.random.default_rng(13).uniform(0.5, 1.5, 128).astype(np.float32)
    eps = 1e-6
    log(f"case qk_norm_rope rotate={rotate} gain={with_gain} inplace={inplace} heads={heads}")
    xd = to_dev(x)
    gd = torch.from_numpy(g).cuda() if with_gain else None
    mode = 1 if rotate == "half" else 0  # "half": half-split pairs
    r = vx.Rope(grid=grid, dims=(44, 42, 42), theta=10000.0, pair_mode=mode) if rotate else None
    y = vx.qk_norm_rope(xd, r, gain=gd, eps=eps, out=xd if inplace else None)
    torch.cuda.synchronize()
    got = oracle.bf16_bits_to_f64(to_bits(y))
    spec = oracle.RopeSpec(grid=grid, pair_mode=mode) if rotate else None
    xf = oracle.bf16_bits_to_f64(x)
    gain = g.astype(np.float64) if with_gain else None
    ref = oracle.qk_norm_ref(xf, gain=gain, eps=eps, rope=spec)
    err = np.abs(got - ref)
    bound = _norm_bound(xf, gain, eps, ref, spec, np.arange(x.shape[1]))
    assert np.all(err <= bound), (err.max(), float((err / bound).max()))
    exact = np.mean(to_bits(y) == oracle.f64_to_bf16_bits(ref))
    log(f"  correctly rounded fraction {exact:.5f}")
    assert exact > 0.99


def test_qk_norm_rope_full_size_wan13b():
    import torch

    w = inputs.WORKLOADS["wan13b_480p"]
    k = inputs.bf16_tensor(w.seed, inputs.T_K, (w.B, w.Lk, w.H, w.d))  # before normalisation
    g = np.random.default_rng(14).uniform(0.5, 1.5, 128).astype(np.float32)
    log("case qk_norm_rope wan13b_480p K")
    y = vx.qk_norm_rope(to_dev(k), rope_of(w), gain=torch.from_numpy(g).cuda(), eps=1e-6)
    torch.cuda.synchronize()
    yb = to_bits(y)
    rows = np.unique(np.r_[0, 1, 51, 52, 1559, 1560, w.Lk - 1, np.random.default_rng(0).integers(0, w.Lk, 300)])
    xf = oracle.bf16_bits_to_f64(k[:, rows])
    ref = oracle.qk_norm_ref(xf, gain=g.astype(np.float64), eps=1e-6, rope=spec_of(w), token_index=rows)
    got = oracle.bf16_bits_to_f64(yb[:, rows])
    assert np.all(np.abs(got - ref) <= _norm_bound(xf, g.astype(np.float64), 1e-6, ref, spec_of(w), rows))


def test_qk_norm_rope_empty():
    import torch

    x = torch.empty((0, 5, 2, 128), dtype=torch.bfloat16, device="cuda")
    assert vx.qk_norm_rope(x).shape == x.shape


# ------------------------------------------------------- attention: small ---

def test_tiny_workload():
    _full_case(inputs.WORKLOADS["tiny"])


def test_tiny_workload_naive_kernel():
    _full_case(inputs.WORKLOADS["tiny"], impl=vx.attn_fwd_naive)


RAGGED = [
    # several tiles with ragged tails in queries and keys, rotated prefix + unrotated suffix
    inputs.custom("ragged_self", B=2, H=3, Lq=1000, Lk=1000, seed=21, grid=(2, 20, 24), kv_valid=("fixed", [1000, 517])),
    # Lq != Lk with rotation (rotated tokens <= min(Lq, Lk))
    inputs.custom("ragged_qk", B=1, H=2, Lq=777, Lk=1001, seed=22, grid=(1, 21, 37)),
    # cross-attention shape, short keys, per-batch lengths incl. clamp above Lk
    inputs.custom("cross_small", B=3, H=4, Lq=700, Lk=512, seed=23, kv_valid=("fixed", [64, 511, 900])),
    # keys fewer than one tile, queries fewer than one wave
    inputs.custom("few", B=1, H=1, Lq=5, Lk=3, seed=24),
    inputs.custom("one", B=2, H=1, Lq=1, Lk=1, seed=25),
    inputs.custom("tile_plus_one", B=1, H=2, Lq=257, Lk=65, seed=26, grid=(1, 5, 13)),
    # dense kernel, batches of very different valid lengths: 60 query tiles a
    # batch, so each XCD's run holds a part of every batch (eighths of 8 and
    # 7 tiles) and the position -> tile map is exercised past its one-batch case
    inputs.custom("mixed_lengths", B=3, H=5, Lq=3000, Lk=2500, seed=27, kv_valid=("fixed", [2500, 70, 1900])),
]


@pytest.mark.parametrize("w", RAGGED, ids=lambda w: w.name)
def test_ragged_and_edge_shapes(w):
    _full_case(w)


def _random_shapes(n=16, seed=2026):
    """Seeded random shapes between the hand-picked ones: batches, heads,
    query and key counts off the tile grid, a rotated prefix (grid no larger
    than either sequence) or none, per-batch valid lengths from 0 to past Lk,
    raw or RMS-normalised q and k."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B, H = int(rng.integers(1, 4)), int(rng.integers(1, 5))
        Lq, Lk = int(rng.integers(1, 1201)), int(rng.integers(1, 1201))
        grid = None
        if rng.random() < 0.6:
            t, h, w = int(rng.integers(1, 4)), int(rng.integers(1, 11)), int(rng.integers(1, 41))
            if t * h * w <= min(Lq, Lk):
                grid = (t, h, w)
        kv = ("fixed", [int(x) for x in rng.integers(0, Lk + 50, B)]) if rng.random() < 0.5 else None
        cases.append(inputs.custom(f"random{i}", B=B, H=H, Lq=Lq, Lk=Lk, seed=100 + i, grid=grid, kv_valid=kv,
                                   rms_norm_qk=bool(rng.random() < 0.5)))
    return cases


@pytest.mark.parametrize("w", _random_shapes(), ids=lambda w: w.name)
def test_random_shapes(w):
    _full_case(w)


@pytest.mark.parametrize("w", RAGGED[:3], ids=lambda w: w.name)
def test_naive_kernel_agrees(w):
    _full_case(w, impl=vx.attn_fwd_naive)


@pytest.mark.parametrize("w", [inputs.WORKLOADS["tiny"], RAGGED[0], RAGGED[5]], ids=lambda w: w.name)
def test_prerotated_keys(w):
    """vidax_rope3d on k, then attention rotating only q: same result as the
    fused rotation of both, against the oracle."""
    import dataclasses

    import torch

    q, k, v, lv = inputs.make_qkv(w)
    log(f"case prerotated keys {w.name}")
    r = rope_of(w)
    kd = to_dev(k)
    krot = vx.rope3d(kd, r)
    o, l = vx.attn_fwd(to_dev(q), krot, to_dev(v), scale=w.scale, kv_valid_len=lengths_dev(lv),
                       rope=dataclasses.replace(r, keys_prerotated=True), return_lse=True)
    torch.cuda.synchronize()
    ro, rl = _oracle_full(w, q, k, v, lv)
    assert_parity(to_bits(o), ro, f"{w.name} prerotated")
    assert_lse(l.cpu().numpy(), rl, f"{w.name} prerotated")


@pytest.mark.parametrize("w", [inputs.WORKLOADS["tiny"], RAGGED[0], RAGGED[5]], ids=lambda w: w.name)
def test_half_split_pairs_prerotated_keys(w):
    """Half-split pairs (channel o_a + j with o_a + j + d_a/2): k rotated by
    vidax_rope3d, q inside the attention kernel (each channel's partner from
    the staged query row), against the oracle with the same convention."""
    import dataclasses

    import torch

    q, k, v, lv = inputs.make_qkv(w)
    log(f"case half-split pairs {w.name}")
    r = dataclasses.replace(rope_of(w), pair_mode=1)
    krot = vx.rope3d(to_dev(k), r)
    o, l = vx.attn_fwd(to_dev(q), krot, to_dev(v), scale=w.scale, kv_valid_len=lengths_dev(lv),
                       rope=dataclasses.replace(r, keys_prerotated=True), return_lse=True)
    torch.cuda.synchronize()
    dec = oracle.bf16_bits_to_f64
    spec = dataclasses.replace(spec_of(w), pair_mode=1)
    ro, rl = oracle.attn_ref(dec(q), dec(k), dec(v), w.scale, kv_valid_len=lv, rope=spec, workers=8)
    assert_parity(to_bits(o), ro, f"{w.name} half split")
    assert_lse(l.cpu().numpy(), rl, f"{w.name} half split")
    # the interleaved result differs (the convention is really applied)
    ri, _ = _oracle_full(w, q, k, v, lv)
    assert np.abs(ri - ro).max() > 1e-2


def test_zero_and_single_valid_keys():
    import torch

    w = inputs.custom("lv_edge", B=4, H=2, Lq=300, Lk=200, seed=27, grid=(1, 10, 20))
    q, k, v, _ = inputs.make_qkv(w)
    lv = [0, 1, -5, 199]
    log("case lv_edge", lv)
    ob, lse = _run(w, q, k, v, lv)
    # no valid key (0 or negative): zero output, -inf lse
    assert np.all(ob[0] == 0) and np.all(ob[2] == 0)
    assert np.all(np.isneginf(lse[0])) and np.all(np.isneginf(lse[2]))
    # one valid key: the output is that key's value row, bit for bit
    assert np.array_equal(ob[1], np.broadcast_to(v[1, :1], ob[1].shape))
    ro, rl = _oracle_full(w, q, k, v, lv)
    assert_parity(ob, ro, "lv_edge")
    assert_lse(lse, rl, "lv_edge")
    del torch


def test_empty_calls_are_noops():
    import torch

    z = torch.zeros((0, 4, 2, 128), dtype=torch.bfloat16, device="cuda")
    assert vx.attn_fwd(z, z, z).shape == z.shape
    q = torch.zeros((1, 0, 2, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((1, 4, 2, 128), dtype=torch.bfloat16, device="cuda")
    assert vx.attn_fwd(q, k, k).shape == q.shape
    # no keys at all: zero output
    q = torch.randn((1, 9, 2, 128), device="cuda").to(torch.bfloat16)
    k = torch.zeros((1, 0, 2, 128), dtype=torch.bfloat16, device="cuda")
    o, l = vx.attn_fwd(q, k, k, return_lse=True)
    torch.cuda.synchronize()
    assert torch.all(o == 0) and torch.all(torch.isneginf(l))


@pytest.mark.parametrize("scale", [0.0, -0.05, 0.7])
def test_scale_values(scale):
    """Zero, negative and large scales.  The kernel rounds the rotated key,
    and the rotated query multiplied by scale * log2(e), to bf16 before the
    products (as documented); with a large scale the logits are large and that
    input rounding dominates, so the reference here is the oracle's attention
    over the oracle's rotated inputs rounded the same way -- the remaining
    difference is the kernel's own arithmetic."""
    import torch

    w = inputs.custom(f"scale{scale}", B=1, H=2, Lq=300, Lk=400, seed=28, grid=(1, 15, 20))
    q, k, v, _ = inputs.make_qkv(w)
    log(f"case scale {scale}")
    res = vx.attn_fwd(to_dev(q), to_dev(k), to_dev(v), scale=scale, rope=rope_of(w), return_lse=True)
    torch.cuda.synchronize()
    ob, lse = to_bits(res[0]), res[1].cpu().numpy()
    dec = oracle.bf16_bits_to_f64
    spec = spec_of(w)
    # the query's multiplier as the kernel forms it (fp32 product)
    c = float(np.float32(np.float32(scale) * np.float32(1.4426950408889634)))
    qrot = oracle.rope3d_ref(dec(q), spec)
    qr = dec(oracle.f64_to_bf16_bits(qrot * c)) / c if c != 0.0 else qrot
    kr = dec(oracle.f64_to_bf16_bits(oracle.rope3d_ref(dec(k), spec)))
    ro, rl = oracle.attn_ref(qr, kr, dec(v), scale)
    assert_parity(ob, ro, f"scale {scale} vs rounded rotated inputs")
    assert_lse(lse, rl, f"scale {scale}")
    # against the exact oracle: same contract where the logits are moderate
    ro2, _ = oracle.attn_ref(dec(q), dec(k), dec(v), scale, rope=spec)
    e = errors(ob, ro2)
    log(f"  vs exact rotation: {e}")
    assert e["rel_rms"] <= 1e-2
    if abs(scale) <= 0.1:
        assert_parity(ob, ro2, f"scale {scale} exact")


def test_peaked_and_rescaling_logits():
    """Scores that grow along the keys force a rescale of the running sum at
    every tile; a large scale makes the softmax nearly one-hot."""
    import torch

    B, L, H, d = 1, 1000, 2, 128
    rng = np.random.default_rng(29)
    qf = np.zeros((B, L, H, d), np.float32)
    qf[..., 0] = 1.0
    qf[..., 1:] = 0.01 * rng.standard_normal((B, L, H, d - 1))
    kf = 0.01 * rng.standard_normal((B, L, H, d)).astype(np.float32)
    kf[..., 0] = 0.1 * np.arange(L)[None, :, None]            # increasing
    kf[:, :, 1, 0] = 0.1 * np.arange(L)[::-1]                  # head 1: decreasing
    vf = rng.standard_normal((B, L, H, d)).astype(np.float32)
    q, k, v = (inputs.f32_to_bf16_bits(a).reshape(a.shape) for a in (qf, kf, vf))
    dec = oracle.bf16_bits_to_f64
    for scale in (1.0, 30.0):
        log(f"case peaked scale={scale}")
        o, l = vx.attn_fwd(to_dev(q), to_dev(k), to_dev(v), scale=scale, return_lse=True)
        torch.cuda.synchronize()
        ro, rl = oracle.attn_ref(dec(q), dec(k), dec(v), scale)
        assert_parity(to_bits(o), ro, f"peaked {scale}")
        assert_lse(l.cpu().numpy(), rl, f"peaked {scale}")


def test_deterministic():
    import torch

    w = RAGGED[0]
    q, k, v, lv = inputs.make_qkv(w)
    qd, kd, vd, ld = to_dev(q), to_dev(k), to_dev(v), lengths_dev(lv)
    log("case determinism")
    outs = []
    for _ in range(3):
        o, l = vx.attn_fwd(qd, kd, vd, scale=w.scale, kv_valid_len=ld, rope=rope_of(w), return_lse=True)
        torch.cuda.synchronize()
        outs.append((to_bits(o), l.cpu().numpy()))
    for o, l in outs[1:]:
        assert np.array_equal(o, outs[0][0]) and np.array_equal(l, outs[0][1])


# ----------------------------------------------------- full-size workloads ---

def _sample_rows(L, rng, n=160):
    fixed = [0, 1, 31, 32, 63, 64, 255, 256, 257, L // 2, L - 257, L - 256, L - 65, L - 64, L - 33, L - 2, L - 1]
    fixed = [r for r in fixed if 0 <= r < L]
    return np.unique(np.r_[fixed, rng.integers(0, L, n)])


def _convex_bounds_ok(ob, v, lv, heads):
    """Every output component lies in [min, max] of the valid value rows (per
    batch, head, channel), up to one bf16 rounding of the output; a batch
    without valid keys has an all-zero output."""
    got = oracle.bf16_bits_to_f64(ob)
    for b in range(ob.shape[0]):
        n = v.shape[1] if lv is None else int(np.clip(lv[b], 0, v.shape[1]))
        if n == 0:
            if np.any(got[b][:, heads] != 0):
                return False
            continue
        vv = oracle.bf16_bits_to_f64(v[b, :n][:, heads])  # [n, Hs, d]
        lo = vv.min(axis=0)
        hi = vv.max(axis=0)
        g = got[b][:, heads]
        slack = 2.0 ** -8 * np.maximum(np.abs(lo), np.abs(hi)) + 1e-30
        if not (np.all(g >= lo - slack) and np.all(g <= hi + slack)):
            return False
    return True


# Short key sequences without rotation at more than four query tiles per CU
# run as one persistent workgroup per CU looping over query tiles; three K/V
# tile buffers keep the last tiles of a head between its query tiles, and a
# query tile with more than three key tiles copies the others as it goes (in
# an order that depends on the tiles kept from the query tile before): empty
# batches (Lv = 0), a ragged last query tile, Lk at the persistent-form limit
# (1024 keys, 16 tiles), batches of 2, 7, 3, 4 and 1 tiles in turn (the 192/193-key
# boundary between copying and not), of 5, 6 and 8 tiles (every tile count
# mod 3; partial and full last tiles), and a case without per-batch lengths
# where no query tile copies.
PERSISTENT = [
    inputs.custom("persist_empty_batch", B=2, H=8, Lq=20000, Lk=300, seed=31, kv_valid=("fixed", [0, 173])),
    inputs.custom("persist_long_keys", B=1, H=16, Lq=17000, Lk=1024, seed=32),
    inputs.custom("persist_alternating", B=5, H=8, Lq=7000, Lk=512, seed=33,
                  kv_valid=("fixed", [100, 400, 192, 193, 1])),
    inputs.custom("persist_tile_counts", B=4, H=8, Lq=9000, Lk=512, seed=35,
                  kv_valid=("fixed", [257, 384, 449, 512])),
    inputs.custom("persist_short_nolen", B=1, H=16, Lq=17000, Lk=150, seed=34),
]


def _random_persistent(n=6, seed=2027):
    """Seeded random shapes that reach the short-key kernel: no rotation,
    Lk <= 1024, ragged Lq, per-batch valid lengths (some 0, some past Lk,
    some not a multiple of the 64-key tile) and more than 4 query tiles per
    CU (B * H * ceil(Lq / 256) > 1024)."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B = int(rng.integers(1, 5))
        H = int(rng.integers(4, 17))
        Lk = int(rng.choice([1, 63, 64, 65, 300, 512, 777, 1024]))
        need = 1024 // (B * H) + 2  # query tiles per (b, h) beyond the threshold
        Lq = int(rng.integers(need * 256 - 255, need * 256 + 3000))
        lens = [int(x) for x in rng.integers(-3, Lk + 40, B)]
        if i == 0:
            lens[0] = 0
        cases.append(inputs.custom(f"prand{i}", B=B, H=H, Lq=Lq, Lk=Lk, seed=300 + i, kv_valid=("fixed", lens)))
    return cases


def _random_persistent_many_batches(n=6, seed=2031):
    """More seeded random short-key shapes: 3 to 6 batches with lengths drawn
    from [1, Lk], Lk up to 1024, so consecutive batches have different tile
    counts (1 to 16) and the kept K/V buffers meet head changes between them
    often; ragged Lq."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B = int(rng.integers(3, 7))
        H = int(rng.integers(2, 9))
        Lk = int(rng.choice([300, 640, 1000, 1024]))
        need = 1024 // (B * H) + 2
        Lq = int(rng.integers(need * 256 - 255, need * 256 + 2000))
        lens = [int(x) for x in rng.integers(1, Lk + 1, B)]
        cases.append(inputs.custom(f"prand_many{i}", B=B, H=H, Lq=Lq, Lk=Lk, seed=320 + i,
                                   kv_valid=("fixed", lens)))
    return cases


@pytest.mark.parametrize("w", PERSISTENT + _random_persistent() + _random_persistent_many_batches(),
                         ids=lambda w: w.name)
def test_persistent_short_keys_sampled(w):
    import torch

    q, k, v, lv = inputs.make_qkv(w)
    log(f"case persistent form {w.name}")
    o, l = vx.attn_fwd(to_dev(q), to_dev(k), to_dev(v), scale=w.scale, kv_valid_len=lengths_dev(lv), return_lse=True)
    torch.cuda.synchronize()
    ob, lse = to_bits(o), l.cpu().numpy()
    rows = _sample_rows(w.Lq, np.random.default_rng(w.seed + 100))
    dec = oracle.bf16_bits_to_f64
    ro, rl = oracle.attn_ref_rows(dec(q), dec(k), dec(v), w.scale, rows, kv_valid_len=lv, workers=8)
    assert_parity(ob[:, rows], ro, w.name)
    assert_lse(lse[:, :, rows], rl, w.name)
    assert _convex_bounds_ok(ob, v, lv, list(range(w.H)))


def test_batch_at_the_2gib_limit():
    """One batch of q, k, v and o just below 2 GiB, the largest the forward
    accepts (max(Lq, Lk) * H * d * 2 <= 2^31 - 1 - 4096): B=1, H=64,
    L=131071; element (n, h) sits at byte (n * 64 + h) * 256, so the last rows
    of the last head are at the top of the 32-bit offset range.  The dense
    kernel (Lq = Lk, no rotation) and the short-key kernel (the first 64
    keys, 50 valid).  Inputs are seeded N(0, 1) drawn on the GPU (torch's
    generator) and copied back for the heads the oracle checks: sampled rows,
    the last ones included, of the first and last head."""
    import torch

    B, H, L = 1, 64, 131071
    assert L * H * 128 * 2 <= 2 ** 31 - 1 - 4096 < (L + 1) * H * 128 * 2
    g = torch.Generator(device="cuda")
    g.manual_seed(41)
    mk = lambda n: torch.randn((B, n, H, 128), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    q, k, v = mk(L), mk(L), mk(L)
    scale = float(np.float32(1 / np.sqrt(128)))
    hs = [0, H - 1]
    rows = np.array([0, 1, 255, 256, 65535, 130815, 130816, 131040, 131069, 131070])
    bits = lambda t: t[:, :, hs].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    dec = oracle.bf16_bits_to_f64
    qh = dec(bits(q))
    for name, lk, lens in (("dense", L, None), ("short keys", 64, [50])):
        log(f"case 2 GiB limit, {name}: B{B} H{H} Lq{L} Lk{lk} lens={lens}")
        kk, vv = (k, v) if lk == L else (k[:, :lk].contiguous(), v[:, :lk].contiguous())
        o, lse = vx.attn_fwd(q, kk, vv, scale=scale, kv_valid_len=lengths_dev(lens), return_lse=True)
        torch.cuda.synchronize()
        ob = bits(o)[:, rows]
        lb = lse[:, hs].cpu().numpy()[:, :, rows]
        ro, rl = oracle.attn_ref_rows(qh, dec(bits(kk)), dec(bits(vv)), scale, rows, kv_valid_len=lens, workers=8)
        assert_parity(ob, ro, f"2 GiB limit, {name}")
        assert_lse(lb, rl, f"2 GiB limit, {name}")
        del o, lse, kk, vv
    del q, k, v
    torch.cuda.empty_cache()


def test_full_size_prerotated_wan13b_sampled():
    import dataclasses

    import torch

    w = inputs.WORKLOADS["wan13b_480p"]
    q, k, v, lv = inputs.make_qkv(w)
    log("case full-size wan13b_480p, keys rotated by vidax_rope3d")
    r = rope_of(w)
    krot = vx.rope3d(to_dev(k), r)
    o = vx.attn_fwd(to_dev(q), krot, to_dev(v), scale=w.scale, rope=dataclasses.replace(r, keys_prerotated=True))
    torch.cuda.synchronize()
    ob = to_bits(o)
    rows = _sample_rows(w.Lq, np.random.default_rng(w.seed + 100))
    dec = oracle.bf16_bits_to_f64
    ro, _ = oracle.attn_ref_rows(dec(q), dec(k), dec(v), w.scale, rows, rope=spec_of(w), workers=8)
    assert_parity(ob[:, rows], ro, "wan13b_480p prerotated")


@pytest.mark.parametrize("name,heads", [
    ("wan13b_480p", None),
    ("cross_text", None),
    ("wan14b_720p", [0, 13, 26, 39]),
    ("hunyuan_joint", [0, 11, 23]),
])
def test_full_size_workload_sampled(name, heads):
    import torch

    w = inputs.WORKLOADS[name]
    log(f"case full-size {name}: generating inputs")
    q, k, v, lv = inputs.make_qkv(w)
    log(f"case full-size {name}: GPU call")
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    o, l = vx.attn_fwd(qd, kd, vd, scale=w.scale, kv_valid_len=lengths_dev(lv), rope=rope_of(w), return_lse=True)
    torch.cuda.synchronize()
    ob = to_bits(o)
    lse = l.cpu().numpy()
    del qd, kd, vd, o, l
    torch.cuda.empty_cache()
    hs = list(range(w.H)) if heads is None else heads
    # every head, every row: finite and inside the convex hull of the valid value rows
    log(f"case full-size {name}: finiteness and convex hull on all {w.H} heads")
    for h in range(w.H):
        assert np.all(np.isfinite(oracle.bf16_bits_to_f64(ob[:, :, h]))), h
        assert _convex_bounds_ok(ob, v, lv, [h]), h
    rows = _sample_rows(w.Lq, np.random.default_rng(w.seed))
    log(f"case full-size {name}: oracle on {len(rows)} rows x {len(hs)} heads")
    dec = oracle.bf16_bits_to_f64
    ro, rl = oracle.attn_ref_rows(dec(q[:, :, hs]), dec(k[:, :, hs]), dec(v[:, :, hs]), w.scale, rows,
                                  kv_valid_len=lv, rope=spec_of(w), workers=8)
    assert_parity(ob[:, rows][:, :, hs], ro, name)
    assert_lse(lse[:, hs][:, :, rows], rl, name)
    e = errors(ob[:, rows][:, :, hs], ro)
    log(f"  {name}: {e}")
