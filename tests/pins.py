"""Checks that pin the oracle to facts other than itself.

Each check takes the functions under test as arguments so that the same checks
run against the oracle (tests/test_oracle_pins.py) and against deliberately
broken copies of it (tests/test_oracle_mutations.py, which shows that each
plausible mistake is caught).  Every check raises AssertionError on failure.

Sources of truth used here:
  * closed forms of a plane rotation (unit vectors, the exact frequency
    theta**(-1/2) = 0.01 of the middle time-pair for theta = 1e4, d_t = 44);
  * identities the rotary embedding must satisfy (norm preservation,
    relative-position invariance, identity at the origin, untouched tokens
    beyond the grid);
  * the pure-Python brute force in tests/brute.py (complex-number rotation,
    math.fsum softmax);
  * torch.nn.functional.scaled_dot_product_attention in float64 on the CPU as a
    library cross-check of the unmasked / prefix-masked attention;
  * invariants of softmax attention (single key, constant V, permutations,
    shifts of all keys, Q = 0, one-hot limit, linearity in V, lse consistency);
  * for the query/key prologue (RMS normalisation + gain + rotation): closed
    forms of a constant vector (with eps dominant and negligible), unit RMS
    of every (token, head) whatever the heads' own scales, invariance to a
    positive scale, the gain as a per-channel factor, commutation of the
    normalisation with the rotation, and the pure-Python brute force;
  * for the attention gradient: central finite differences of the (pinned)
    forward oracle, torch autograd in float64, and identities of the softmax
    gradient (sum of dK over keys is zero, sum of dV over keys is the sum of
    dO, linearity in dO, zero gradient of masked keys and of empty batches),
    plus the adjoint identity of the rotation's transpose.
"""

from __future__ import annotations

import math

import numpy as np

from tests import brute


def _rng(seed):
    return np.random.default_rng(seed)


# ----------------------------------------------------------------- rotary ---

def check_rope_unit_vectors(rope_fn, spec_cls):
    """A unit vector in the first channel of an axis block, at a token whose
    coordinate on that axis is p, becomes (cos p, sin p) on that pair (j = 0,
    frequency 1); the other axes' blocks are untouched."""
    grid = (3, 4, 5)
    dims = (4, 4, 4)
    for mode in (0, 1):
        spec = spec_cls(grid=grid, dims=dims, theta=10000.0, pair_mode=mode)
        for axis, (t, h, w) in enumerate([(2, 0, 0), (0, 3, 0), (0, 0, 4)]):
            n = (t * grid[1] + h) * grid[2] + w
            p = (t, h, w)[axis]
            off = sum(dims[:axis])
            partner = off + 1 if mode == 0 else off + dims[axis] // 2
            x = np.zeros((1, n + 1, 1, 12))
            x[0, n, 0, off] = 1.0
            y = rope_fn(x, spec)[0, n, 0]
            exp = np.zeros(12)
            exp[off] = math.cos(p)
            exp[partner] = math.sin(p)
            assert np.allclose(y, exp, atol=1e-15), (mode, axis, y, exp)


def check_rope_known_frequency(rope_fn, spec_cls):
    """theta = 1e4, d_t = 44: pair j = 11 of the time block has frequency
    1e4 ** (-22/44) = 0.01, so a unit vector there turns by 0.01 * t."""
    spec = spec_cls(grid=(21, 2, 3), dims=(44, 42, 42), theta=10000.0, pair_mode=0)
    t = 17
    n = t * 2 * 3
    x = np.zeros((1, n + 1, 1, 128))
    x[0, n, 0, 22] = 1.0
    y = rope_fn(x, spec)[0, n, 0]
    assert abs(y[22] - math.cos(0.17)) < 1e-15 and abs(y[23] - math.sin(0.17)) < 1e-15, y[20:26]
    assert np.count_nonzero(np.abs(y) > 1e-15) == 2


def check_rope_identities(rope_fn, spec_cls):
    rng = _rng(7)
    spec = spec_cls(grid=(3, 4, 5), dims=(44, 42, 42), theta=10000.0, pair_mode=0)
    L = 70  # 60 grid tokens + 10 appended tokens
    x = rng.standard_normal((2, L, 3, 128))
    y = rope_fn(x, spec)
    # origin token is unchanged, tokens beyond the grid are unchanged
    assert np.array_equal(y[:, 0], x[:, 0])
    assert np.array_equal(y[:, 60:], x[:, 60:])
    # every channel pair keeps its length
    for mode in (0, 1):
        s = spec_cls(grid=spec.grid, dims=spec.dims, theta=spec.theta, pair_mode=mode)
        yy = rope_fn(x, s)
        off = 0
        for da in s.dims:
            for j in range(da // 2):
                c0, c1 = (off + 2 * j, off + 2 * j + 1) if mode == 0 else (off + j, off + da // 2 + j)
                n0 = x[..., c0] ** 2 + x[..., c1] ** 2
                n1 = yy[..., c0] ** 2 + yy[..., c1] ** 2
                assert np.allclose(n0, n1, rtol=1e-13, atol=1e-13)
            off += da


def check_rope_relative(rope_fn, spec_cls):
    """<R(p) q, R(p') k> depends only on p - p': shifting both tokens by the
    same step along any one axis leaves the inner product unchanged."""
    rng = _rng(11)
    grid = (4, 5, 6)
    T, Hp, Wp = grid
    for mode in (0, 1):
        spec = spec_cls(grid=grid, dims=(44, 42, 42), theta=10000.0, pair_mode=mode)
        L = T * Hp * Wp
        q = rng.standard_normal(128)
        k = rng.standard_normal(128)
        x = np.zeros((1, L, 2, 128))
        x[0, :, 0] = q
        x[0, :, 1] = k
        y = rope_fn(x, spec)

        def tok(t, h, w):
            return (t * Hp + h) * Wp + w

        for (a, b), shift in [(((0, 1, 2), (2, 3, 0)), (1, 0, 0)),
                              (((1, 0, 1), (0, 3, 2)), (0, 1, 0)),
                              (((2, 2, 0), (1, 1, 3)), (0, 0, 2))]:
            a2 = tuple(a[i] + shift[i] for i in range(3))
            b2 = tuple(b[i] + shift[i] for i in range(3))
            s1 = y[0, tok(*a), 0] @ y[0, tok(*b), 1]
            s2 = y[0, tok(*a2), 0] @ y[0, tok(*b2), 1]
            assert abs(s1 - s2) < 1e-11, (mode, a, b, shift, s1, s2)
        # and it does change with the relative offset (the rotation is not trivial)
        s_same = y[0, tok(1, 1, 1), 0] @ y[0, tok(1, 1, 1), 1]
        s_off = y[0, tok(1, 1, 1), 0] @ y[0, tok(1, 1, 2), 1]
        assert abs(s_same - q @ k) < 1e-11
        assert abs(s_off - q @ k) > 1e-6


def check_rope_brute(rope_fn, spec_cls):
    rng = _rng(3)
    for mode in (0, 1):
        for grid, dims in [((2, 3, 2), (4, 4, 4)), ((1, 1, 7), (2, 4, 6)), ((3, 2, 2), (6, 2, 4))]:
            spec = spec_cls(grid=grid, dims=dims, theta=100.0, pair_mode=mode)
            L = grid[0] * grid[1] * grid[2] + 3
            d = sum(dims)
            x = rng.standard_normal((1, L, 2, d))
            y = rope_fn(x, spec)
            for n in range(L):
                for h in range(2):
                    yb = brute.rope_row(list(x[0, n, h]), n, grid, dims, 100.0, mode)
                    assert np.allclose(y[0, n, h], yb, rtol=1e-13, atol=1e-13), (mode, grid, n)


# -------------------------------------------------------------- attention ---

def _tiny_case(rng, B=2, Lq=7, Lk=9, H=2, d=12):
    q = rng.standard_normal((B, Lq, H, d))
    k = rng.standard_normal((B, Lk, H, d))
    v = rng.standard_normal((B, Lk, H, d))
    return q, k, v


def check_attn_brute(attn_fn, spec_cls):
    rng = _rng(5)
    for with_rope in (False, True):
        for lv in (None, [9, 4], [1, 0], [12, 3]):
            q, k, v = _tiny_case(rng)
            spec = spec_cls(grid=(2, 2, 2), dims=(4, 4, 4), theta=100.0, pair_mode=0) if with_rope else None
            o, lse = attn_fn(q, k, v, 0.37, kv_valid_len=lv, rope=spec)
            rope = (spec.grid, spec.dims, spec.theta, spec.pair_mode) if with_rope else None
            ob, lb = brute.attention(q.tolist(), k.tolist(), v.tolist(), 0.37, kv_valid_len=lv, rope=rope)
            ob = np.array(ob)
            lb = np.array(lb)
            assert np.allclose(o, ob, rtol=1e-12, atol=1e-12), (with_rope, lv)
            fin = np.isfinite(lb)
            assert np.array_equal(fin, np.isfinite(lse))
            assert np.allclose(lse[fin], lb[fin], rtol=1e-12, atol=1e-12)


def check_attn_torch(attn_fn):
    import torch

    rng = _rng(9)
    B, L, H, d = 2, 300, 3, 128
    q, k, v = _tiny_case(rng, B=B, Lq=L, Lk=L, H=H, d=d)
    scale = 1 / math.sqrt(d)
    o, lse = attn_fn(q, k, v, scale)
    tq, tk, tv = (torch.from_numpy(a).permute(0, 2, 1, 3) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale).permute(0, 2, 1, 3).numpy()
    assert np.allclose(o, ref, rtol=1e-11, atol=1e-12)
    s = torch.einsum("bhqd,bhkd->bhqk", tq, tk) * scale
    assert np.allclose(lse, torch.logsumexp(s, dim=-1).numpy(), rtol=1e-12, atol=1e-12)
    # prefix mask == attention over the truncated key/value sequence
    lv = [173, 300]
    o2, _ = attn_fn(q, k, v, scale, kv_valid_len=lv)
    for b in range(B):
        r = torch.nn.functional.scaled_dot_product_attention(
            tq[b:b + 1], tk[b:b + 1, :, :lv[b]], tv[b:b + 1, :, :lv[b]], scale=scale
        ).permute(0, 2, 1, 3).numpy()
        assert np.allclose(o2[b:b + 1], r, rtol=1e-11, atol=1e-12)


def check_attn_invariants(attn_fn, spec_cls):
    rng = _rng(13)
    B, Lq, Lk, H, d = 2, 17, 23, 2, 16
    q, k, v = _tiny_case(rng, B, Lq, Lk, H, d)
    sc = 0.29
    o, lse = attn_fn(q, k, v, sc)
    # single valid key returns that value row exactly
    o1, l1 = attn_fn(q, k, v, sc, kv_valid_len=[1, 1])
    assert np.array_equal(o1, np.broadcast_to(v[:, :1], o1.shape))
    s0 = sc * np.einsum("bqhd,bhd->bhq", q, k[:, 0])
    assert np.allclose(l1, s0, rtol=1e-13, atol=1e-13)
    # no valid key: zero output and -inf lse; lengths beyond Lk are clamped
    oz, lz = attn_fn(q, k, v, sc, kv_valid_len=[0, Lk + 5])
    assert np.all(oz[0] == 0) and np.all(np.isneginf(lz[0]))
    assert np.allclose(oz[1], o[1], rtol=1e-14, atol=1e-14)
    # constant V returns the constant
    vc = np.broadcast_to(rng.standard_normal((1, 1, H, d)), v.shape).copy()
    oc, _ = attn_fn(q, k, vc, sc)
    assert np.allclose(oc, np.broadcast_to(vc[:, :1], oc.shape), rtol=1e-13, atol=1e-13)
    # keys and values permuted together: same output
    perm = rng.permutation(Lk)
    op, lp = attn_fn(q, k[:, perm], v[:, perm], sc)
    assert np.allclose(op, o, rtol=1e-12, atol=1e-13) and np.allclose(lp, lse, rtol=1e-13)
    # queries permuted: output rows permuted
    qp = rng.permutation(Lq)
    oq, _ = attn_fn(q[:, qp], k, v, sc)
    assert np.allclose(oq, o[:, qp], rtol=1e-13, atol=1e-14)
    # the same vector added to every key: unchanged output (max subtraction, softmax shift)
    u = rng.standard_normal((B, 1, H, d))
    ou, _ = attn_fn(q, k + u, v, sc)
    assert np.allclose(ou, o, rtol=1e-10, atol=1e-12)
    # Q = 0 (or scale = 0) gives the mean of the valid value rows
    for lv in (None, [5, 11]):
        oq0, lq0 = attn_fn(np.zeros_like(q), k, v, sc, kv_valid_len=lv)
        os0, _ = attn_fn(q, k, v, 0.0, kv_valid_len=lv)
        for b in range(B):
            n = Lk if lv is None else lv[b]
            mean = v[b, :n].mean(axis=0)
            assert np.allclose(oq0[b], np.broadcast_to(mean, oq0[b].shape), rtol=1e-13, atol=1e-14)
            assert np.allclose(os0[b], np.broadcast_to(mean, os0[b].shape), rtol=1e-13, atol=1e-14)
            assert np.allclose(lq0[b], math.log(n), rtol=1e-14)
    # one-hot limit: with a large scale the output is the value row of the argmax
    big = 1e4
    ob, _ = attn_fn(q, k, v, big)
    s = np.einsum("bqhd,bkhd->bhqk", q, k)
    am = s.argmax(axis=-1)
    for b in range(B):
        for h in range(H):
            assert np.allclose(ob[b, :, h], v[b, am[b, h], h], rtol=1e-9, atol=1e-9)
    # linear in V
    v2 = rng.standard_normal(v.shape)
    ol, _ = attn_fn(q, k, 2.0 * v - 3.0 * v2, sc)
    o2, _ = attn_fn(q, k, v2, sc)
    assert np.allclose(ol, 2.0 * o - 3.0 * o2, rtol=1e-12, atol=1e-12)
    # weights implied by lse sum to one: sum_j exp(s_ij - lse_i) == 1
    w = np.exp(sc * s - lse[..., None])
    assert np.allclose(w.sum(-1), 1.0, rtol=1e-13)
    # and with rotary embedding, the output equals plain attention over rotated inputs
    spec = spec_cls(grid=(2, 3, 3), dims=(6, 6, 4), theta=50.0, pair_mode=0)
    orr, _ = attn_fn(q, k, v, sc, rope=spec)
    assert not np.allclose(orr, o)


ALL_ROPE_CHECKS = [check_rope_unit_vectors, check_rope_known_frequency, check_rope_identities,
                   check_rope_relative, check_rope_brute]


# ------------------------------------------------------ query/key prologue ---

def check_norm_constant(norm_fn, spec_cls):
    """x = c * 1 (all channels equal) becomes c / sqrt(c^2 + eps) in every
    channel: eps negligible for c = +-3, dominant for c = 1e-5."""
    for c, eps in [(3.0, 1e-6), (-3.0, 1e-6), (1e-5, 1e-6), (2.0, 0.0)]:
        x = np.full((1, 2, 3, 8), c)
        y = norm_fn(x, eps=eps)
        assert np.allclose(y, c / math.sqrt(c * c + eps), rtol=1e-14, atol=0), (c, eps)


def check_norm_unit_rms(norm_fn, spec_cls):
    """With eps = 0 and unit gain every (token, head) vector leaves with mean
    square 1, even when the heads (and tokens) carry very different scales."""
    rng = _rng(41)
    x = rng.standard_normal((2, 5, 4, 16)) * np.array([1e-3, 1.0, 7.0, 1e3])[None, None, :, None]
    x = x * np.linspace(0.5, 4.0, 5)[None, :, None, None]
    y = norm_fn(x, eps=0.0)
    assert np.allclose(np.mean(y * y, axis=-1), 1.0, rtol=1e-13)
    # direction kept: y is a positive multiple of x in each (token, head)
    cos = np.sum(x * y, axis=-1) / (np.linalg.norm(x, axis=-1) * np.linalg.norm(y, axis=-1))
    assert np.allclose(cos, 1.0, rtol=1e-13)


def check_norm_scale_invariance(norm_fn, spec_cls):
    """eps = 0: f(a x) = f(x) for a > 0 and f(-x) = -f(x)."""
    rng = _rng(42)
    x = rng.standard_normal((1, 6, 2, 12))
    y = norm_fn(x, eps=0.0)
    assert np.allclose(norm_fn(37.5 * x, eps=0.0), y, rtol=1e-13, atol=1e-14)
    assert np.allclose(norm_fn(-x, eps=0.0), -y, rtol=1e-13, atol=1e-14)


def check_norm_gain(norm_fn, spec_cls):
    """The gain multiplies channel c of every head by g[c]; a one-hot gain
    keeps one channel only."""
    rng = _rng(43)
    x = rng.standard_normal((2, 3, 2, 12))
    g = rng.uniform(0.5, 2.0, 12)
    base = norm_fn(x, eps=1e-6)
    assert np.allclose(norm_fn(x, gain=g, eps=1e-6), base * g, rtol=1e-14, atol=1e-15)
    oh = np.zeros(12)
    oh[5] = 2.0
    y = norm_fn(x, gain=oh, eps=1e-6)
    assert np.all(y[..., np.arange(12) != 5] == 0.0)
    assert np.allclose(y[..., 5], 2.0 * base[..., 5], rtol=1e-14)


def check_norm_rope_commute(norm_fn, spec_cls):
    """With unit gain the normalisation commutes with the rotation, which keeps
    every pair's norm: normalising x rotated by the brute-force rotation equals
    normalise-then-rotate."""
    rng = _rng(44)
    grid, dims, theta = (2, 2, 3), (4, 4, 4), 100.0
    spec = spec_cls(grid=grid, dims=dims, theta=theta, pair_mode=0)
    x = rng.standard_normal((1, 14, 2, 12))  # 12 rotated tokens, 2 beyond the grid
    xr = np.array([[[brute.rope_row(list(x[0, n, h]), n, grid, dims, theta, 0) for h in range(2)] for n in range(14)]])
    assert not np.allclose(xr, x)
    assert np.allclose(norm_fn(xr, eps=1e-6), norm_fn(x, eps=1e-6, rope=spec), rtol=1e-12, atol=1e-13)


def check_norm_brute(norm_fn, spec_cls):
    """Element-wise agreement with the pure-Python brute force (fsum of
    squares, complex rotation), with and without gain and rotation."""
    rng = _rng(45)
    B, L, H, d = 2, 9, 2, 12
    x = rng.standard_normal((B, L, H, d)) * 3.0
    g = rng.uniform(0.5, 1.5, d)
    for gain, rope in [(None, None), (g, None), (g, ((2, 2, 2), (4, 4, 4), 30.0, 0)), (None, ((1, 3, 2), (2, 4, 6), 7.0, 1))]:
        spec = None if rope is None else spec_cls(grid=rope[0], dims=rope[1], theta=rope[2], pair_mode=rope[3])
        y = norm_fn(x, gain=gain, eps=1e-3, rope=spec)
        for b in range(B):
            for n in range(L):
                for h in range(H):
                    want = brute.qk_norm_row(list(x[b, n, h]), None if gain is None else list(gain), 1e-3, n, rope)
                    assert np.allclose(y[b, n, h], want, rtol=1e-12, atol=1e-13), (b, n, h)


ALL_NORM_CHECKS = [check_norm_constant, check_norm_unit_rms, check_norm_scale_invariance, check_norm_gain,
                   check_norm_rope_commute, check_norm_brute]


# ------------------------------------------------------ attention gradient ---

def _bwd_case(rng, B=2, Lq=5, Lk=6, H=2, d=8):
    q = rng.standard_normal((B, Lq, H, d))
    k = rng.standard_normal((B, Lk, H, d))
    v = rng.standard_normal((B, Lk, H, d))
    do = rng.standard_normal((B, Lq, H, d))
    return q, k, v, do


def check_bwd_finite_diff(bwd_fn, fwd_fn):
    """Central differences of L = sum(dO * attn(q, k, v)) match every element
    of dq, dk, dv, with a masked key prefix in one batch."""
    rng = _rng(51)
    q, k, v, do = _bwd_case(rng)
    sc, lv = 0.6, np.array([6, 4])
    dq, dk, dv = bwd_fn(q, k, v, do, sc, kv_valid_len=lv)

    def loss(q_, k_, v_):
        return float(np.sum(do * fwd_fn(q_, k_, v_, sc, kv_valid_len=lv)[0]))

    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = {"q": (xp, k, v), "k": (q, xp, v), "v": (q, k, xp)}[name]
            args_m = {"q": (xm, k, v), "k": (q, xm, v), "v": (q, k, xm)}[name]
            num[idx] = (loss(*args_p) - loss(*args_m)) / (2 * h)
        assert np.allclose(g, num, rtol=1e-6, atol=1e-7), (name, np.abs(g - num).max())


def check_bwd_torch(bwd_fn, fwd_fn):
    """torch autograd through float64 SDPA (prefix mask as an additive mask)."""
    import torch

    rng = _rng(52)
    q, k, v, do = _bwd_case(rng, B=2, Lq=7, Lk=9, H=3, d=16)
    sc, lv = 0.3, np.array([9, 5])
    dq, dk, dv = bwd_fn(q, k, v, do, sc, kv_valid_len=lv)
    tq, tk, tv = (torch.tensor(x.transpose(0, 2, 1, 3), requires_grad=True) for x in (q, k, v))
    mask = torch.zeros((2, 1, 7, 9), dtype=torch.float64)
    mask[1, :, :, 5:] = -math.inf
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=sc)
    out.backward(torch.tensor(do.transpose(0, 2, 1, 3)))
    for g, t in ((dq, tq), (dk, tk), (dv, tv)):
        assert np.allclose(g, t.grad.numpy().transpose(0, 2, 1, 3), rtol=1e-10, atol=1e-12)


def check_bwd_identities(bwd_fn, fwd_fn):
    rng = _rng(53)
    q, k, v, do = _bwd_case(rng, B=3, Lq=6, Lk=8, H=2, d=8)
    sc, lv = 0.8, np.array([8, 3, 0])
    dq, dk, dv = bwd_fn(q, k, v, do, sc, kv_valid_len=lv)
    # shifting every key by one vector leaves the output unchanged: sum_j dK_j = 0
    assert np.allclose(dk.sum(axis=1), 0.0, atol=1e-12)
    # softmax weights sum to one: sum_j dV_j = sum_i dO_i (batches with keys)
    for b in range(2):
        assert np.allclose(dv[b].sum(axis=0), do[b].sum(axis=0), rtol=1e-12, atol=1e-12)
    # masked keys and empty batches get exactly zero gradient
    assert np.all(dk[1, 3:] == 0) and np.all(dv[1, 3:] == 0)
    assert np.all(dq[2] == 0) and np.all(dk[2] == 0) and np.all(dv[2] == 0)
    # linear in dO
    do2 = rng.standard_normal(do.shape)
    g1 = bwd_fn(q, k, v, 2.0 * do - 0.5 * do2, sc, kv_valid_len=lv)
    g2 = bwd_fn(q, k, v, do2, sc, kv_valid_len=lv)
    for a, b_, c in zip(g1, (dq, dk, dv), g2):
        assert np.allclose(a, 2.0 * b_ - 0.5 * c, rtol=1e-11, atol=1e-12)


def check_bwd_saved_output(bwd_fn, fwd_fn):
    """D formed from a saved (perturbed) output O + E: with e_i = <dO_i, E_i>,
    dS moves by -P_ij e_i, so dv is unchanged, dq moves by
    -scale e_i sum_j P_ij k_j (the forward with values k), and the key sum of
    dk moves by -scale sum_i e_i q_i (each row of P sums to one)."""
    rng = _rng(55)
    q, k, v, do = _bwd_case(rng, B=2, Lq=6, Lk=7, H=2, d=8)
    sc, lv = 0.7, np.array([7, 4])
    o, _ = fwd_fn(q, k, v, sc, kv_valid_len=lv)
    g0 = bwd_fn(q, k, v, do, sc, kv_valid_len=lv)
    g1 = bwd_fn(q, k, v, do, sc, kv_valid_len=lv, o_saved=o)
    for a, b_ in zip(g0, g1):
        assert np.allclose(a, b_, rtol=1e-12, atol=1e-13)
    err = 1e-2 * rng.standard_normal(o.shape)
    dq, dk, dv = bwd_fn(q, k, v, do, sc, kv_valid_len=lv, o_saved=o + err)
    e = np.sum(do * err, axis=-1, keepdims=True)  # [B, Lq, H, 1]
    pk, _ = fwd_fn(q, k, k, sc, kv_valid_len=lv)
    assert np.allclose(dv, g0[2], rtol=1e-13, atol=1e-14)
    assert np.allclose(dq - g0[0], -sc * e * pk, rtol=1e-9, atol=1e-12)
    assert np.allclose((dk - g0[1]).sum(axis=1), -sc * (e * q).sum(axis=1), rtol=1e-9, atol=1e-12)
    assert not np.allclose(dq, g0[0], rtol=1e-6, atol=1e-8)


def check_rope_transpose(transpose_fn, rope_fn, spec_cls):
    """<R x, y> = <x, R^T y> for every token and head; R^T R x = x."""
    rng = _rng(54)
    for mode in (0, 1):
        spec = spec_cls(grid=(2, 3, 2), dims=(4, 4, 4), theta=30.0, pair_mode=mode)
        x = rng.standard_normal((2, 14, 2, 12))
        y = rng.standard_normal((2, 14, 2, 12))
        lhs = np.sum(rope_fn(x, spec) * y, axis=-1)
        rhs = np.sum(x * transpose_fn(y, spec), axis=-1)
        assert np.allclose(lhs, rhs, rtol=1e-12, atol=1e-12)
        assert np.allclose(transpose_fn(rope_fn(x, spec), spec), x, rtol=1e-12, atol=1e-12)
        assert not np.allclose(transpose_fn(y, spec), rope_fn(y, spec))


ALL_BWD_CHECKS = [check_bwd_finite_diff, check_bwd_torch, check_bwd_identities, check_bwd_saved_output]


# ------------------------------------------------ neighbourhood attention ---

def _na_case(rng, grid, H=2, d=6, B=1):
    L = grid[0] * grid[1] * grid[2]
    return tuple(rng.standard_normal((B, L, H, d)) for _ in range(3))


def check_na_brute(na_fn, attn_fn):
    """Every row against the all-pairs brute force, both border readings,
    asymmetric grids and windows (axis order and radius matter)."""
    from tests import brute

    rng = _rng(61)
    for grid, window in (((3, 4, 5), (3, 3, 3)), ((2, 5, 6), (1, 3, 5)), ((4, 3, 7), (3, 1, 5))):
        q, k, v = _na_case(rng, grid)
        for border in ("clip", "shift"):
            o, lse = na_fn(q, k, v, 0.7, grid, window, border)
            bo, bl = brute.na3d(q.tolist(), k.tolist(), v.tolist(), 0.7, grid, window, border)
            assert np.allclose(o, np.array(bo), rtol=1e-11, atol=1e-12), (grid, window, border)
            assert np.allclose(lse, np.array(bl), rtol=1e-11, atol=1e-12), (grid, window, border)


def check_na_full_window(na_fn, attn_fn):
    """A window covering the whole grid is full attention (both readings)."""
    rng = _rng(62)
    grid = (2, 3, 4)
    q, k, v = _na_case(rng, grid, H=3, d=8, B=2)
    ref, rl = attn_fn(q, k, v, 0.5)
    for border, window in (("clip", (3, 5, 7)), ("shift", (3, 3, 5)), ("clip", (5, 9, 11))):
        o, lse = na_fn(q, k, v, 0.5, grid, window, border)
        assert np.allclose(o, ref, rtol=1e-12, atol=1e-13), (border, window)
        assert np.allclose(lse, rl, rtol=1e-12, atol=1e-13), (border, window)


def check_na_single_key(na_fn, attn_fn):
    """A 1 x 1 x 1 window: each query sees only its own token: o = v, lse = s."""
    rng = _rng(63)
    grid = (2, 3, 5)
    q, k, v = _na_case(rng, grid)
    for border in ("clip", "shift"):
        o, lse = na_fn(q, k, v, 0.3, grid, (1, 1, 1), border)
        assert np.allclose(o, v, rtol=1e-13, atol=1e-14)
        assert np.allclose(lse, 0.3 * np.einsum("blhd,blhd->bhl", q, k), rtol=1e-12, atol=1e-13)


def check_na_interior_agree(na_fn, attn_fn):
    """Queries whose centred window lies inside the grid see the same keys in
    both readings; near the border they differ."""
    rng = _rng(64)
    grid, window = (5, 6, 7), (3, 3, 5)
    q, k, v = _na_case(rng, grid)
    oc, _ = na_fn(q, k, v, 0.6, grid, window, "clip")
    os_, _ = na_fn(q, k, v, 0.6, grid, window, "shift")
    t, h, w = np.meshgrid(np.arange(5), np.arange(6), np.arange(7), indexing="ij")
    inner = ((t >= 1) & (t <= 3) & (h >= 1) & (h <= 4) & (w >= 2) & (w <= 4)).ravel()
    assert np.allclose(oc[:, inner], os_[:, inner], rtol=1e-13, atol=1e-14)
    assert not np.allclose(oc[:, ~inner], os_[:, ~inner])


ALL_NA_CHECKS = [check_na_brute, check_na_full_window, check_na_single_key, check_na_interior_agree]


# ------------------------------------------------------ Q/K/V projection ---

def _qkv_case(rng, B=1, L=6, H=2, d=12, C=10):
    x = rng.standard_normal((B * L, C))
    w = rng.standard_normal((3 * H * d, C)) / np.sqrt(C)
    bias = 0.3 * rng.standard_normal(3 * H * d)
    gq = 1.0 + 0.2 * rng.standard_normal(d)
    gk = 1.0 + 0.2 * rng.standard_normal(d)
    return x, w, bias, gq, gk


def check_qkv_brute(qkv_fn, spec_cls):
    """Against scalar loops (projection, norm, gain, complex rotation)."""
    from tests import brute

    rng = _rng(71)
    B, L, H, d = 2, 6, 2, 12
    x, w, bias, gq, gk = _qkv_case(rng, B, L, H, d)
    grid, dims = (1, 2, 3), (4, 4, 4)
    spec = spec_cls(grid=grid, dims=dims, theta=50.0)
    got = qkv_fn(x, w, bias, B, L, H, d, gq, gk, 1e-5, spec)
    ref = brute.qkv_proj(x.tolist(), w.tolist(), bias.tolist(), B, L, H, d, gq.tolist(), gk.tolist(), 1e-5,
                         (grid, dims, 50.0, 0))
    for g, r in zip(got, ref):
        assert np.allclose(g, np.array(r), rtol=1e-11, atol=1e-12)


def check_qkv_permutation_weight(qkv_fn, spec_cls):
    """A permutation weight picks input channels: output channel n of the
    projection is x[:, pi(n)] (tests the orientation of W and the q, k, v
    order of its rows)."""
    rng = _rng(72)
    B, L, H, d = 1, 5, 2, 8
    C = 3 * H * d
    x = rng.standard_normal((B * L, C))
    pi = rng.permutation(C)
    w = np.zeros((C, C))
    w[np.arange(C), pi] = 1.0
    q, k, v = qkv_fn(x, w, None, B, L, H, d, None, None, 0.0, None)
    y = x[:, pi]
    hd = H * d

    def normed(z):
        z = z.reshape(B, L, H, d)
        return z / np.sqrt(np.mean(z * z, axis=-1, keepdims=True))

    assert np.allclose(v, y[:, 2 * hd:].reshape(B, L, H, d), rtol=1e-14, atol=0)
    assert np.allclose(q, normed(y[:, :hd]), rtol=1e-12, atol=1e-14)
    assert np.allclose(k, normed(y[:, hd:2 * hd]), rtol=1e-12, atol=1e-14)


def check_qkv_scale_and_gains(qkv_fn, spec_cls):
    """Without bias, scaling x by a > 0 leaves q and k alone and scales v;
    each gain acts on its own part only."""
    rng = _rng(73)
    B, L, H, d = 1, 4, 3, 8
    x, w, _, gq, gk = _qkv_case(rng, B, L, H, d, C=9)
    spec = spec_cls(grid=(1, 2, 2), dims=(2, 2, 4), theta=100.0)
    q, k, v = qkv_fn(x, w, None, B, L, H, d, gq, gk, 1e-9, spec)
    q2, k2, v2 = qkv_fn(3.5 * x, w, None, B, L, H, d, gq, gk, 1e-9, spec)
    assert np.allclose(q2, q, rtol=1e-8) and np.allclose(k2, k, rtol=1e-8)
    assert np.allclose(v2, 3.5 * v, rtol=1e-12)
    q3, k3, v3 = qkv_fn(x, w, None, B, L, H, d, 2.0 * gq, gk, 1e-9, spec)
    assert np.allclose(q3, 2.0 * q, rtol=1e-12) and np.allclose(k3, k, rtol=1e-14) and np.allclose(v3, v)


ALL_QKV_CHECKS = [check_qkv_brute, check_qkv_permutation_weight, check_qkv_scale_and_gains]
