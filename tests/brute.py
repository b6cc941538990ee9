"""Pure-Python brute force of 3D RoPE + softmax attention, for tiny shapes.

A second formulation, written independently of the oracle: the rotation of a
channel pair is the complex product (x0 + i x1) * exp(i phi) with the token's
coordinates found by walking the (t, h, w) grid, and the softmax is a direct
sum of math.exp terms accumulated with math.fsum (no max subtraction, no
matrix products).  Only usable for small sizes and moderate logits.
"""

import cmath
import math


def coords_by_walk(n, grid):
    """(t, h, w) of token n found by enumerating the grid in patchify order."""
    T, Hp, Wp = grid
    idx = 0
    for t in range(T):
        for h in range(Hp):
            for w in range(Wp):
                if idx == n:
                    return (t, h, w)
                idx += 1
    return None  # token beyond the grid: not rotated


def rope_row(x, n, grid, dims, theta, pair_mode):
    """Rotate one head vector x (list of floats) of token n."""
    pos = coords_by_walk(n, grid)
    y = list(x)
    if pos is None:
        return y
    off = 0
    for a in range(3):
        da = dims[a]
        half = da // 2
        for j in range(half):
            if pair_mode == 0:
                c0, c1 = off + 2 * j, off + 2 * j + 1
            else:
                c0, c1 = off + j, off + half + j
            phi = pos[a] * math.pow(theta, -(2.0 * j) / da)
            z = complex(x[c0], x[c1]) * cmath.exp(1j * phi)
            y[c0], y[c1] = z.real, z.imag
        off += da
    return y


def attention(q, k, v, scale, kv_valid_len=None, rope=None):
    """q [B][Lq][H][d], k/v [B][Lk][H][d] nested lists; rope = (grid, dims, theta, mode).

    Returns (o, lse) as nested lists o[B][Lq][H][d], lse[B][H][Lq].
    """
    B, Lq, H, d = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    Lk = len(k[0])
    o = [[[[0.0] * d for _ in range(H)] for _ in range(Lq)] for _ in range(B)]
    lse = [[[float("-inf")] * Lq for _ in range(H)] for _ in range(B)]
    for b in range(B):
        lv = Lk if kv_valid_len is None else max(0, min(Lk, int(kv_valid_len[b])))
        for h in range(H):
            keys = []
            for j in range(lv):
                kj = k[b][j][h]
                if rope is not None:
                    kj = rope_row(kj, j, *rope)
                keys.append(kj)
            for i in range(Lq):
                qi = q[b][i][h]
                if rope is not None:
                    qi = rope_row(qi, i, *rope)
                if lv == 0:
                    continue
                w = [math.exp(scale * math.fsum(qi[c] * keys[j][c] for c in range(d))) for j in range(lv)]
                z = math.fsum(w)
                for c in range(d):
                    o[b][i][h][c] = math.fsum(w[j] * v[b][j][h][c] for j in range(lv)) / z
                lse[b][h][i] = math.log(z)
    return o, lse


def qk_norm_row(x, gain, eps, n, rope):
    """RMS-normalise one head vector x (list of floats) by a math.fsum of its
    squares, scale channel c by gain[c] (None: 1), then rotate it as token n
    (rope = (grid, dims, theta, mode) or None)."""
    d = len(x)
    r = math.sqrt(math.fsum(v * v for v in x) / d + eps)
    y = [x[c] / r * (1.0 if gain is None else gain[c]) for c in range(d)]
    if rope is None:
        return y
    grid, dims, theta, mode = rope
    return rope_row(y, n, grid, dims, theta, mode)


def _shift_start(c, N, K):
    """Start of the K-position window holding c whose centre lies nearest to c
    (found by trying every start)."""
    r = (K - 1) // 2
    return min(range(0, N - K + 1), key=lambda s: abs(s + r - c))


def _in_window(c, cp, N, K, border):
    """Does a key at axis position cp lie in the window of a query at c?"""
    r = (K - 1) // 2
    if border == "clip" or N <= K:
        return abs(cp - c) <= r if border == "clip" else True
    s = _shift_start(c, N, K)
    return s <= cp < s + K


def na3d(q, k, v, scale, grid, window, border):
    """Neighbourhood attention by testing every (query, key) pair of the grid
    (coordinates found by walking it).  q/k/v [B][L][H][d] nested lists.
    Returns (o [B][L][H][d], lse [B][H][L])."""
    B, L, H, d = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    pos = [coords_by_walk(n, grid) for n in range(L)]
    o = [[[[0.0] * d for _ in range(H)] for _ in range(L)] for _ in range(B)]
    lse = [[[0.0] * L for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            for i in range(L):
                keys = [j for j in range(L)
                        if all(_in_window(pos[i][a], pos[j][a], grid[a], window[a], border) for a in range(3))]
                e = [math.exp(scale * math.fsum(q[b][i][h][c] * k[b][j][h][c] for c in range(d))) for j in keys]
                z = math.fsum(e)
                for c in range(d):
                    o[b][i][h][c] = math.fsum(ej * v[b][j][h][c] for ej, j in zip(e, keys)) / z
                lse[b][h][i] = math.log(z)
    return o, lse


def qkv_proj(x, w, bias, B, L, H, d, gain_q, gain_k, eps, rope):
    """Projection, per-head RMS norm, gain and rotation with scalar loops.
    x [M][C], w [3Hd][C], bias [3Hd] (lists); gains [d] lists or None;
    rope = (grid, dims, theta, mode) or None.  Returns (q, k, v) as
    nested lists [B][L][H][d]."""
    C = len(x[0])
    hd = H * d
    out = []
    for part in range(3):
        t = [[[[0.0] * d for _ in range(H)] for _ in range(L)] for _ in range(B)]
        gain = gain_q if part == 0 else gain_k if part == 1 else None
        for b in range(B):
            for n in range(L):
                m = b * L + n
                for h in range(H):
                    row = []
                    for c in range(d):
                        col = part * hd + h * d + c
                        acc = math.fsum(x[m][cc] * w[col][cc] for cc in range(C))
                        row.append(acc + (bias[col] if bias is not None else 0.0))
                    if part < 2:
                        r = 1.0 / math.sqrt(math.fsum(z * z for z in row) / d + eps)
                        row = [z * r * (gain[c] if gain is not None else 1.0) for c, z in enumerate(row)]
                        if rope is not None:
                            row = rope_row(row, n, *rope)
                    t[b][n][h] = row
        out.append(t)
    return tuple(out)
