"""3D neighbourhood (windowed) attention, float64 reference (test infrastructure only).

The paper's LTX-2.5 VAE decoder uses neighbourhood attention over the
(t, h, w) token grid with an 11 x 11 x 11 window (Section 2, "3D RoPE, 3D
VAEs, and flash attention", and the porting-bug table, "Memory, Tiling &
Execution Graphs"); vidax evaluates it one query row at a time with a gather
of that row's window.  Each query attends only to the keys of its own window:

    W(i)  = keys (t', h', w') with t' in T(t), h' in H(h), w' in Ww(w)
    s_ij  = scale * <q_i, k_j>,  j in W(i)
    o_i   = sum_j exp(s_ij - m_i) v_j / sum_j exp(s_ij - m_i),  m_i = max_j s_ij
    lse_i = m_i + ln sum_j exp(s_ij - m_i)

with the per-axis window of a query at coordinate c on an axis of N positions
and odd size K = 2 r + 1.  The paper does not say what happens at the border;
two readings are provided:

    border "clip":  [max(0, c - r), min(N - 1, c + r)]   (fewer keys at borders)
    border "shift": the window keeps its K positions and moves inward,
                    start = clamp(c - r, 0, N - K)        (the whole axis if N <= K)

Tokens are in patchify order n = (t * Hp + h) * Wp + w.  Heads are independent;
there is no rotation (a VAE decoder attention) and no other masking.  The
softmax is the two-pass definition over each row's own key set.
"""

from __future__ import annotations

import concurrent.futures as cf

import numpy as np

BORDERS = ("clip", "shift")


def axis_window(c: int, N: int, K: int, border: str):
    """Inclusive key range [lo, hi] on one axis for a query at coordinate c."""
    if K < 1 or K % 2 == 0:
        raise ValueError("window sizes must be odd and >= 1")
    r = (K - 1) // 2
    if border == "clip":
        return max(0, c - r), min(N - 1, c + r)
    if border == "shift":
        if N <= K:
            return 0, N - 1
        lo = min(max(c - r, 0), N - K)
        return lo, lo + K - 1
    raise ValueError(f"border must be one of {BORDERS}")


def window_keys(t: int, h: int, w: int, grid, window, border: str) -> np.ndarray:
    """Token indices of the keys that query (t, h, w) attends to, ascending."""
    T, Hp, Wp = grid
    t0, t1 = axis_window(t, T, window[0], border)
    h0, h1 = axis_window(h, Hp, window[1], border)
    w0, w1 = axis_window(w, Wp, window[2], border)
    tt, hh, ww = np.meshgrid(np.arange(t0, t1 + 1), np.arange(h0, h1 + 1), np.arange(w0, w1 + 1), indexing="ij")
    return ((tt * Hp + hh) * Wp + ww).ravel()


def na3d_ref(q, k, v, scale, grid, window=(11, 11, 11), border: str = "clip", rows=None, workers: int = 1):
    """Neighbourhood attention.  q, k, v: [B, L, H, d] (float64 after decoding),
    L = T * Hp * Wp.  rows: query token indices to evaluate (default all; rows
    are independent, so each is exact).  Returns (o [B, R, H, d], lse [B, H, R])."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    T, Hp, Wp = (int(x) for x in grid)
    B, L, H, d = q.shape
    if L != T * Hp * Wp or k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must be [B, T*Hp*Wp, H, d]")
    rows = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    o = np.zeros((B, len(rows), H, d))
    lse = np.zeros((B, H, len(rows)))
    scale = float(scale)

    def run(ri):
        n = int(rows[ri])
        t, rem = divmod(n, Hp * Wp)
        h, w = divmod(rem, Wp)
        idx = window_keys(t, h, w, (T, Hp, Wp), window, border)
        kk, vv = k[:, idx], v[:, idx]  # [B, N, H, d]
        s = scale * np.einsum("bhd,bnhd->bhn", q[:, n], kk)
        m = s.max(axis=2, keepdims=True)
        e = np.exp(s - m)
        l = e.sum(axis=2, keepdims=True)
        o[:, ri] = np.einsum("bhn,bnhd->bhd", e, vv) / l
        lse[:, :, ri] = (m + np.log(l))[..., 0]

    if workers <= 1:
        for ri in range(len(rows)):
            run(ri)
    else:
        with cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(run, range(len(rows))))
    return o, lse
