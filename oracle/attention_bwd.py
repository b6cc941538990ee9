"""Gradient of non-causal scaled dot-product attention, float64 reference
(test infrastructure only).

The paper names post-training (LoRA and full fine-tuning) as the next use of
its execution graph (Section 5, "Conclusions & Future Work"); that needs the
gradient of the attention of attention.py.  For batch b, head h, with the
saved forward output O and log-sum-exp, and the gradient dO of the loss with
respect to O, the definition of softmax attention gives (keys j < Lv_b only):

    P_ij  = exp(scale * <q_i, k_j> - lse_i)
    dV_j  = sum_i P_ij dO_i
    dP_ij = <dO_i, v_j>
    D_i   = sum_j P_ij dP_ij  = <dO_i, O_i>
    dS_ij = P_ij (dP_ij - D_i)
    dQ_i  = scale * sum_j dS_ij k_j
    dK_j  = scale * sum_i dS_ij q_i

Keys j >= Lv_b receive zero gradient; a batch with Lv_b = 0 has O = 0 and a
zero gradient everywhere.  q and k are the vectors the scores are formed from
(rotated ones when the forward rotated them; rope_transpose takes a gradient
back through the rotation).  Each (b, h) is evaluated with whole matrices,
P from lse recomputed here with the two-pass softmax of attention.py.

D_i is formed from O by its second expression; a backward pass has only the
output the forward saved (in practice rounded to the storage type), so
``o_saved`` may supply that O.  Without it O is the exact output.
"""

from __future__ import annotations

import numpy as np

from .attention import _valid_lengths, attn_ref, attn_ref_rows
from .rope3d import RopeSpec, rope3d_ref


def _one_head(q, k, v, do, scale, o_saved=None):
    """Gradients for one (b, h): q, do [Lq, d]; k, v [N, d] (valid keys only);
    o_saved [Lq, d] replaces the exact O in D."""
    s = scale * (q @ k.T)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    p = e / e.sum(axis=1, keepdims=True)
    o = p @ v if o_saved is None else o_saved
    dv = p.T @ do
    dp = do @ v.T
    delta = np.sum(do * o, axis=1, keepdims=True)
    ds = p * (dp - delta)
    dq = scale * (ds @ k)
    dk = scale * (ds.T @ q)
    return dq, dk, dv


def attn_bwd_ref(q, k, v, do, scale, kv_valid_len=None, o_saved=None):
    """(dq [B, Lq, H, d], dk [B, Lk, H, d], dv [B, Lk, H, d]) in float64;
    o_saved [B, Lq, H, d]: the forward output D is formed from (default: the
    exact output)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    B, Lq, H, d = q.shape
    Lk = k.shape[1]
    lv = _valid_lengths(kv_valid_len, B, Lk)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        n = lv[b]
        if n == 0:
            continue
        for h in range(H):
            os_ = None if o_saved is None else np.asarray(o_saved[b, :, h], dtype=np.float64)
            gq, gk, gv = _one_head(q[b, :, h], k[b, :n, h], v[b, :n, h], do[b, :, h], float(scale), os_)
            dq[b, :, h] = gq
            dk[b, :n, h] = gk
            dv[b, :n, h] = gv
    return dq, dk, dv


def attn_bwd_ref_rows(q, k, v, do, scale, q_rows, k_rows, kv_valid_len=None, workers: int = 1):
    """Exact gradient at selected rows: dq at query rows q_rows [B, Rq, H, d],
    dk and dv at key rows k_rows [B, Rk, H, d].  A dq row needs only its own
    probabilities and output (the forward of those rows); a dk/dv row needs
    every query's lse and D, which come from the full forward of attention.py
    (O exact), computed only when k_rows is not empty.  P is taken from lse by
    its definition, P_ij = exp(scale <q_i, k_j> - lse_i)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    q_rows = np.asarray(q_rows, dtype=np.int64)
    k_rows = np.asarray(k_rows, dtype=np.int64)
    B, Lq, H, d = q.shape
    Lk = k.shape[1]
    lv = _valid_lengths(kv_valid_len, B, Lk)
    oq, lq = attn_ref_rows(q, k, v, scale, q_rows, kv_valid_len=kv_valid_len, workers=workers)
    if len(k_rows):
        o, lse = attn_ref(q, k, v, scale, kv_valid_len=kv_valid_len, workers=workers)
    dq = np.zeros((B, len(q_rows), H, d))
    dk = np.zeros((B, len(k_rows), H, d))
    dv = np.zeros((B, len(k_rows), H, d))
    sc = float(scale)
    for b in range(B):
        n = lv[b]
        if n == 0:
            continue
        for h in range(H):
            K, V, Q, dO = k[b, :n, h], v[b, :n, h], q[b, :, h], do[b, :, h]
            # query rows
            dOr = dO[q_rows]
            p = np.exp(sc * (Q[q_rows] @ K.T) - lq[b, h][:, None])
            ds = p * (dOr @ V.T - np.sum(dOr * oq[b, :, h], axis=1)[:, None])
            dq[b, :, h] = sc * (ds @ K)
            # key rows (rows at or past n keep zero gradient)
            live = k_rows < n
            if live.any():
                D = np.sum(dO * o[b, :, h], axis=1)  # [Lq]
                kj, vj = K[k_rows[live]], V[k_rows[live]]
                p = np.exp(sc * (Q @ kj.T) - lse[b, h][:, None])  # [Lq, R]
                dv[b, live, h] = p.T @ dO
                ds = p * (dO @ vj.T - D[:, None])
                dk[b, live, h] = sc * (ds.T @ Q)
    return dq, dk, dv


def rope_transpose_ref(g, spec: RopeSpec, token_index=None):
    """Gradient through the rotation: R^T g, every pair rotated by -phi (the
    rotation is orthogonal).  A plane rotation by -phi is the rotation by phi
    conjugated by the reflection of the pair's second channel."""
    from .rope3d import pair_channels

    g = np.asarray(g, dtype=np.float64)
    flip = np.ones(g.shape[-1])
    for (_a, _j, _c0, c1, _om) in pair_channels(spec):
        flip[c1] = -1.0
    return rope3d_ref(g * flip, spec, token_index=token_index) * flip
