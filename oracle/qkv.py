"""Query/key/value projection with the Q/K prologue applied to its output --
float64 reference (test infrastructure only).

The served video DiTs (Section 3, "Supported Models") form each attention
call's queries, keys and values with one linear projection of the hidden
states, normalise the query and key heads and rotate them (Section 2, "3D
RoPE, 3D VAEs, and flash attention") before the attention.  With hidden
states x [M, C] (M = B * L tokens), a weight W [3 H d, C] (rows = output
channels, in the order q heads, k heads, v heads) and an optional bias
[3 H d]:

    y      = x W^T + bias                   [M, 3 H d]
    q, k, v = the three [M, H d] column blocks of y, as [B, L, H, d]
    q      = qk_norm_ref(q, gain_q, eps, rope)   (per-head RMS norm, gain, rotation)
    k      = qk_norm_ref(k, gain_k, eps, rope)
    v      unchanged

qk_norm_ref is the reading of the prologue (qknorm.py); the matrix product is
a library routine.
"""

from __future__ import annotations

import numpy as np

from .qknorm import qk_norm_ref
from .rope3d import RopeSpec


def qkv_proj_ref(x, w, bias, B: int, L: int, H: int, d: int, gain_q=None, gain_k=None, eps: float = 1e-6,
                 rope: RopeSpec | None = None, token_index=None):
    """x [B*L, C], w [3*H*d, C], bias [3*H*d] or None -> (q, k, v) [B, L, H, d] float64.
    token_index: positions of the L tokens (default 0..L-1), for row subsets."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    y = x @ w.T
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64)
    hd = H * d
    q = y[:, :hd].reshape(B, L, H, d)
    k = y[:, hd:2 * hd].reshape(B, L, H, d)
    v = y[:, 2 * hd:].reshape(B, L, H, d)
    q = qk_norm_ref(q, gain_q, eps, rope, token_index=token_index)
    k = qk_norm_ref(k, gain_k, eps, rope, token_index=token_index)
    return q, k, v
