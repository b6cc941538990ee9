"""Query/key prologue: per-(token, head) RMS normalisation with a learned
per-channel gain, then the 3D rotary embedding -- float64 reference (test
infrastructure only).

The 3D-RoPE video DiTs the paper serves (Section 3, "Supported Models": Wan,
HunyuanVideo and the others) normalise each attention head's query and key
vector before rotating them; the benchmark workload's queries and keys are
prepared that way.  The paper prints no formula, so the standard RMS
normalisation is the reading taken:

  y[c] = x[c] / sqrt(mean_c'(x[c']^2) + eps) * g[c]      over the d channels
                                                          of one (token, head)

with the gain g shared by all heads (unit gain when absent), followed by the
rotation of rope3d_ref (Section 2, "3D RoPE, 3D VAEs, and flash attention").
"""

from __future__ import annotations

import numpy as np

from .rope3d import RopeSpec, rope3d_ref


def mean_square(x):
    """Mean of x^2 over the channels of each (token, head): shape [..., 1]."""
    return np.mean(x * x, axis=-1, keepdims=True)


def rms_scale(ms, eps):
    """1 / sqrt(mean square + eps)."""
    return 1.0 / np.sqrt(ms + eps)


def qk_norm_ref(x, gain=None, eps: float = 1e-6, rope: RopeSpec | None = None, token_index=None):
    """x [B, L, H, d] -> RMS-normalised, gained and (if rope) rotated, float64."""
    x = np.asarray(x, dtype=np.float64)
    y = x * rms_scale(mean_square(x), float(eps))
    if gain is not None:
        y = y * np.asarray(gain, dtype=np.float64)
    if rope is not None:
        y = rope3d_ref(y, rope, token_index=token_index)
    return y
