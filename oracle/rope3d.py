"""3D rotary position embedding, float64 reference (test infrastructure only).

Definition (paper Section 2, "3D RoPE, 3D VAEs, and flash attention": each
video token carries a (time, height, width) coordinate and its query/key
channels are rotated by angles proportional to those coordinates; the paper
keeps each model family's own convention, so the convention is a parameter).

Readings taken where the paper gives no formula:
  * tokens are in patchify order n = (t * Hp + h) * Wp + w, so
    t = n // (Hp*Wp), h = (n // Wp) % Hp, w = n % Wp; only tokens n < T*Hp*Wp
    are rotated (later tokens, e.g. appended text, are left unchanged);
  * the head dim is split into consecutive channel blocks for (t, h, w) of
    widths (d_t, d_h, d_w), each even, summing to d;
  * inside the block of axis a (offset o_a, width d_a), pair j in [0, d_a/2)
    has frequency omega = theta ** (-2 j / d_a) and angle phi = pos_a * omega;
  * pair_mode 0 ("interleaved") pairs channels (o_a + 2j, o_a + 2j + 1);
    pair_mode 1 ("half split") pairs (o_a + j, o_a + j + d_a/2);
  * a pair (x0, x1) becomes (x0 cos phi - x1 sin phi, x0 sin phi + x1 cos phi).
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class RopeSpec:
    grid: tuple  # (T, Hp, Wp): tokens n < T*Hp*Wp are rotated
    dims: tuple = (44, 42, 42)  # channel widths of the t, h, w blocks
    theta: float = 10000.0
    pair_mode: int = 0  # 0 interleaved, 1 half split

    @property
    def n_rot(self) -> int:
        t, h, w = self.grid
        return t * h * w


def token_coords(n: np.ndarray, grid) -> np.ndarray:
    """(t, h, w) integer coordinates of token indices n (shape [..., 3])."""
    T, Hp, Wp = grid
    n = np.asarray(n, dtype=np.int64)
    return np.stack([n // (Hp * Wp), (n // Wp) % Hp, n % Wp], axis=-1)


def pair_channels(spec: RopeSpec):
    """List of (axis, j, c0, c1, omega) for every rotated channel pair."""
    out = []
    off = 0
    for a, da in enumerate(spec.dims):
        for j in range(da // 2):
            omega = float(spec.theta) ** (-2.0 * j / da)
            if spec.pair_mode == 0:
                c0, c1 = off + 2 * j, off + 2 * j + 1
            else:
                c0, c1 = off + j, off + j + da // 2
            out.append((a, j, c0, c1, omega))
        off += da
    return out


def rope_angles(spec: RopeSpec, n: np.ndarray) -> np.ndarray:
    """Angles phi[token, pair] (float64) for token indices n."""
    coords = token_coords(n, spec.grid).astype(np.float64)
    pairs = pair_channels(spec)
    phi = np.empty((coords.shape[0], len(pairs)), np.float64)
    for p, (a, _j, _c0, _c1, omega) in enumerate(pairs):
        phi[:, p] = coords[:, a] * omega
    return phi


def rope3d_ref(x: np.ndarray, spec: RopeSpec, token_index: np.ndarray | None = None) -> np.ndarray:
    """Rotate x [B, L, H, d] (float64).  Row l of axis 1 is token token_index[l]
    (default: l).  Returns a new float64 array."""
    x = np.asarray(x, dtype=np.float64)
    B, L, H, d = x.shape
    if sum(spec.dims) != d or any(da % 2 for da in spec.dims):
        raise ValueError("rotary channel blocks must be even and sum to d")
    n = np.arange(L) if token_index is None else np.asarray(token_index, dtype=np.int64)
    y = x.copy()
    rot = n < spec.n_rot
    if not np.any(rot):
        return y
    rows = np.nonzero(rot)[0]
    phi = rope_angles(spec, n[rows])  # [R, P]
    cos = np.cos(phi)[None, :, None, :]
    sin = np.sin(phi)[None, :, None, :]
    pairs = pair_channels(spec)
    c0 = np.array([p[2] for p in pairs])
    c1 = np.array([p[3] for p in pairs])
    x0 = x[:, rows][..., c0]
    x1 = x[:, rows][..., c1]
    y0 = x0 * cos - x1 * sin
    y1 = x0 * sin + x1 * cos
    sub = y[:, rows]
    sub[..., c0] = y0
    sub[..., c1] = y1
    y[:, rows] = sub
    return y
