"""Seeded synthetic workloads shaped like the paper's video-DiT attention calls.

This module only draws random numbers and lays them out; it holds none of the
attention or rotary-embedding arithmetic.  It is the one piece of code that the
HIP path's tests/benchmark and the CPU oracle both consume: every tensor is
produced here as raw bfloat16 bit patterns (``numpy.uint16``), and each side
decodes those bits by itself.

Workload shapes follow the paper's benchmarked video models (Section 4 and the
full benchmark table): Wan2.1 at 832x480 and 1280x720 with 81 frames, and
HunyuanVideo 13B at 1280x720 with 129 frames, patchified to token grids
(T x Hp x Wp); head counts and head dim (d = 128) are those of the models.

Recipe (all tensors are [B, L, H, d] in that memory order):
  * each tensor is filled in chunks of ``CHUNK`` elements; chunk ``i`` of tensor
    ``t`` draws float32 N(0, 1) from ``PCG64(SeedSequence([seed, t, i]))`` so the
    result does not depend on the number of threads used;
  * optional per-(token, head) RMS normalisation over d in float32:
    ``x / sqrt(mean(x^2) + 1e-6)`` (unit gain) -- the input preparation of the
    Wan-style per-head-normalised Q/K;
  * rounding float32 -> bfloat16 to nearest, ties to even;
  * per-batch valid key lengths, when drawn, come from
    ``PCG64(SeedSequence([seed, 3]))`` as integers uniform on [lo, hi].
"""

from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass, field

import numpy as np

CHUNK = 1 << 22
HEAD_DIM = 128

# tensor ids used in the seed sequence
T_Q, T_K, T_V, T_LEN, T_DO = 0, 1, 2, 3, 4
# projection inputs: hidden states, weight, bias, gains
T_X, T_W, T_BIAS, T_GQ, T_GK = 5, 6, 7, 8, 9


@dataclass(frozen=True)
class Workload:
    """One attention call: shapes, rotary grid and masking recipe."""

    name: str
    B: int
    H: int
    Lq: int
    Lk: int
    seed: int
    d: int = HEAD_DIM
    # rotary grid (T, Hp, Wp) of the video tokens, or None for no rotary embedding
    grid: tuple | None = None
    dims: tuple = (44, 42, 42)
    theta: float = 10000.0
    rms_norm_qk: bool = False
    # key-length recipe: None (all keys valid), ("fixed", [..per batch..]) or
    # ("uniform", lo, hi)
    kv_valid: tuple | None = None
    description: str = field(default="", compare=False)

    @property
    def n_rot(self) -> int:
        if self.grid is None:
            return 0
        t, h, w = self.grid
        return t * h * w

    @property
    def scale(self) -> float:
        # the fp32 value of 1/sqrt(d), widened exactly
        return float(np.float32(1.0 / np.sqrt(self.d)))


WORKLOADS = {
    w.name: w
    for w in [
        Workload(
            "tiny", B=1, H=2, Lq=512, Lk=512, seed=1, grid=(2, 16, 16),
            description="tiny self-attention, grid 2x16x16",
        ),
        Workload(
            "wan13b_480p", B=1, H=12, Lq=32760, Lk=32760, seed=2, grid=(21, 30, 52),
            rms_norm_qk=True,
            description="Wan2.1-1.3B 832x480 81f self-attention, grid 21x30x52",
        ),
        Workload(
            "wan14b_720p", B=1, H=40, Lq=75600, Lk=75600, seed=3, grid=(21, 45, 80),
            description="Wan2.1-14B 1280x720 81f self-attention, grid 21x45x80",
        ),
        Workload(
            "cross_text", B=2, H=40, Lq=32760, Lk=512, seed=4, grid=None,
            kv_valid=("uniform", 64, 512),
            description="text cross-attention, 32760 video queries x 512 padded text keys",
        ),
        Workload(
            "hunyuan_joint", B=1, H=24, Lq=119056, Lk=119056, seed=5, grid=(33, 45, 80),
            kv_valid=("fixed", [118800 + 180]),
            description="HunyuanVideo-13B 1280x720 129f joint video+text attention",
        ),
    ]
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def normal_f32(seed: int, tensor_id: int, n: int) -> np.ndarray:
    """n float32 N(0,1) samples, chunked and thread-count independent."""
    out = np.empty(n, np.float32)
    nchunks = (n + CHUNK - 1) // CHUNK

    def fill(i):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tensor_id, i])))
        lo, hi = i * CHUNK, min(n, (i + 1) * CHUNK)
        g.standard_normal(out=out[lo:hi], dtype=np.float32)

    if nchunks == 1:
        fill(0)
    else:
        with _cf.ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(fill, range(nchunks)))
    return out


def _rms_norm_rows(x: np.ndarray, d: int) -> np.ndarray:
    """Per-row RMS normalisation of a flat float32 array viewed as rows of d."""
    rows = x.reshape(-1, d)
    step = 1 << 18

    def work(i):
        blk = rows[i:i + step]
        ms = np.mean(blk * blk, axis=1, dtype=np.float32)
        blk *= (1.0 / np.sqrt(ms + np.float32(1e-6))).astype(np.float32)[:, None]

    with _cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(work, range(0, rows.shape[0], step)))
    return x


def bf16_tensor(seed: int, tensor_id: int, shape, rms_norm: bool = False, std: float = 1.0) -> np.ndarray:
    """A bfloat16 tensor (uint16 bits) of the given shape, drawn N(0, std^2)."""
    n = int(np.prod(shape))
    x = normal_f32(seed, tensor_id, n)
    if std != 1.0:
        x *= np.float32(std)
    if rms_norm:
        x = _rms_norm_rows(x, shape[-1])
    out = np.empty(n, np.uint16)
    step = CHUNK

    def cvt(i):
        out[i:i + step] = f32_to_bf16_bits(x[i:i + step])

    with _cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(cvt, range(0, n, step)))
    return out.reshape(shape)


def kv_valid_len(w: Workload) -> np.ndarray | None:
    """Per-batch valid key lengths (int32[B]) or None when every key is valid."""
    if w.kv_valid is None:
        return None
    if w.kv_valid[0] == "fixed":
        return np.asarray(w.kv_valid[1], dtype=np.int32)
    if w.kv_valid[0] == "uniform":
        lo, hi = w.kv_valid[1], w.kv_valid[2]
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, T_LEN])))
        return g.integers(lo, hi + 1, size=w.B).astype(np.int32)
    raise ValueError(w.kv_valid)


def make_qkv(w: Workload):
    """(q, k, v, kv_valid_len) for a workload; q/k/v are uint16 bf16 bits."""
    q = bf16_tensor(w.seed, T_Q, (w.B, w.Lq, w.H, w.d), rms_norm=w.rms_norm_qk)
    k = bf16_tensor(w.seed, T_K, (w.B, w.Lk, w.H, w.d), rms_norm=w.rms_norm_qk)
    v = bf16_tensor(w.seed, T_V, (w.B, w.Lk, w.H, w.d))
    return q, k, v, kv_valid_len(w)


def make_dout(w: Workload) -> np.ndarray:
    """Upstream gradient of the attention output (bf16 bits, [B, Lq, H, d])."""
    return bf16_tensor(w.seed, T_DO, (w.B, w.Lq, w.H, w.d))


@dataclass(frozen=True)
class NaWorkload:
    """One neighbourhood-attention call: token grid, window, border reading."""

    name: str
    B: int
    H: int
    grid: tuple
    seed: int
    window: tuple = (11, 11, 11)
    border: str = "clip"
    d: int = HEAD_DIM
    description: str = field(default="", compare=False)

    @property
    def L(self) -> int:
        return self.grid[0] * self.grid[1] * self.grid[2]

    @property
    def scale(self) -> float:
        return float(np.float32(1.0 / np.sqrt(self.d)))


# The paper names the LTX-2.5 VAE decoder's 11 x 11 x 11 neighbourhood
# attention but not its shapes: the stand-in is a decoder stage at 1/16 of
# 1280 x 720 (80 x 45 positions) over 16 latent frames, 512 channels as 4
# heads of 128.
NA_WORKLOADS = {
    w.name: w
    for w in [
        NaWorkload("ltx_vae_na", B=1, H=4, grid=(16, 45, 80), seed=6,
                   description="VAE-decoder neighbourhood attention, grid 16x45x80, window 11^3"),
    ]
}


def make_na_qkv(w: NaWorkload):
    """(q, k, v) uint16 bf16 bits [B, L, H, d] of a neighbourhood-attention workload."""
    shape = (w.B, w.L, w.H, w.d)
    return tuple(bf16_tensor(w.seed, t, shape) for t in (T_Q, T_K, T_V))


@dataclass(frozen=True)
class ProjWorkload:
    """A Q/K/V projection of hidden states [B*L, C] into H heads of d, with the
    rotary grid of the tokens (None: no rotation)."""

    name: str
    B: int
    L: int
    H: int
    C: int
    seed: int
    grid: tuple | None = None
    dims: tuple = (44, 42, 42)
    theta: float = 10000.0
    bias: bool = True
    gains: bool = True
    eps: float = 1e-6
    d: int = HEAD_DIM
    description: str = field(default="", compare=False)


# Wan2.1-1.3B at 832 x 480, 81 frames: hidden size 1536 = 12 heads of 128
PROJ_WORKLOADS = {
    w.name: w
    for w in [
        ProjWorkload("wan13b_480p_qkv", B=1, L=32760, H=12, C=1536, seed=7, grid=(21, 30, 52),
                     description="Wan2.1-1.3B 832x480 81f: QKV projection of 32760 tokens, hidden 1536"),
    ]
}


def make_proj_inputs(w: ProjWorkload):
    """(x bf16 [B*L, C], W bf16 [3 H d, C], bias fp32 [3 H d] or None, gain_q,
    gain_k fp32 [d] or None): x ~ N(0, 1), W ~ N(0, 1/C) (unit-variance
    outputs), bias ~ N(0, 0.1^2), gains ~ 1 + N(0, 0.1^2)."""
    n = 3 * w.H * w.d
    x = bf16_tensor(w.seed, T_X, (w.B * w.L, w.C))
    wt = bf16_tensor(w.seed, T_W, (n, w.C), std=float(1.0 / np.sqrt(w.C)))
    bias = 0.1 * normal_f32(w.seed, T_BIAS, n) if w.bias else None
    gq = 1.0 + 0.1 * normal_f32(w.seed, T_GQ, w.d) if w.gains else None
    gk = 1.0 + 0.1 * normal_f32(w.seed, T_GK, w.d) if w.gains else None
    return x, wt, bias, gq, gk


def custom(name="custom", **kw) -> Workload:
    """A workload with explicit fields (used for parity cases between the named ones)."""
    return Workload(name=name, **kw)
