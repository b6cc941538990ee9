"""MI355X-native 3D-RoPE + flash-attention forward (video-DiT attention hot path).

Thin ctypes binding over ``libvidax.so`` (C ABI declared in include/vidax.h).
This module only marshals arguments: torch provides device memory and the
current HIP stream; every step of the computation runs in the library's
kernels.  If the library has not been built the calls raise immediately --
there is no fallback implementation.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvidax.so")

VIDAX_OK = 0
_STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported configuration", 3: "kernel launch failed",
           4: "request exceeds the fixed device scratch of an allocation-free entry point"}

EXPORTED_SYMBOLS = (
    "vidax_rope3d",
    "vidax_rope3d_transpose",
    "vidax_attn_bwd",
    "vidax_attn_bwd_workspace_floats",
    "vidax_attn_bwd_noalloc",
    "vidax_na3d_fwd",
    "vidax_qkv_proj",
    "vidax_qk_norm_rope",
    "vidax_attn_fwd",
    "vidax_attn_fwd_naive",
    "vidax_status_string",
    "vidax_abi_version",
)


class VidaxError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} returned {status} ({_STATUS.get(status, 'unknown')})")
        self.status = status


class RopeDesc(ctypes.Structure):
    """Mirror of vidax_rope3d_desc."""

    _fields_ = [
        ("grid_t", ctypes.c_int32),
        ("grid_h", ctypes.c_int32),
        ("grid_w", ctypes.c_int32),
        ("dim_t", ctypes.c_int32),
        ("dim_h", ctypes.c_int32),
        ("dim_w", ctypes.c_int32),
        ("theta", ctypes.c_float),
        ("pair_mode", ctypes.c_int32),
        ("keys_prerotated", ctypes.c_int32),
    ]


@dataclass(frozen=True)
class Rope:
    """3D rotary convention: token grid (T, Hp, Wp), channel split, theta, pairing."""

    grid: tuple
    dims: tuple = (44, 42, 42)
    theta: float = 10000.0
    pair_mode: int = 0
    keys_prerotated: bool = False  # attention: k already rotated (rotate q only)

    def desc(self) -> RopeDesc:
        return RopeDesc(*self.grid, *self.dims, float(self.theta), int(self.pair_mode), int(self.keys_prerotated))


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libvidax.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2609_18077_amd.build` "
                "(or __graft_entry__.build()); there is no fallback path"
            )
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
        L.vidax_rope3d.argtypes = [vp, vp, i32, i32, i32, i32, ctypes.POINTER(RopeDesc), vp]
        L.vidax_rope3d.restype = i32
        L.vidax_rope3d_transpose.argtypes = [vp, vp, i32, i32, i32, i32, ctypes.POINTER(RopeDesc), vp]
        L.vidax_rope3d_transpose.restype = i32
        L.vidax_attn_bwd.argtypes = [vp] * 10 + [ctypes.c_size_t, i32, i32, i32, i32, i32, f32, vp, vp]
        L.vidax_attn_bwd.restype = i32
        L.vidax_attn_bwd_workspace_floats.argtypes = [i32, i32, i32, i32, i32]
        L.vidax_attn_bwd_workspace_floats.restype = ctypes.c_size_t
        L.vidax_attn_bwd_noalloc.argtypes = [vp] * 9 + [i32, i32, i32, i32, i32, f32, vp, vp]
        L.vidax_attn_bwd_noalloc.restype = i32
        L.vidax_na3d_fwd.argtypes = [vp] * 5 + [i32] * 10 + [f32, vp]
        L.vidax_na3d_fwd.restype = i32
        L.vidax_qkv_proj.argtypes = [vp] * 5 + [f32] + [vp] * 3 + [i32] * 5 + [ctypes.POINTER(RopeDesc), vp]
        L.vidax_qkv_proj.restype = i32
        L.vidax_qk_norm_rope.argtypes = [vp, vp, vp, f32, i32, i32, i32, i32, ctypes.POINTER(RopeDesc), vp]
        L.vidax_qk_norm_rope.restype = i32
        for name in ("vidax_attn_fwd", "vidax_attn_fwd_naive"):
            fn = getattr(L, name)
            fn.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, f32, vp, ctypes.POINTER(RopeDesc), vp]
            fn.restype = i32
        L.vidax_status_string.argtypes = [i32]
        L.vidax_status_string.restype = ctypes.c_char_p
        L.vidax_abi_version.argtypes = []
        L.vidax_abi_version.restype = i32
        _lib = L
    return _lib


def _check(fn: str, status: int):
    if status != VIDAX_OK:
        raise VidaxError(fn, status)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(stream):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check_bshd(name, t):
    import torch

    if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
        raise ValueError(f"{name} must be a contiguous bfloat16 [B, L, H, d] device tensor")


def rope3d(x, rope: Rope, out=None, stream=None):
    """Rotated copy of x (bf16 [B, L, H, d]); out may be x itself (in place)."""
    import torch

    _check_bshd("x", x)
    y = torch.empty_like(x) if out is None else out
    _check_bshd("out", y)
    if y.shape != x.shape:
        raise ValueError("out must have the shape of x")
    B, L, H, d = x.shape
    desc = rope.desc()
    _check("vidax_rope3d", lib().vidax_rope3d(_ptr(x), _ptr(y), B, L, H, d, ctypes.byref(desc), _stream(stream)))
    return y


def rope3d_transpose(x, rope: Rope, out=None, stream=None):
    """R^T x (every pair rotated by minus its angle); out may be x itself."""
    import torch

    _check_bshd("x", x)
    y = torch.empty_like(x) if out is None else out
    _check_bshd("out", y)
    if y.shape != x.shape:
        raise ValueError("out must have the shape of x")
    B, L, H, d = x.shape
    desc = rope.desc()
    _check("vidax_rope3d_transpose",
           lib().vidax_rope3d_transpose(_ptr(x), _ptr(y), B, L, H, d, ctypes.byref(desc), _stream(stream)))
    return y


def attn_bwd(q, k, v, o, dout, lse, scale=None, kv_valid_len=None, stream=None, noalloc=False, out=None,
             workspace=None):
    """(dq, dk, dv) of attention without rotation, from the forward's o and lse.

    noalloc=True calls vidax_attn_bwd_noalloc (D in the library's fixed
    device array instead of a workspace tensor); `out` = (dq, dk, dv) tensors
    to write into instead of new ones; `workspace` = a contiguous float32
    device tensor to use as the workspace (by default one of
    vidax_attn_bwd_workspace_floats values is allocated)."""
    import torch

    for n, t in (("q", q), ("k", k), ("v", v), ("o", o), ("dout", dout)):
        _check_bshd(n, t)
    B, Lq, H, d = q.shape
    Lk = k.shape[1]
    if k.shape != v.shape or o.shape != q.shape or dout.shape != q.shape:
        raise ValueError("shapes: q, o, dout [B, Lq, H, d]; k, v [B, Lk, H, d]")
    if lse.dtype != torch.float32 or not lse.is_cuda or not lse.is_contiguous() or lse.shape != (B, H, Lq):
        raise ValueError("lse must be a contiguous float32 [B, H, Lq] device tensor")
    if scale is None:
        scale = float(torch.tensor(1.0 / d ** 0.5, dtype=torch.float32))
    if kv_valid_len is not None:
        if kv_valid_len.dtype != torch.int32 or not kv_valid_len.is_cuda or kv_valid_len.numel() != B:
            raise ValueError("kv_valid_len must be an int32 device tensor of B elements")
        kv_valid_len = kv_valid_len.contiguous()
    if out is None:
        dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    else:
        dq, dk, dv = out
        for n, t, ref in (("dq", dq, q), ("dk", dk, k), ("dv", dv, v)):
            _check_bshd(n, t)
            if t.shape != ref.shape:
                raise ValueError(f"{n} must have shape {tuple(ref.shape)}")
    if noalloc:
        _check("vidax_attn_bwd_noalloc",
               lib().vidax_attn_bwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse), _ptr(dq),
                                            _ptr(dk), _ptr(dv), B, H, Lq, Lk, d, float(scale), _ptr(kv_valid_len),
                                            _stream(stream)))
        return dq, dk, dv
    if workspace is None:
        n = lib().vidax_attn_bwd_workspace_floats(B, H, Lq, Lk, d)
        workspace = torch.empty((max(n, B * H * Lq),), dtype=torch.float32, device=q.device)
    elif workspace.dtype != torch.float32 or not workspace.is_cuda or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous float32 device tensor")
    _check("vidax_attn_bwd", lib().vidax_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse), _ptr(dq),
                                                  _ptr(dk), _ptr(dv), _ptr(workspace), workspace.numel(), B, H, Lq,
                                                  Lk, d, float(scale), _ptr(kv_valid_len), _stream(stream)))
    return dq, dk, dv


def na3d_fwd(q, k, v, grid, window=(11, 11, 11), border: str = "clip", scale=None, return_lse=False, out=None,
             stream=None):
    """3D neighbourhood attention on a token grid (T, Hp, Wp); q, k, v bf16
    [B, T*Hp*Wp, H, d].  border "clip" or "shift"."""
    import torch

    for n, t in (("q", q), ("k", k), ("v", v)):
        _check_bshd(n, t)
    if k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must have the same shape [B, L, H, d]")
    B, L, H, d = q.shape
    T, Hp, Wp = (int(x) for x in grid)
    if T * Hp * Wp != L:
        raise ValueError("grid does not match L")
    if border not in ("clip", "shift"):
        raise ValueError("border must be 'clip' or 'shift'")
    if scale is None:
        scale = float(torch.tensor(1.0 / d ** 0.5, dtype=torch.float32))
    o = torch.empty_like(q) if out is None else out
    _check_bshd("out", o)
    lse = torch.empty((B, H, L), dtype=torch.float32, device=q.device) if return_lse else None
    _check("vidax_na3d_fwd", lib().vidax_na3d_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, H, T, Hp, Wp, d,
                                                  *(int(x) for x in window), 0 if border == "clip" else 1,
                                                  float(scale), _stream(stream)))
    return (o, lse) if return_lse else o


def qkv_proj(x, w, B: int, L: int, H: int, bias=None, gain_q=None, gain_k=None, eps: float = 1e-6,
             rope: Rope | None = None, stream=None):
    """(q, k, v) bf16 [B, L, H, 128] from hidden states x (bf16 [B*L, C]) and
    the projection weight w (bf16 [3*H*128, C]); q and k RMS-normalised per
    head, gained and rotated."""
    import torch

    for n, t in (("x", x), ("w", w)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() or t.dim() != 2:
            raise ValueError(f"{n} must be a contiguous 2-D bfloat16 device tensor")
    C = x.shape[1]
    d = w.shape[0] // (3 * H) if H > 0 else 0
    if x.shape[0] != B * L or w.shape[1] != C or w.shape[0] != 3 * H * d:
        raise ValueError("x must be [B*L, C] and w [3*H*d, C]")
    for n, t, size in (("bias", bias, 3 * H * d), ("gain_q", gain_q, d), ("gain_k", gain_k, d)):
        if t is not None and (t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous()
                              or t.numel() != size):
            raise ValueError(f"{n} must be a contiguous float32 device tensor of {size} elements")
    q, k, v = (torch.empty((B, L, H, d), dtype=torch.bfloat16, device=x.device) for _ in range(3))
    desc = rope.desc() if rope is not None else None
    _check("vidax_qkv_proj", lib().vidax_qkv_proj(_ptr(x), _ptr(w), _ptr(bias), _ptr(gain_q), _ptr(gain_k),
                                                  float(eps), _ptr(q), _ptr(k), _ptr(v), B, L, H, d, C,
                                                  ctypes.byref(desc) if desc is not None else None,
                                                  _stream(stream)))
    return q, k, v


def qk_norm_rope(x, rope: Rope | None = None, gain=None, eps: float = 1e-6, out=None, stream=None):
    """Per-(token, head) RMS normalisation of x (bf16 [B, L, H, d]), channel
    gain (fp32 [d] device tensor or None), then the 3D rotation (or none);
    out may be x itself (in place)."""
    import torch

    _check_bshd("x", x)
    y = torch.empty_like(x) if out is None else out
    _check_bshd("out", y)
    if y.shape != x.shape:
        raise ValueError("out must have the shape of x")
    B, L, H, d = x.shape
    if gain is not None:
        if gain.dtype != torch.float32 or not gain.is_cuda or not gain.is_contiguous() or gain.numel() != d:
            raise ValueError("gain must be a contiguous float32 device tensor of d elements")
    desc = rope.desc() if rope is not None else None
    _check("vidax_qk_norm_rope", lib().vidax_qk_norm_rope(_ptr(x), _ptr(y), _ptr(gain), float(eps), B, L, H, d,
                                                          ctypes.byref(desc) if desc is not None else None,
                                                          _stream(stream)))
    return y


def _attn(fn_name, q, k, v, scale, kv_valid_len, rope, return_lse, out, stream):
    import torch

    for n, t in (("q", q), ("k", k), ("v", v)):
        _check_bshd(n, t)
    B, Lq, H, d = q.shape
    if k.shape != v.shape or k.shape[0] != B or k.shape[2] != H or k.shape[3] != d:
        raise ValueError("k and v must be [B, Lk, H, d] matching q's B, H, d")
    Lk = k.shape[1]
    if scale is None:
        scale = float(torch.tensor(1.0 / d ** 0.5, dtype=torch.float32))
    o = torch.empty_like(q) if out is None else out
    _check_bshd("out", o)
    lse = torch.empty((B, H, Lq), dtype=torch.float32, device=q.device) if return_lse else None
    if kv_valid_len is not None:
        if kv_valid_len.dtype != torch.int32 or not kv_valid_len.is_cuda or kv_valid_len.numel() != B:
            raise ValueError("kv_valid_len must be an int32 device tensor of B elements")
        kv_valid_len = kv_valid_len.contiguous()
    desc = rope.desc() if rope is not None else None
    fn = getattr(lib(), fn_name)
    st = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, H, Lq, Lk, d, float(scale),
            _ptr(kv_valid_len), ctypes.byref(desc) if desc is not None else None, _stream(stream))
    _check(fn_name, st)
    return (o, lse) if return_lse else o


def attn_fwd(q, k, v, scale=None, kv_valid_len=None, rope: Rope | None = None, return_lse=False, out=None,
             stream=None):
    """softmax(scale * rope(q) rope(k)^T) v on the matrix-core kernel (bf16 in/out, fp32 accumulate)."""
    return _attn("vidax_attn_fwd", q, k, v, scale, kv_valid_len, rope, return_lse, out, stream)


def attn_fwd_naive(q, k, v, scale=None, kv_valid_len=None, rope: Rope | None = None, return_lse=False, out=None,
                   stream=None):
    """Same contract on the scalar fp32 cross-check kernel (small sizes only)."""
    return _attn("vidax_attn_fwd_naive", q, k, v, scale, kv_valid_len, rope, return_lse, out, stream)
