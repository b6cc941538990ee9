"""The C-ABI library on the CPU: it loads, exports what include/vidax.h
declares, and rejects invalid arguments synchronously (no kernel is launched,
no GPU is needed)."""

import ctypes
import os
import re

import pytest

import paper_2609_18077_amd as vx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "vidax.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(vidax_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = vx.lib()
    declared = _header_functions()
    assert set(declared) == set(vx.EXPORTED_SYMBOLS), declared
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.vidax_abi_version() == 8
    for s, text in [(0, b"ok"), (1, b"invalid argument"), (2, b"unsupported configuration"), (3, b"kernel launch failed")]:
        assert lib.vidax_status_string(s) == text
    assert b"allocation-free" in lib.vidax_status_string(4)
    assert lib.vidax_status_string(99) == b"unknown status"


P = 1 << 40  # fake, 16-byte aligned "device" addresses far apart; never dereferenced


def _attn(fn="vidax_attn_fwd", q=P, k=2 * P, v=3 * P, o=4 * P, lse=None, B=1, H=2, Lq=64, Lk=64, d=128,
          scale=0.088, kv=None, rope=None):
    f = getattr(vx.lib(), fn)
    return f(ctypes.c_void_p(q), ctypes.c_void_p(k), ctypes.c_void_p(v), ctypes.c_void_p(o),
             ctypes.c_void_p(lse) if lse else None, B, H, Lq, Lk, d, scale,
             ctypes.c_void_p(kv) if kv else None, ctypes.byref(rope) if rope is not None else None, None)


@pytest.mark.parametrize("fn", ["vidax_attn_fwd", "vidax_attn_fwd_naive"])
def test_attn_rejects_invalid_arguments(fn):
    INV, UNS = 1, 2
    assert _attn(fn, q=0) == INV
    assert _attn(fn, o=0) == INV
    assert _attn(fn, q=0, o=0, k=0, v=0, Lq=0, Lk=0) == 0  # empty: no-op, NULL allowed
    assert _attn(fn, q=P + 8) == INV            # misaligned
    assert _attn(fn, lse=5 * P + 2) == INV      # misaligned lse
    assert _attn(fn, kv=6 * P + 1) == INV       # misaligned lengths
    assert _attn(fn, B=-1) == INV
    assert _attn(fn, Lk=-3) == INV
    assert _attn(fn, scale=float("nan")) == INV
    assert _attn(fn, scale=float("inf")) == INV
    assert _attn(fn, d=64) == UNS
    assert _attn(fn, H=64, Lq=140000, Lk=64) == UNS   # one batch of q beyond 2 GiB
    assert _attn(fn, o=P) == INV                # output aliases q
    assert _attn(fn, o=2 * P + 4096) == INV     # output overlaps k
    assert _attn(fn, lse=2 * P + 256) == INV    # lse overlaps k
    assert _attn(fn, lse=3 * P) == INV          # lse aliases v
    assert _attn(fn, lse=5 * P, kv=4 * P + 64) == INV        # lengths overlap o
    assert _attn(fn, lse=5 * P, kv=5 * P + 16) == INV        # lengths overlap lse
    assert _attn(fn, lse=5 * P, kv=6 * P, Lq=0, q=0, o=0) == 0  # no query rows: nothing to check or launch
    good = vx.Rope((1, 8, 8), (44, 42, 42)).desc()
    bad = [vx.Rope((1, 8, 8), (44, 42, 40)).desc(),     # dims do not sum to d
           vx.Rope((1, 8, 8), (43, 43, 42)).desc(),     # odd dims
           vx.Rope((0, 8, 8), (44, 42, 42)).desc(),     # empty grid
           vx.Rope((1, 8, 8), (44, 42, 42), theta=0.0).desc(),
           vx.Rope((1, 8, 8), (44, 42, 42), theta=-1.0).desc(),
           vx.Rope((1, 8, 8), (44, 42, 42), pair_mode=2).desc(),
           vx.Rope((2, 8, 8), (44, 42, 42)).desc()]     # 128 rotated tokens > Lq = 64
    flag = vx.Rope((1, 8, 8), (44, 42, 42)).desc()
    flag.keys_prerotated = 2
    bad.append(flag)
    for r in bad:
        assert _attn(fn, rope=r) == INV
    # rotary table larger than the on-chip table
    assert _attn(fn, Lq=1 << 20, Lk=1 << 20, rope=vx.Rope((64, 128, 128), (44, 42, 42)).desc()) == UNS
    del good


def test_half_split_attention_needs_prerotated_keys():
    # the fused key rotation pairs interleaved channels only
    r = vx.Rope((1, 8, 8), (44, 42, 42), pair_mode=1).desc()
    assert _attn("vidax_attn_fwd", rope=r) == 2


def test_rope3d_rejects_invalid_arguments():
    f = vx.lib().vidax_rope3d
    good = vx.Rope((2, 4, 8), (44, 42, 42)).desc()

    def call(x=P, y=2 * P, B=1, L=64, H=2, d=128, rope=good):
        return f(ctypes.c_void_p(x), ctypes.c_void_p(y), B, L, H, d,
                 ctypes.byref(rope) if rope is not None else None, None)

    assert call(rope=None) == 1
    assert call(x=0) == 1
    assert call(x=0, y=0, L=0, rope=vx.Rope((1, 1, 1), (44, 42, 42)).desc()) == 1  # 1 rotated token > L = 0
    assert call(y=2 * P + 2) == 1
    assert call(L=-1) == 1
    assert call(d=96) == 2
    assert call(L=63) == 1                    # 64 rotated tokens > L
    assert call(y=P + 256) == 1               # partial overlap (in place is x == y)
    assert call(rope=vx.Rope((2, 4, 8), (42, 42, 42)).desc()) == 1


def test_qk_norm_rope_rejects_invalid_arguments():
    f = vx.lib().vidax_qk_norm_rope
    good = vx.Rope((2, 4, 8), (44, 42, 42)).desc()

    def call(x=P, y=2 * P, gain=3 * P, eps=1e-6, B=1, L=64, H=2, d=128, rope=good):
        return f(ctypes.c_void_p(x), ctypes.c_void_p(y), ctypes.c_void_p(gain) if gain else None, eps, B, L, H, d,
                 ctypes.byref(rope) if rope is not None else None, None)

    assert call(x=0) == 1
    assert call(x=0, y=0, L=0, rope=None) == 0       # empty: no-op, NULL allowed
    assert call(y=2 * P + 2) == 1                    # misaligned output
    assert call(gain=3 * P + 4) == 1                 # misaligned gain
    assert call(eps=-1e-6) == 1
    assert call(eps=float("nan")) == 1
    assert call(eps=float("inf")) == 1
    assert call(L=-1) == 1
    assert call(d=64) == 2
    assert call(L=63) == 1                           # 64 rotated tokens > L
    assert call(y=P + 256) == 1                      # partial overlap (in place is x == y)
    assert call(gain=2 * P + 512) == 1               # gain overlaps the output
    assert call(rope=vx.Rope((2, 4, 8), (44, 42, 42), pair_mode=2).desc()) == 1  # no such pair convention
    assert call(rope=vx.Rope((2, 4, 8), (40, 42, 42)).desc()) == 1               # widths do not sum to d


def _bwd_call(noalloc=False):
    f = vx.lib().vidax_attn_bwd_noalloc if noalloc else vx.lib().vidax_attn_bwd

    def call(q=P, k=2 * P, v=3 * P, o=4 * P, do=5 * P, lse=6 * P, dq=7 * P, dk=8 * P, dv=9 * P, delta=10 * P,
             B=1, H=2, Lq=64, Lk=64, d=128, scale=0.088, kv=None, ws_floats=None):
        ptr = lambda x: ctypes.c_void_p(x) if x else None
        if noalloc:
            return f(ptr(q), ptr(k), ptr(v), ptr(o), ptr(do), ptr(lse), ptr(dq), ptr(dk), ptr(dv),
                     B, H, Lq, Lk, d, scale, ptr(kv), None)
        n = max(B * H * Lq, 0) if ws_floats is None else ws_floats
        return f(ptr(q), ptr(k), ptr(v), ptr(o), ptr(do), ptr(lse), ptr(dq), ptr(dk), ptr(dv), ptr(delta), n,
                 B, H, Lq, Lk, d, scale, ptr(kv), None)
    return call


def test_attn_bwd_rejects_invalid_arguments():
    INV, UNS = 1, 2
    call = _bwd_call()

    assert call(q=0) == INV
    assert call(delta=0) == INV
    assert call(lse=0) == INV
    assert call(q=0, o=0, do=0, dq=0, lse=0, delta=0, k=0, v=0, dk=0, dv=0, Lq=0, Lk=0) == 0  # empty
    assert call(dq=7 * P + 8) == INV          # misaligned
    assert call(delta=10 * P + 4) == INV      # misaligned workspace
    assert call(kv=11 * P + 2) == INV
    assert call(B=-1) == INV
    assert call(scale=float("nan")) == INV
    assert call(d=64) == UNS
    assert call(H=140000) == UNS              # one 64-row tile beyond 2 GiB
    assert call(dq=P) == INV                  # output aliases an input
    assert call(dk=7 * P + 1024) == INV       # outputs overlap each other
    assert call(delta=6 * P) == INV           # workspace aliases lse
    assert call(kv=7 * P + 32) == INV         # lengths overlap dq
    assert call(kv=10 * P) == INV             # lengths alias the workspace
    assert call(ws_floats=2 * 64 - 1) == INV  # workspace smaller than D
    assert call(ws_floats=P // 4, kv=10 * P + P // 2) == INV  # a larger workspace reaching the lengths
    assert call(ws_floats=P // 4, dv=10 * P + 4096) == INV     # ... or an output
    assert call(ws_floats=2 ** 62) == INV     # absurd size


def test_attn_bwd_workspace_floats():
    f = vx.lib().vidax_attn_bwd_workspace_floats
    assert f(-1, 2, 64, 64, 128) == 0
    assert f(1, 2, 64, 64, 96) == 0
    assert f(1, 2, 0, 64, 128) == 0
    # many key workgroups, or too few query tiles to cut: D only
    assert f(1, 12, 32760, 32760, 128) == 12 * 32760
    assert f(1, 2, 512, 512, 128) == 2 * 512
    # text cross-attention shape: 2 x 40 x ceil(512 / 128) = 320 key workgroups
    # -> cut into runs; D (padded to 64 values) then 2 x qsplit partial tensors
    n = f(2, 40, 32760, 512, 128)
    rows = 2 * 40 * 32760
    grad = 2 * 512 * 40 * 128
    assert n > rows and (n - (rows + 63) // 64 * 64) % (2 * grad) == 0
    assert 2 <= (n - (rows + 63) // 64 * 64) // (2 * grad) <= 16


def test_attn_bwd_noalloc_rejects_invalid_arguments():
    INV, UNS, BIG = 1, 2, 4
    call = _bwd_call(noalloc=True)
    max_rows = 4194304  # VIDAX_NOALLOC_MAX_ROWS
    assert call(q=0) == INV
    assert call(lse=0) == INV
    assert call(q=0, o=0, do=0, dq=0, lse=0, k=0, v=0, dk=0, dv=0, Lq=0, Lk=0) == 0  # empty
    assert call(dq=7 * P + 8) == INV
    assert call(d=64) == UNS
    assert call(dq=P) == INV
    assert call(kv=9 * P) == INV              # lengths alias dv
    # beyond the fixed scratch: rejected before any HIP call
    assert call(B=1, H=64, Lq=max_rows // 64 + 1, Lk=64) == BIG
    assert call(B=2, H=32, Lq=max_rows // 64 + 64, Lk=64) == BIG
    # at the limit it would launch: only checked on the GPU


def test_rope3d_transpose_rejects_invalid_arguments():
    f = vx.lib().vidax_rope3d_transpose
    good = vx.Rope((2, 4, 8), (44, 42, 42)).desc()
    assert f(ctypes.c_void_p(P), ctypes.c_void_p(2 * P), 1, 64, 2, 128, None, None) == 1
    assert f(ctypes.c_void_p(P), ctypes.c_void_p(2 * P), 1, 63, 2, 128, ctypes.byref(good), None) == 1
    assert f(ctypes.c_void_p(P), ctypes.c_void_p(2 * P), 1, 64, 2, 96, ctypes.byref(good), None) == 2


def test_na3d_rejects_invalid_arguments():
    f = vx.lib().vidax_na3d_fwd
    INV, UNS = 1, 2

    def call(q=P, k=2 * P, v=3 * P, o=4 * P, lse=5 * P, B=1, H=2, g=(3, 5, 7), d=128, win=(3, 3, 3), border=0,
             scale=0.088):
        ptr = lambda x: ctypes.c_void_p(x) if x else None
        return f(ptr(q), ptr(k), ptr(v), ptr(o), ptr(lse), B, H, *g, d, *win, border, scale, None)

    assert call(win=(2, 3, 3)) == INV       # even window
    assert call(win=(3, 0, 3)) == INV
    assert call(border=2) == INV
    assert call(scale=float("inf")) == INV
    assert call(q=0) == INV
    assert call(B=-1) == INV
    assert call(o=4 * P + 8) == INV         # misaligned
    assert call(lse=5 * P + 2) == INV
    assert call(d=64) == UNS
    assert call(win=(3, 3, 13)) == UNS      # w window beyond one 16-key run
    assert call(o=P) == INV                 # output aliases q
    assert call(lse=3 * P + 64) == INV      # lse inside v
    assert call(lse=4 * P + 1024) == INV    # lse overlaps o
    assert call(B=0, q=0, k=0, v=0, o=0, lse=0) == 0  # empty
    assert call(g=(0, 5, 7), q=0, k=0, v=0, o=0) == 0


def test_qkv_proj_rejects_invalid_arguments():
    f = vx.lib().vidax_qkv_proj
    INV, UNS = 1, 2
    good = vx.Rope((2, 4, 8), (44, 42, 42)).desc()

    def call(x=P, w=2 * P, bias=3 * P, gq=4 * P, gk=5 * P, eps=1e-6, q=6 * P, k=7 * P, v=8 * P, B=1, L=64, H=2,
             d=128, C=256, rope=None):
        ptr = lambda a: ctypes.c_void_p(a) if a else None
        return f(ptr(x), ptr(w), ptr(bias), ptr(gq), ptr(gk), eps, ptr(q), ptr(k), ptr(v), B, L, H, d, C,
                 ctypes.byref(rope) if rope is not None else None, None)

    assert call(x=0) == INV
    assert call(q=0) == INV
    assert call(B=-1) == INV
    assert call(eps=-1.0) == INV
    assert call(eps=float("nan")) == INV
    assert call(bias=3 * P + 4) == INV      # misaligned
    assert call(k=7 * P + 8) == INV
    assert call(d=64) == UNS
    assert call(C=96) == UNS                # not a multiple of 64
    assert call(q=P) == INV                 # output aliases x
    assert call(v=2 * P + 512) == INV       # output inside w
    assert call(k=6 * P + 1024) == INV      # outputs overlap
    bad = vx.Rope((2, 4, 8), (44, 42, 42), pair_mode=2).desc()
    assert call(rope=bad) == INV            # no such pair convention
    assert call(rope=good, L=63) == INV     # more rotated tokens than L
    assert call(B=0, x=0, w=0, q=0, k=0, v=0) == 0  # empty
    assert call(bias=0, gq=0, gk=0, C=0, L=0) == 0


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(vx, "_lib", None)
    monkeypatch.setattr(vx, "LIB_PATH", "/nonexistent/libvidax.so")
    with pytest.raises(RuntimeError, match="no fallback"):
        vx.lib()
