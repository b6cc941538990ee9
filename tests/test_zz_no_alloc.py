"""The allocation-free backward (vidax_attn_bwd_noalloc) against the backward
with a caller workspace (vidax_attn_bwd), through the C ABI.

Both run the same kernels when the workspace holds exactly D (B * H * Lq
values: no query-stream split); only where D is kept differs, so the
gradients must agree bit for bit.  Two calls in a row share the library's device array:
the first at the array's maximum size (B * H * Lq = VIDAX_NOALLOC_MAX_ROWS),
the second smaller, so a second call that read stale values of the first
would differ.  A request one row beyond the maximum is rejected with
VIDAX_ERR_TOO_LARGE and launches nothing.
"""

import pytest

import paper_2609_18077_amd as vx
from tests.gpu_util import log

pytestmark = pytest.mark.gpu

MAX_ROWS = 4194304  # VIDAX_NOALLOC_MAX_ROWS


def _case(torch, B, H, Lq, Lk, lens, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    mk = lambda L: torch.randn((B, L, H, 128), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    q, k, v, do = mk(Lq), mk(Lk), mk(Lk), mk(Lq)
    lv = None if lens is None else torch.tensor(lens, dtype=torch.int32, device="cuda")
    o, lse = vx.attn_fwd(q, k, v, kv_valid_len=lv, return_lse=True)
    return q, k, v, o, do, lse, lv


def _same_bits(torch, a, b):
    return bool(torch.equal(a.view(torch.int16), b.view(torch.int16)))


def test_noalloc_matches_workspace_backward_twice():
    import torch

    cases = [
        # first: the array's maximum size (one batch, 32 heads x 131072 queries)
        dict(B=1, H=32, Lq=MAX_ROWS // 32, Lk=96, lens=[77], seed=11),
        # second: smaller, ragged, two batches with different valid lengths
        dict(B=2, H=3, Lq=333, Lk=200, lens=[200, 45], seed=12),
    ]
    for c in cases:
        log(f"noalloc backward B={c['B']} H={c['H']} Lq={c['Lq']} Lk={c['Lk']} lens={c['lens']}")
        q, k, v, o, do, lse, lv = _case(torch, c["B"], c["H"], c["Lq"], c["Lk"], c["lens"], c["seed"])
        ws = torch.empty((c["B"] * c["H"] * c["Lq"],), dtype=torch.float32, device="cuda")
        ref = vx.attn_bwd(q, k, v, o, do, lse, kv_valid_len=lv, workspace=ws)
        out = tuple(torch.full_like(t, float("nan")) for t in ref)  # stale contents must be overwritten
        got = vx.attn_bwd(q, k, v, o, do, lse, kv_valid_len=lv, noalloc=True, out=out)
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv"), got, ref):
            assert _same_bits(torch, a, b), name
            assert bool(torch.isfinite(a.float()).all()), name
        del q, k, v, o, do, lse, ref, got, out, ws
        torch.cuda.empty_cache()


def test_noalloc_rejects_more_rows_than_the_array():
    import torch

    q = torch.zeros((1, MAX_ROWS // 64 + 1, 64, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((1, 64, 64, 128), dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros((1, 64, q.shape[1]), dtype=torch.float32, device="cuda")
    with pytest.raises(vx.VidaxError) as e:
        vx.attn_bwd(q, k, k, q, q, lse, noalloc=True)
    assert e.value.status == 4
