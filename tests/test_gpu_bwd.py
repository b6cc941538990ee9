"""GPU parity of the attention gradient (vidax_attn_bwd) and of the rotation's
transpose (vidax_rope3d_transpose) against the fp64 oracle, through the C ABI.

Tolerance.  The kernels round P and dS to bf16 before the products that
consume them (relative error <= 2^-9 each, independent across the summed
terms), accumulate in fp32 and round the gradients to bf16 (at most half an
ulp, <= 2^-8 relative).  D = <dO, O> is formed from the saved output, which
is bf16: the kernel-level tests give the oracle the same saved output (in
strongly peaked attention, dP - D cancels and the rounding of O alone would
move dq and dk by far more than 2^-9); the end-to-end tests compare with the
exact gradient at the models' scale 1/sqrt(d).  Each gradient
element is a sum over many terms whose rounding errors are independent, so
beyond its own output rounding its error is about 2^-9 of the typical
magnitude of its (batch, head) slice.  The test allows, per slice, 1%
relative RMS error (about five times the expected 2^-9) and, per element, one
bf16 ulp of the reference (2^-7 |ref|) plus 2^-5 of the slice's RMS (the
largest of ~10^6 independent 2^-9-relative errors is near 5 sigma, about 1%
of the RMS).  A key slice counts only its valid keys.  Gradients that
are zero by definition (keys at or past the valid length, queries of a batch
without valid keys) must be exactly zero.
"""

import numpy as np
import pytest

import oracle
import paper_2609_18077_amd as vx
from paper_2609_18077_amd import inputs
from tests.gpu_util import lengths_dev, log, rope_of, spec_of, to_bits, to_dev

pytestmark = pytest.mark.gpu

REL_RMS = 1e-2
ULP_REL = 2.0 ** -7
ABS_OVER_RMS = 2.0 ** -5


def _check_grad(got_bits, ref, what, rows=None):
    """Per (batch, head) slice of the first rows[b] rows (all rows when
    None): the natural magnitude of a gradient differs between batches (a
    batch with few valid keys has larger dv rows)."""
    got = oracle.bf16_bits_to_f64(got_bits)
    assert np.all(np.isfinite(got)), what
    worst_rel, worst_excess = 0.0, -np.inf
    for b in range(ref.shape[0]):
        for h in range(ref.shape[2]):
            n = ref.shape[1] if rows is None else int(rows[b])
            g, r = got[b, :n, h], ref[b, :n, h]
            rms = float(np.sqrt(np.mean(r * r))) if r.size else 0.0
            if rms == 0.0:
                # e.g. a single key: P = 1 and dP = D exactly, while the kernel
                # forms dP and D as fp32 sums in different orders (~1e-7)
                assert np.all(np.abs(g) <= 1e-4), (what, b, h, float(np.abs(g).max()))
                continue
            diff = np.abs(g - r)
            rel = float(np.sqrt(np.mean(diff * diff))) / rms
            excess = float(np.max(diff - ULP_REL * np.abs(r))) / rms
            worst_rel, worst_excess = max(worst_rel, rel), max(worst_excess, excess)
            assert rel <= REL_RMS, (what, b, h, rel)
            assert excess <= ABS_OVER_RMS, (what, b, h, excess)
    log(f"  {what}: worst slice rel_rms {worst_rel:.3e} (max err - ulp)/rms {worst_excess:.3e}")


def _key_rows(lv, w):
    return None if lv is None else np.minimum(np.maximum(lv, 0), w.Lk)


def _check_zeros(dq, dk, dv, lv, Lk):
    """Keys at or past Lv_b have dk = dv = 0; a batch with Lv_b = 0 has dq = 0."""
    if lv is None:
        return
    for b, n in enumerate(np.minimum(np.maximum(lv, 0), Lk)):
        assert np.all(oracle.bf16_bits_to_f64(dk[b, n:]) == 0.0)
        assert np.all(oracle.bf16_bits_to_f64(dv[b, n:]) == 0.0)
        if n == 0:
            assert np.all(oracle.bf16_bits_to_f64(dq[b]) == 0.0)


def _oracle_fwd_inputs(q, k, v, scale, lv):
    """o (bf16 bits) and lse (fp32) of the oracle's forward."""
    o, lse = oracle.attn_ref(q, k, v, scale, kv_valid_len=lv, workers=8)
    return oracle.f64_to_bf16_bits(o), np.where(np.isfinite(lse), lse, 0.0).astype(np.float32)


def _bwd_case(w, scale=None, lv="default"):
    """Backward kernels alone: o and lse come from the oracle's forward."""
    import torch

    q, k, v, lv0 = inputs.make_qkv(w)
    lv = lv0 if lv == "default" else lv
    do = inputs.make_dout(w)
    scale = w.scale if scale is None else scale
    log(f"case bwd {w.name} B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk} lv={None if lv is None else list(lv)} scale={scale}")
    dec = oracle.bf16_bits_to_f64
    ob, lse = _oracle_fwd_inputs(dec(q), dec(k), dec(v), scale, lv)
    dq, dk, dv = vx.attn_bwd(to_dev(q), to_dev(k), to_dev(v), to_dev(ob), to_dev(do),
                             torch.from_numpy(lse).cuda(), scale=scale, kv_valid_len=lengths_dev(lv))
    torch.cuda.synchronize()
    dq, dk, dv = to_bits(dq), to_bits(dk), to_bits(dv)
    # D from the same saved (bf16) output the kernels get
    rq, rk, rv = oracle.attn_bwd_ref(dec(q), dec(k), dec(v), dec(do), scale, kv_valid_len=lv, o_saved=dec(ob))
    kr = _key_rows(lv, w)
    _check_grad(dv, rv, "dv", kr)
    _check_grad(dk, rk, "dk", kr)
    _check_grad(dq, rq, "dq")
    _check_zeros(dq, dk, dv, lv, w.Lk)


BWD = [
    inputs.custom("bwd_tiny", B=1, H=2, Lq=512, Lk=512, seed=31),
    # several own-row tiles (256 rows) and streamed tiles (64 rows), ragged in both
    inputs.custom("bwd_ragged", B=2, H=3, Lq=1000, Lk=777, seed=32, kv_valid=("fixed", [777, 300])),
    # cross-attention shape: few keys, a batch without valid keys, a clamp above Lk
    inputs.custom("bwd_cross", B=3, H=2, Lq=600, Lk=512, seed=33, kv_valid=("fixed", [0, 37, 900])),
    inputs.custom("bwd_few", B=1, H=1, Lq=5, Lk=3, seed=34),
    inputs.custom("bwd_one", B=2, H=1, Lq=1, Lk=1, seed=35),
    inputs.custom("bwd_edges", B=1, H=2, Lq=257, Lk=65, seed=36),
    inputs.custom("bwd_normed", B=1, H=2, Lq=1536, Lk=1536, seed=37, rms_norm_qk=True),
    # few key workgroups and a long query stream: the key-side kernels cut the
    # 127 query tiles into 15 runs of 9 (fp32 partials summed afterwards), the
    # last run one tile; a batch with few valid keys
    inputs.custom("bwd_split", B=2, H=4, Lq=8100, Lk=300, seed=38, kv_valid=("fixed", [300, 45])),
]


@pytest.mark.parametrize("w", BWD, ids=lambda w: w.name)
def test_attn_bwd_matches_oracle(w):
    _bwd_case(w)


def _random_bwd_shapes(n=10, seed=2027):
    """Seeded random shapes: batches, heads, query and key counts off the
    256-row and 64-row tile grids, per-batch valid lengths from 0 to past Lk
    or none, raw or RMS-normalised q and k."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B, H = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        Lq, Lk = int(rng.integers(1, 900)), int(rng.integers(1, 900))
        kv = ("fixed", [int(x) for x in rng.integers(0, Lk + 50, B)]) if rng.random() < 0.5 else None
        cases.append(inputs.custom(f"bwd_random{i}", B=B, H=H, Lq=Lq, Lk=Lk, seed=200 + i, kv_valid=kv,
                                   rms_norm_qk=bool(rng.random() < 0.5)))
    return cases


@pytest.mark.parametrize("w", _random_bwd_shapes(), ids=lambda w: w.name)
def test_attn_bwd_random_shapes(w):
    _bwd_case(w)


@pytest.mark.parametrize("scale", [0.0, -0.05, 0.3])
def test_attn_bwd_scale_values(scale):
    _bwd_case(inputs.custom("bwd_scale", B=1, H=2, Lq=300, Lk=200, seed=38), scale=scale)


def test_attn_bwd_workspace_holds_d():
    """The first B * H * Lq values of the workspace hold D_i = <dO_i, O_i>
    ([B, H, Lq]) on return, also for a batch without valid keys and for the
    rows of a ragged last query tile: against the fp64 sum of the bf16
    products, within the fp32 accumulation error (129 roundings of partial
    sums bounded by sum |dO O|: 2^-17 of it)."""
    import torch

    w = [c for c in BWD if c.name == "bwd_cross"][0]
    q, k, v, lv = inputs.make_qkv(w)
    do = inputs.make_dout(w)
    log(f"case workspace D {w.name}")
    dec = oracle.bf16_bits_to_f64
    ob, lse = _oracle_fwd_inputs(dec(q), dec(k), dec(v), w.scale, lv)
    rows = w.B * w.H * w.Lq
    ws = torch.full((rows,), float("nan"), dtype=torch.float32, device="cuda")
    vx.attn_bwd(to_dev(q), to_dev(k), to_dev(v), to_dev(ob), to_dev(do), torch.from_numpy(lse).cuda(),
                scale=w.scale, kv_valid_len=lengths_dev(lv), workspace=ws)
    torch.cuda.synchronize()
    got = ws.cpu().numpy().astype(np.float64).reshape(w.B, w.H, w.Lq)
    prod = dec(do) * dec(ob)  # [B, Lq, H, d]
    ref = prod.sum(axis=3).transpose(0, 2, 1)
    bound = 2.0 ** -17 * np.abs(prod).sum(axis=3).transpose(0, 2, 1) + 1e-30
    assert np.isfinite(got).all()
    assert (np.abs(got - ref) <= bound).all(), float(np.max(np.abs(got - ref) / bound))


def test_attn_bwd_split_matches_unsplit():
    """The same call with a workspace that holds only D (no query-stream
    split) and with the size vidax_attn_bwd_workspace_floats asks for (split
    into runs): dq identical, dk and dv equal up to the order of the fp32 sums:
    one bf16 ulp of the larger magnitude, plus 2^-12 of the (batch, head)
    slice's RMS where a sum cancels to near zero (the summation-order error
    scales with the summands, not with the result); zeros exactly zero."""
    import torch

    w = [c for c in BWD if c.name == "bwd_split"][0]
    q, k, v, lv = inputs.make_qkv(w)
    do = inputs.make_dout(w)
    log(f"case split vs unsplit {w.name}")
    dev = [to_dev(x) for x in (q, k, v, do)]
    lvd = lengths_dev(lv)
    o, lse = vx.attn_fwd(dev[0], dev[1], dev[2], scale=w.scale, kv_valid_len=lvd, return_lse=True)
    n_split = vx.lib().vidax_attn_bwd_workspace_floats(w.B, w.H, w.Lq, w.Lk, w.d)
    rows = w.B * w.H * w.Lq
    assert n_split > rows  # this shape splits
    full = vx.attn_bwd(dev[0], dev[1], dev[2], o, dev[3], lse, scale=w.scale, kv_valid_len=lvd)
    ws = torch.empty((rows,), dtype=torch.float32, device="cuda")
    one = vx.attn_bwd(dev[0], dev[1], dev[2], o, dev[3], lse, scale=w.scale, kv_valid_len=lvd, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(full[0].view(torch.int16), one[0].view(torch.int16)), "dq"
    for name, a, b in zip(("dk", "dv"), full[1:], one[1:]):
        a, b = a.float(), b.float()
        assert bool(torch.isfinite(a).all()), name
        rms = torch.sqrt((a * a).mean(dim=(1, 3), keepdim=True))  # per (b, h)
        tol = 2.0 ** -7 * torch.maximum(a.abs(), b.abs()) + 2.0 ** -12 * rms
        excess = ((a - b).abs() - tol).max()
        assert bool(excess <= 0), (name, float((a - b).abs().max()), float(excess))
        assert bool(((a == 0) == (b == 0)).all()), name


def test_attn_bwd_batch_over_2gib():
    """One batch of k, v (and dk, dv) larger than 2 GiB: B=1, H=40, Lk=220000
    keys, 64 queries.  Element (n, h) of k sits at byte (n * 40 + h) * 256,
    past 2 GiB from key row 209716 on; the kernels rebase each 64-row tile
    with 64-bit pointers and keep 32-bit offsets inside it.  Checked against
    the oracle's exact gradient: dq of every query and dk, dv of key rows on
    both sides of the 2 GiB offset and at the end, for the first and last
    head (the largest offsets).  Inputs are seeded N(0, 1) drawn on the GPU
    (torch's generator) and copied back for the heads the oracle checks; the
    forward takes batches below 2 GiB only, so o and lse come from plain fp32
    attention on the GPU."""
    import torch

    B, H, Lq, Lk = 1, 40, 64, 220000
    g = torch.Generator(device="cuda")
    g.manual_seed(39)
    mk = lambda L: torch.randn((B, L, H, 128), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    q, k, v, do = mk(Lq), mk(Lk), mk(Lk), mk(Lq)
    assert k.numel() * 2 > 2 ** 31
    scale = float(np.float32(1 / np.sqrt(128)))
    log(f"case bwd over 2 GiB B{B} H{H} Lq{Lq} Lk{Lk}")
    # the forward takes batches below 2 GiB only: o and lse here are plain
    # fp32 softmax attention, one head at a time (an input of the backward;
    # the expected gradients come from the oracle alone)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, Lq), dtype=torch.float32, device="cuda")
    for h in range(H):
        sc = (q[0, :, h].float() @ k[0, :, h].float().T) * scale
        lse[0, h] = torch.logsumexp(sc, dim=1)
        o[0, :, h] = (torch.softmax(sc, dim=1) @ v[0, :, h].float()).to(torch.bfloat16)
    del sc
    dq, dk, dv = vx.attn_bwd(q, k, v, o, do, lse, scale=scale)
    torch.cuda.synchronize()
    hs = [0, H - 1]
    krows = np.array([0, 1, 4097, 100000, 209663, 209715, 209716, 209790, 215000, 219935, 219998, 219999])
    bits = lambda t: t[:, :, hs].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    dec = oracle.bf16_bits_to_f64
    qh, kh, vh, doh = (dec(bits(t)) for t in (q, k, v, do))
    got_dq = bits(dq)
    got_dk = dk[:, torch.from_numpy(krows).cuda()][:, :, hs].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    got_dv = dv[:, torch.from_numpy(krows).cuda()][:, :, hs].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    rq, rk, rv = oracle.attn_bwd_ref_rows(qh, kh, vh, doh, scale, np.arange(Lq), krows, workers=16)
    _check_grad(got_dq, rq, "dq, heads 0 and 39")
    _check_grad(got_dk, rk, "dk rows across 2 GiB")
    _check_grad(got_dv, rv, "dv rows across 2 GiB")


def test_attn_bwd_empty_calls():
    import torch

    for B, Lq, Lk in ((0, 64, 64), (1, 0, 64), (1, 64, 0)):
        z = lambda L: torch.zeros((B, L, 2, 128), dtype=torch.bfloat16, device="cuda")
        q, k = z(Lq), z(Lk)
        lse = torch.zeros((B, 2, Lq), dtype=torch.float32, device="cuda")
        dq, dk, dv = vx.attn_bwd(q, k, k.clone(), q.clone(), q.clone(), lse)
        torch.cuda.synchronize()
        assert dq.shape == q.shape and dk.shape == k.shape
    # Lk = 0 with queries present: no key, dq must still be written as zeros
    q = torch.ones((1, 70, 2, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((1, 0, 2, 128), dtype=torch.bfloat16, device="cuda")
    dq, _, _ = vx.attn_bwd(q, k, k.clone(), q.clone(), q.clone(),
                           torch.zeros((1, 2, 70), dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    assert torch.count_nonzero(dq).item() == 0


def _product_path(w, q, k, v, do, lv):
    """How a caller trains through the library: rotate, forward, backward,
    rotate the q/k gradients back."""
    import torch

    r = rope_of(w)
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    lvd = lengths_dev(lv)
    if r is not None:
        qd, kd = vx.rope3d(qd, r), vx.rope3d(kd, r)
    o, lse = vx.attn_fwd(qd, kd, vd, scale=w.scale, kv_valid_len=lvd, return_lse=True)
    dq, dk, dv = vx.attn_bwd(qd, kd, vd, o, to_dev(do), lse, scale=w.scale, kv_valid_len=lvd)
    if r is not None:
        dq, dk = vx.rope3d_transpose(dq, r), vx.rope3d_transpose(dk, r, out=dk)
    torch.cuda.synchronize()
    return to_bits(dq), to_bits(dk), to_bits(dv)


@pytest.mark.parametrize("w", [
    inputs.custom("bwd_rope_self", B=1, H=2, Lq=1000, Lk=1000, seed=41, grid=(2, 20, 24)),
    inputs.custom("bwd_rope_ragged", B=2, H=2, Lq=700, Lk=900, seed=42, grid=(1, 21, 30), kv_valid=("fixed", [900, 450])),
], ids=lambda w: w.name)
def test_rope_attention_gradient_end_to_end(w):
    q, k, v, lv = inputs.make_qkv(w)
    do = inputs.make_dout(w)
    log(f"case bwd+rope {w.name} B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk} grid={w.grid}")
    dq, dk, dv = _product_path(w, q, k, v, do, lv)
    dec = oracle.bf16_bits_to_f64
    spec = spec_of(w)
    qr, kr = oracle.rope3d_ref(dec(q), spec), oracle.rope3d_ref(dec(k), spec)
    gq, gk, gv = oracle.attn_bwd_ref(qr, kr, dec(v), dec(do), w.scale, kv_valid_len=lv)
    rq, rk = oracle.rope_transpose_ref(gq, spec), oracle.rope_transpose_ref(gk, spec)
    kr = _key_rows(lv, w)
    _check_grad(dv, gv, "dv", kr)
    _check_grad(dk, rk, "dk", kr)
    _check_grad(dq, rq, "dq")
    _check_zeros(dq, dk, dv, lv, w.Lk)


@pytest.mark.parametrize("mode", [0, 1])
def test_rope3d_transpose_matches_oracle(mode):
    import torch

    from tests.test_gpu_parity import _rope_bound

    grid = (3, 10, 30)  # 900 video tokens, then 100 unrotated tokens
    x = inputs.bf16_tensor(12, 0, (2, 1000, 3, 128))
    log(f"case rope3d_transpose mode={mode}")
    r = vx.Rope(grid=grid, dims=(44, 42, 42), theta=10000.0, pair_mode=mode)
    y = vx.rope3d_transpose(to_dev(x), r)
    torch.cuda.synchronize()
    spec = oracle.RopeSpec(grid=grid, pair_mode=mode)
    xf = oracle.bf16_bits_to_f64(x)
    ref = oracle.rope_transpose_ref(xf, spec)
    err = np.abs(oracle.bf16_bits_to_f64(to_bits(y)) - ref)
    bound = _rope_bound(xf, ref, spec, np.arange(x.shape[1]))
    assert np.all(err <= bound), (err.max(), float((err / bound).max()))
    assert np.array_equal(to_bits(y)[:, 900:], x[:, 900:])


# ------------------------------------------------------------ full size ---

def _edge_rows(L, rng, n=64):
    return np.unique(np.r_[0, 1, 63, 64, 255, 256, L - 257, L - 256, L - 65, L - 64, L - 1,
                           rng.integers(0, L, n)].clip(0, L - 1))


@pytest.mark.parametrize("name,dkv_heads", [("wan13b_480p", [5]), ("cross_text", [0, 39])])
def test_attn_bwd_full_size_sampled(name, dkv_heads):
    """The benchmark's shape, sampled rows against the oracle's exact gradient
    (D from the exact output): dq rows of every head (each needs only its own
    row of P), dk/dv rows of a few heads (each needs the lse and D of every
    query, a full forward of that head in the oracle)."""
    import torch

    w = inputs.WORKLOADS[name]
    q, k, v, lv = inputs.make_qkv(w)
    do = inputs.make_dout(w)
    log(f"case bwd full {name} B{w.B} H{w.H} Lq{w.Lq} Lk{w.Lk}")
    qd, kd, vd, lvd = to_dev(q), to_dev(k), to_dev(v), lengths_dev(lv)
    o, lse = vx.attn_fwd(qd, kd, vd, scale=w.scale, kv_valid_len=lvd, return_lse=True)
    dq, dk, dv = vx.attn_bwd(qd, kd, vd, o, to_dev(do), lse, scale=w.scale, kv_valid_len=lvd)
    torch.cuda.synchronize()
    del o, lse, qd, kd, vd
    dq, dk, dv = to_bits(dq), to_bits(dk), to_bits(dv)
    dec = oracle.bf16_bits_to_f64
    rng = np.random.default_rng(7)
    qrows, krows = _edge_rows(w.Lq, rng), _edge_rows(w.Lk, rng)
    # dq rows of every head: rows are independent, so the oracle gets only them
    nr = len(qrows)
    rq, _, _ = oracle.attn_bwd_ref_rows(dec(q[:, qrows]), dec(k), dec(v), dec(do[:, qrows]), w.scale,
                                        np.arange(nr), [], kv_valid_len=lv, workers=16)
    _check_grad(dq[:, qrows], rq, "dq, every head")
    # dk/dv rows of a few heads
    hs = dkv_heads
    _, rk, rv = oracle.attn_bwd_ref_rows(dec(q[:, :, hs]), dec(k[:, :, hs]), dec(v[:, :, hs]), dec(do[:, :, hs]),
                                         w.scale, [], krows, kv_valid_len=lv, workers=16)
    # krows is sorted: the valid keys of batch b are its first n[b] entries
    n = None if lv is None else np.array([np.sum(krows < min(max(x, 0), w.Lk)) for x in lv])
    _check_grad(dv[:, krows][:, :, hs], rv, f"dv heads {hs}", n)
    _check_grad(dk[:, krows][:, :, hs], rk, f"dk heads {hs}", n)
    for g in (dq, dk, dv):
        assert np.all(np.isfinite(dec(g)))
    _check_zeros(dq, dk, dv, lv, w.Lk)
