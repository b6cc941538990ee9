"""Non-causal scaled dot-product attention, float64 reference (test infrastructure only).

What is computed (paper Section 2: flash-attention dispatch for the unmasked
attention ops, which avoids materialising the query-key matrix but computes the
same softmax attention; Appendix table of porting bugs, "Sharding, Parallelism &
Custom Kernels": padded keys are skipped per sequence instead of via a dense
mask).  For batch b, head h, query i:

    s_ij  = scale * <q~_i, k~_j>              for keys j < Lv_b
    m_i   = max_j s_ij
    o_i   = sum_j exp(s_ij - m_i) v_j / sum_j exp(s_ij - m_i)
    lse_i = m_i + ln sum_j exp(s_ij - m_i)

where q~, k~ are the 3D-rotated queries/keys when a rotary spec is given, and
Lv_b = clamp(kv_valid_len[b], 0, Lk).  Every query sees the same key prefix
[0, Lv_b); with Lv_b = 0 the output row is 0 and lse is -inf.

The softmax is evaluated in two passes per block of query rows (row max, then
exponentials and sums) over all valid keys at once -- deliberately not the
online/streaming form used by the GPU kernel.
"""

from __future__ import annotations

import concurrent.futures as cf

import numpy as np

from .rope3d import RopeSpec, rope3d_ref


def _valid_lengths(kv_valid_len, B: int, Lk: int) -> np.ndarray:
    if kv_valid_len is None:
        return np.full(B, Lk, dtype=np.int64)
    lv = np.asarray(kv_valid_len, dtype=np.int64).reshape(B)
    return np.clip(lv, 0, Lk)


def _one_block(qb, kb, vb, scale):
    """Two-pass softmax attention of query rows qb [R, d] over keys kb/vb [N, d]."""
    s = scale * (qb @ kb.T)  # [R, N]
    m = s.max(axis=1)
    e = np.exp(s - m[:, None])
    l = e.sum(axis=1)
    o = (e @ vb) / l[:, None]
    lse = m + np.log(l)
    return o, lse


def attn_ref(q, k, v, scale, kv_valid_len=None, rope: RopeSpec | None = None,
             q_token_index=None, block: int = 256, workers: int = 1):
    """Reference attention.

    q: [B, Lq, H, d], k/v: [B, Lk, H, d] float64 (already decoded from bf16).
    q_token_index: token index of each query row (default 0..Lq-1); keys are
    always tokens 0..Lk-1.  Returns (o [B, Lq, H, d], lse [B, H, Lq]) float64.
    workers > 1 evaluates independent (b, h, query-block) jobs in a thread pool
    (the arithmetic of each job is unchanged).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, Lq, H, d = q.shape
    Lk = k.shape[1]
    if rope is not None:
        q = rope3d_ref(q, rope, token_index=q_token_index)
        k = rope3d_ref(k, rope)
    lv = _valid_lengths(kv_valid_len, B, Lk)
    o = np.zeros((B, Lq, H, d), np.float64)
    lse = np.full((B, H, Lq), -np.inf, np.float64)
    scale = float(scale)

    jobs = []
    for b in range(B):
        if lv[b] == 0:
            continue
        for h in range(H):
            for r0 in range(0, Lq, block):
                jobs.append((b, h, r0, min(Lq, r0 + block)))

    kh = {}

    def keys(b, h):
        if (b, h) not in kh:
            n = lv[b]
            kh[(b, h)] = (np.ascontiguousarray(k[b, :n, h, :]), np.ascontiguousarray(v[b, :n, h, :]))
        return kh[(b, h)]

    def run(job):
        b, h, r0, r1 = job
        kb, vb = keys(b, h)
        ob, lb = _one_block(q[b, r0:r1, h, :], kb, vb, scale)
        o[b, r0:r1, h, :] = ob
        lse[b, h, r0:r1] = lb

    if workers <= 1:
        for j in jobs:
            run(j)
    else:
        # materialise per-(b, h) key/value copies before the pool starts
        for b in range(B):
            if lv[b]:
                for h in range(H):
                    keys(b, h)
        with cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(run, jobs))
    return o, lse


def attn_ref_rows(q, k, v, scale, rows, kv_valid_len=None, rope: RopeSpec | None = None,
                  workers: int = 1):
    """Reference attention for selected query rows only.

    rows: int array of query indices (token indices of q's axis 1).  Rows are
    independent in attention, so each sampled row is exact.  Returns
    (o [B, R, H, d], lse [B, H, R]).
    """
    rows = np.asarray(rows, dtype=np.int64)
    qs = np.asarray(q)[:, rows]
    return attn_ref(qs, k, v, scale, kv_valid_len=kv_valid_len, rope=rope,
                    q_token_index=rows, workers=workers)
