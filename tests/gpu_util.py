"""Helpers shared by the GPU parity tests (device transfer, error metrics)."""

from __future__ import annotations

import sys

import numpy as np

import oracle
from paper_2609_18077_amd import inputs

# Parity contract for bf16 in / bf16 out attention with fp32 accumulation.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3
# Internal guard: relative RMS error against the oracle.
REL_RMS = 1e-2
# Natural-log sum-exp, absolute.
LSE_ABS = 2e-2


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def to_dev(bits: np.ndarray):
    import torch

    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def to_bits(t) -> np.ndarray:
    import torch

    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def lengths_dev(lv):
    import torch

    if lv is None:
        return None
    return torch.from_numpy(np.asarray(lv, dtype=np.int32)).cuda()


def spec_of(w: inputs.Workload):
    if w.grid is None:
        return None
    return oracle.RopeSpec(grid=w.grid, dims=w.dims, theta=w.theta, pair_mode=0)


def rope_of(w: inputs.Workload):
    import paper_2609_18077_amd as vx

    if w.grid is None:
        return None
    return vx.Rope(grid=w.grid, dims=w.dims, theta=w.theta, pair_mode=0)


def errors(got_bits: np.ndarray, ref: np.ndarray):
    got = oracle.bf16_bits_to_f64(got_bits)
    diff = np.abs(got - ref)
    rms_ref = np.sqrt(np.mean(ref * ref))
    return {
        "max_abs": float(diff.max()) if diff.size else 0.0,
        "mean_abs": float(diff.mean()) if diff.size else 0.0,
        "rel_rms": float(np.sqrt(np.mean(diff * diff)) / rms_ref) if rms_ref > 0 else float(np.sqrt(np.mean(diff * diff))),
    }


def assert_parity(got_bits, ref, what=""):
    e = errors(got_bits, ref)
    log(f"  parity {what}: {e}")
    assert np.all(np.isfinite(oracle.bf16_bits_to_f64(got_bits))), what
    assert e["max_abs"] <= MAX_ABS, (what, e)
    assert e["mean_abs"] <= MEAN_ABS, (what, e)
    assert e["rel_rms"] <= REL_RMS, (what, e)
    return e


def assert_lse(got, ref, what=""):
    got = np.asarray(got, np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(got)), what
    assert np.all(np.isneginf(got[~fin])), what
    if fin.any():
        err = np.abs(got[fin] - ref[fin]).max()
        log(f"  lse {what}: max_abs {err:.3e}")
        assert err <= LSE_ABS, (what, err)
