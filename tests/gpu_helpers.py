"""Shared helpers of the GPU parity tests (imported by tests only)."""

from __future__ import annotations

import numpy as np

from oracle import attention as oatt
from oracle import kvpool as okv

MAX_ABS = 1e-2   # attention tolerance vs the fp64 oracle: bf16 in, fp32 accumulate, bf16 out
MEAN_ABS = 1e-3


def bits(t) -> np.ndarray:
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_to_f64(b):
    return oatt.bf16_to_f64(b)


def compare(gpu_out_bits: np.ndarray, ref: np.ndarray, what: str = ""):
    """gpu bf16 bits vs oracle fp64 (NaN in ref = not computed / not compared)."""
    got = bf16_to_f64(gpu_out_bits)
    sel = ~np.isnan(ref)
    assert sel.any(), "nothing compared"
    assert np.isfinite(got[sel]).all(), f"{what}: non-finite GPU output"
    err = np.abs(got[sel] - ref[sel])
    mx, mean = float(err.max()), float(err.mean())
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: max abs {mx:.3g}, mean abs {mean:.3g}"
    return mx, mean


def oracle_tables(plan_tables):
    return [list(r) for r in plan_tables]


def print_case(msg: str):
    print(f"[case] {msg}", flush=True)


def sample_rows(S: int, rng, n_random: int = 48):
    """First/last suffix rows, tile-boundary rows and random rows of a request's suffix."""
    rows = {0, S - 1}
    bounds = np.arange(0, S, 64)
    for b in rng.choice(bounds, min(8, len(bounds)), replace=False):
        rows.update({int(b), min(S - 1, int(b) + 63)})
    rows.update(rng.integers(0, S, min(n_random, S)).tolist())
    return sorted(r for r in rows if 0 <= r < S)


def oracle_scatter(kp, vp, k_bits, v_bits, slots):
    okv.scatter(kp, vp, k_bits, v_bits, slots)
