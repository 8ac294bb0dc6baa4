"""Prefix-cached prefill attention in fp64 (oracle).  TEST INFRASTRUCTURE ONLY.

During prefill the model runs the whole prompt through one forward pass; with
prefix caching only the tokens after the cached prefix are computed, and they
attend to the reused prefix KV as well as to each other (Sec. 2, "LLM
Serving").  For one request with L prompt tokens of which the first P are
cached, every computed query position j in [P, L) and query head h sees the
keys 0..j of KV head h // g (g = query heads per KV head):

    s_t = scale * <q_{j,h}, k_{t, h//g}>            t = 0..j
    o_{j,h} = sum_t softmax(s)_t * v_{t, h//g}

Readings fixed by this project (the paper gives no attention details): no
positional terms are applied here (inputs are taken as already rotated), the
causal alignment is bottom-right (suffix row j sees keys 0..j), scale is the
caller's value (1/sqrt(head_dim) in every workload).

Inputs are bf16 bit patterns (uint16); all arithmetic is IEEE binary64, so
every product of two bf16 values is exact.  The K/V of a request are first
gathered into contiguous arrays through the block table (``kvpool.gather``);
the attention itself is then the plain definition above.
"""

from __future__ import annotations

import numpy as np

from . import kvpool


def bf16_to_f64(bits) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def causal_rows(q, k, v, positions, scale: float) -> np.ndarray:
    """Attention of query rows at absolute ``positions`` over keys 0..position.

    q: [R, D] float64, k, v: [L, D] float64 (one head), positions: [R] ints.
    """
    positions = np.asarray(positions, dtype=np.int64)
    L = k.shape[0]
    s = scale * (q @ k.T)                                  # [R, L]
    visible = np.arange(L)[None, :] <= positions[:, None]
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    w = np.exp(s - m)
    w = w / w.sum(axis=1, keepdims=True)
    return w @ v


def request_attention(q_bits, k_bits, v_bits, prefix_len: int, scale: float,
                      rows=None, chunk: int = 256) -> np.ndarray:
    """One request: q [S, Hq, D], gathered k/v [L, Hkv, D] (bf16 bits) -> o [S, Hq, D] fp64.

    ``rows`` optionally selects suffix rows (indices into S); others are left as NaN.
    """
    S, hq, d = q_bits.shape
    L, hkv, _ = k_bits.shape
    assert L == prefix_len + S and hq % hkv == 0
    g = hq // hkv
    k = bf16_to_f64(k_bits)
    v = bf16_to_f64(v_bits)
    out = np.full((S, hq, d), np.nan)
    sel = np.arange(S) if rows is None else np.asarray(rows, dtype=np.int64)
    for c0 in range(0, len(sel), chunk):
        rs = sel[c0:c0 + chunk]
        pos = prefix_len + rs
        hi = int(pos.max()) + 1                      # keys beyond the last row are all masked
        qf = bf16_to_f64(q_bits[rs])                 # [R, Hq, D]
        for h in range(hq):
            kh = h // g
            out[rs, h, :] = causal_rows(qf[:, h, :], k[:hi, kh, :], v[:hi, kh, :], pos, scale)
    return out


def prefill_attention(q_bits, k_pool, v_pool, block_tables, cu_q, seq_lens, scale: float,
                      rows_per_request=None) -> np.ndarray:
    """Whole batch: q [sum S, Hq, D] (bf16 bits) through the pool -> o [sum S, Hq, D] fp64."""
    out = np.full(q_bits.shape, np.nan)
    for r in range(len(seq_lens)):
        q0, q1 = int(cu_q[r]), int(cu_q[r + 1])
        L = int(seq_lens[r])
        P = L - (q1 - q0)
        k, v = kvpool.gather(k_pool, v_pool, block_tables[r], L)
        rows = None if rows_per_request is None else rows_per_request[r]
        out[q0:q1] = request_attention(q_bits[q0:q1], k, v, P, scale, rows=rows)
    return out
