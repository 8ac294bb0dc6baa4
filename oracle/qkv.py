"""Query/key/value projection with rotary position embedding (oracle).  TEST INFRASTRUCTURE ONLY.

Sec. 4 serves Qwen3-14B: in a prefill, every computed (uncached) token's hidden state goes
through each layer's query/key/value projection, and queries and keys get rotary position
embedding at the token's absolute position, before attention reads them (the cached prefix's
keys and values were produced the same way when they were computed).  The paper gives no
layer details; this project's reading (following the public Qwen3-14B configuration, not the
paper) is:

1. y = x W^T with x the [T, H] bf16 hidden states and W the [(Hq + 2 Hkv) D, H] bf16 weight
   (rows: the Hq query heads, then the Hkv key heads, then the Hkv value heads, D each);
   y is accumulated in IEEE binary64 (every product of two bf16 values is exact), rounded to
   fp32 and then to bf16, nearest even (bf16 activations accumulated at fp32 or better);
2. rotary embedding, rotate-half pairing, of every query and key head at the token's
   position p: for i < D/2 with frequency f_i = theta^(-2 i / D) and angle a = p f_i,
       out[i]       = u[i] cos a - u[i + D/2] sin a
       out[i + D/2] = u[i + D/2] cos a + u[i] sin a
   in IEEE binary64; values pass through unchanged;
3. q, k, v rounded to bf16 (fp64 -> fp32 -> bf16, round to nearest even each time).

No query/key normalisation or bias is applied (outside this reading).
"""

from __future__ import annotations

import numpy as np

from .attention import bf16_to_f64


def f64_to_bf16_bits(x) -> np.ndarray:
    """float64 -> bf16 bit patterns: to fp32 (nearest even), then to bf16 (nearest even)."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def project(x_bits, w_bits) -> np.ndarray:
    """Step 1 before rounding: y = x W^T in fp64 ([T, H] x [N, H] -> [T, N])."""
    x = bf16_to_f64(x_bits)
    w = bf16_to_f64(w_bits)
    return x @ w.T


def rope(u, positions, theta: float) -> np.ndarray:
    """Step 2 for one set of heads: u [T, heads, D] fp64, positions [T] -> rotated copy."""
    u = np.asarray(u, dtype=np.float64)
    d = u.shape[-1]
    half = d // 2
    f = theta ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    a = np.asarray(positions, dtype=np.float64)[:, None] * f[None, :]     # [T, D/2]
    c, s = np.cos(a)[:, None, :], np.sin(a)[:, None, :]
    lo, hi = u[..., :half], u[..., half:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def qkv_rope(x_bits, w_bits, positions, num_q_heads: int, num_kv_heads: int, head_dim: int,
             theta: float):
    """Steps 1-3: returns (q, k, v) as bf16 bits [T, heads, D] and, for tolerance checks,
    the fp64 values they were rounded from."""
    t = np.asarray(x_bits).shape[0]
    y = bf16_to_f64(f64_to_bf16_bits(project(x_bits, w_bits)))
    nq, nk = num_q_heads * head_dim, num_kv_heads * head_dim
    q = rope(y[:, :nq].reshape(t, num_q_heads, head_dim), positions, theta)
    k = rope(y[:, nq:nq + nk].reshape(t, num_kv_heads, head_dim), positions, theta)
    v = y[:, nq + nk:nq + 2 * nk].reshape(t, num_kv_heads, head_dim)
    exact = (q, k, v)
    return tuple(f64_to_bf16_bits(a) for a in exact), exact


def token_positions(cu_q, seq_lens) -> np.ndarray:
    """Absolute position of every computed token: request r's S_r tokens sit at
    L_r - S_r .. L_r - 1 (the suffix after its cached prefix)."""
    out = []
    for r in range(len(seq_lens)):
        s = int(cu_q[r + 1]) - int(cu_q[r])
        out.append(np.arange(int(seq_lens[r]) - s, int(seq_lens[r])))
    return np.concatenate(out) if out else np.zeros(0, dtype=np.int64)
