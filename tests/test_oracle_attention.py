"""Pins of the oracle's fp64 prefix-cached prefill attention (CPU only)."""

import math

import numpy as np
import pytest
import torch

from oracle import attention as att
from oracle import kvpool


def rand_bf16_bits(rng, shape, sd=1.0):
    x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32) * sd)
    return x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def paged_case(rng, L, P, hq, hkv, d, n_phys=None, sd=1.0):
    """One request: full-sequence bits, a pool holding it at a random placement, block table."""
    nb = (L + 15) // 16
    n_phys = n_phys or nb + 5
    q = rand_bf16_bits(rng, (L, hq, d), sd)
    k = rand_bf16_bits(rng, (L, hkv, d), sd)
    v = rand_bf16_bits(rng, (L, hkv, d), sd)
    table = [int(x) for x in rng.permutation(n_phys)[:nb]]
    kp, vp = kvpool.new_pool(n_phys, hkv, d)
    kvpool.scatter(kp, vp, k, v, [table[j // 16] * 16 + j % 16 for j in range(L)])
    return q, k, v, kp, vp, table


def brute(qf, kf, vf, P, scale):
    """Scalar triple loop with math.exp, no vectorisation (S x Hq x D)."""
    S, hq, d = qf.shape
    g = hq // kf.shape[1]
    out = np.zeros((S, hq, d))
    for i in range(S):
        j = P + i
        for h in range(hq):
            kh = h // g
            s = [scale * sum(qf[i, h, x] * kf[t, kh, x] for x in range(d)) for t in range(j + 1)]
            m = max(s)
            w = [math.exp(x - m) for x in s]
            z = sum(w)
            for x in range(d):
                out[i, h, x] = sum(w[t] * vf[t, kh, x] for t in range(j + 1)) / z
    return out


@pytest.mark.parametrize("L,P,hq,hkv,d", [(1, 0, 2, 1, 4), (20, 16, 4, 2, 8), (37, 32, 2, 2, 6),
                                          (48, 0, 4, 1, 4), (80, 64, 8, 2, 4)])
def test_against_brute_force(L, P, hq, hkv, d):
    rng = np.random.default_rng(L * 7 + P)
    q, k, v, kp, vp, table = paged_case(rng, L, P, hq, hkv, d)
    scale = d ** -0.5
    o = att.prefill_attention(q[P:], kp, vp, [table], [0, L - P], [L], scale)
    ref = brute(att.bf16_to_f64(q[P:]), att.bf16_to_f64(k), att.bf16_to_f64(v), P, scale)
    assert np.max(np.abs(o - ref)) < 1e-12


def test_single_token_returns_its_value():
    rng = np.random.default_rng(3)
    q, k, v, kp, vp, table = paged_case(rng, 1, 0, 4, 2, 16)
    o = att.prefill_attention(q, kp, vp, [table], [0, 1], [1], 0.25)
    vf = att.bf16_to_f64(v)
    assert np.array_equal(o[0, :2], vf[0, [0, 0]]) and np.array_equal(o[0, 2:], vf[0, [1, 1]])


def test_equal_keys_average_values_and_dominant_key_selects_value():
    rng = np.random.default_rng(4)
    L, d = 40, 8
    q = rand_bf16_bits(rng, (L, 1, d))
    k = np.repeat(rand_bf16_bits(rng, (1, 1, d)), L, axis=0)
    v = rand_bf16_bits(rng, (L, 1, d))
    vf = att.bf16_to_f64(v)
    o = att.request_attention(q[24:], k, v, 24, 0.5)
    for i in range(16):
        assert np.allclose(o[i, 0], vf[: 24 + i + 1, 0].mean(axis=0), atol=1e-13)
    # one key aligned with the query by a margin of >= 60 in the score dominates
    k2 = np.zeros((L, 1, d), dtype=np.uint16)
    q2 = np.zeros((L, 1, d), dtype=np.uint16)
    q2[:, 0, 0] = 0x4100                      # 8.0
    k2[5, 0, 0] = 0x4100                      # score 64 * scale(1) vs 0 elsewhere
    o2 = att.request_attention(q2[20:], k2, v, 20, 1.0)
    # every other weight is exp(-64) < 1.7e-28; at most 40 keys with |v| < 10 each
    assert np.max(np.abs(o2[:, 0] - vf[5, 0])) < 40 * 1.7e-28 * 20


def test_gqa_equals_mha_with_repeated_kv_heads():
    rng = np.random.default_rng(5)
    L, P, hq, hkv, d = 50, 32, 8, 2, 8
    q, k, v, *_ = paged_case(rng, L, P, hq, hkv, d)
    o = att.request_attention(q[P:], k, v, P, 0.3)
    o_mha = att.request_attention(q[P:], np.repeat(k, 4, axis=1), np.repeat(v, 4, axis=1), P, 0.3)
    assert np.array_equal(o, o_mha)


def test_matches_torch_sdpa_with_explicit_bottom_right_mask():
    rng = np.random.default_rng(6)
    L, P, hq, hkv, d = 150, 96, 8, 2, 32
    q, k, v, kp, vp, table = paged_case(rng, L, P, hq, hkv, d)
    scale = d ** -0.5
    o = att.prefill_attention(q[P:], kp, vp, [table], [0, L - P], [L], scale)
    S = L - P
    qt = torch.from_numpy(att.bf16_to_f64(q[P:])).permute(1, 0, 2)           # [Hq, S, D]
    kt = torch.from_numpy(att.bf16_to_f64(k)).repeat_interleave(hq // hkv, 1).permute(1, 0, 2)
    vt = torch.from_numpy(att.bf16_to_f64(v)).repeat_interleave(hq // hkv, 1).permute(1, 0, 2)
    mask = torch.arange(L)[None, :] <= (P + torch.arange(S))[:, None]           # bottom-right
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    assert np.max(np.abs(o - ref.permute(1, 0, 2).numpy())) < 1e-12


def test_prefix_cached_equals_full_recompute():
    # Output of the uncached suffix == last S rows of dense causal attention over the
    # whole (non-paged) sequence: reusing cached prefix KV changes nothing (Sec. 2).
    rng = np.random.default_rng(8)
    L, P, hq, hkv, d = 200, 128, 4, 2, 16
    q, k, v, kp, vp, table = paged_case(rng, L, P, hq, hkv, d)
    scale = d ** -0.5
    o = att.prefill_attention(q[P:], kp, vp, [table], [0, L - P], [L], scale)
    qf, kf, vf = (att.bf16_to_f64(x) for x in (q, k, v))
    dense = np.zeros((L, hq, d))
    for h in range(hq):
        s = scale * qf[:, h] @ kf[:, h // 2].T
        s[np.triu_indices(L, 1)] = -np.inf
        w = np.exp(s - s.max(1, keepdims=True))
        dense[:, h] = (w / w.sum(1, keepdims=True)) @ vf[:, h // 2]
    assert np.max(np.abs(o - dense[P:])) < 1e-12


def test_block_table_permutation_is_bitwise_invariant():
    rng = np.random.default_rng(9)
    L, P, hq, hkv, d = 130, 64, 4, 2, 16
    q, k, v, kp, vp, table = paged_case(rng, L, P, hq, hkv, d, n_phys=20)
    o1 = att.prefill_attention(q[P:], kp, vp, [table], [0, L - P], [L], 0.25)
    table2 = [int(x) for x in rng.permutation(20)[: len(table)]]
    kp2, vp2 = kvpool.new_pool(20, hkv, d)
    kvpool.scatter(kp2, vp2, k, v, [table2[j // 16] * 16 + j % 16 for j in range(L)])
    o2 = att.prefill_attention(q[P:], kp2, vp2, [table2], [0, L - P], [L], 0.25)
    assert np.array_equal(o1, o2)


def test_row_sampling_matches_full():
    rng = np.random.default_rng(10)
    L, P, hq, hkv, d = 300, 200, 4, 1, 8
    q, k, v, kp, vp, table = paged_case(rng, L, P, hq, hkv, d)
    full = att.prefill_attention(q[P:], kp, vp, [table], [0, L - P], [L], 0.3)
    rows = [0, 15, 16, 63, 99]
    part = att.prefill_attention(q[P:], kp, vp, [table], [0, L - P], [L], 0.3, rows_per_request=[rows])
    assert np.array_equal(part[rows], full[rows])
    assert np.isnan(part[1]).all()


def test_dominant_key_beyond_the_exponential_range():
    # A score of 6400 is far past exp's fp64 range (overflow above ~709.8); softmax is
    # shift-invariant, so the output is still exactly that key's value: every other weight
    # is exp(-6400) = 0.
    rng = np.random.default_rng(14)
    L, d = 24, 8
    v = rand_bf16_bits(rng, (L, 1, d))
    k = np.zeros((L, 1, d), dtype=np.uint16)
    q = np.zeros((L, 1, d), dtype=np.uint16)
    q[:, 0, 0] = 0x4100                       # 8.0
    k[3, 0, 0] = 0x4100
    o = att.request_attention(q[8:], k, v, 8, 100.0)
    assert np.array_equal(o[:, 0], np.repeat(att.bf16_to_f64(v)[3:4, 0], L - 8, axis=0))
