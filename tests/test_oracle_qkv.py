"""Pins of the QKV projection + rotary embedding oracle (CPU only).

Each check rests on something other than the oracle's own formula: the bf16 format's
rounding of hand-picked values, a brute-force triple loop, rotation-group identities
(position 0 is the identity, rotations compose, norms and relative-position dot products are
preserved), and the rotary pairs written as complex numbers multiplied by e^{i p f}.
"""

import numpy as np
import pytest

from oracle import qkv
from oracle.attention import bf16_to_f64


def bits(x):
    return qkv.f64_to_bf16_bits(np.asarray(x, dtype=np.float64))


def test_bf16_rounding_of_hand_picked_values():
    # bf16 keeps 7 fraction bits: 1 + 2^-8 is the tie between 1 and 1 + 2^-7 (even: 1),
    # 1 + 3 * 2^-8 the tie between 1 + 2^-7 and 1 + 2^-6 (even: 1 + 2^-6)
    assert bits([1.0, -2.0, 0.0])[:].tolist() == [0x3F80, 0xC000, 0x0000]
    assert int(bits(1 + 2 ** -8)) == 0x3F80
    assert int(bits(1 + 3 * 2 ** -8)) == 0x3F82
    assert int(bits(1 + 2 ** -8 + 2 ** -20)) == 0x3F81          # above the tie: up
    x = np.random.default_rng(0).standard_normal(1000)
    err = np.abs(bf16_to_f64(bits(x)) - x)
    assert (err <= np.abs(x) * 2 ** -8 + 1e-300).all()        # half an ulp of 7 fraction bits


def test_projection_equals_brute_force():
    rng = np.random.default_rng(1)
    x = bits(rng.standard_normal((3, 5)))
    w = bits(rng.standard_normal((4, 5)))
    xf, wf = bf16_to_f64(x), bf16_to_f64(w)
    want = np.zeros((3, 4))
    for t in range(3):
        for n in range(4):
            for h in range(5):
                want[t, n] += xf[t, h] * wf[n, h]
    assert np.allclose(qkv.project(x, w), want, rtol=0, atol=1e-12)


def test_rope_is_a_rotation_by_p_times_frequency():
    rng = np.random.default_rng(2)
    d, theta = 16, 10000.0
    u = rng.standard_normal((5, 3, d))
    pos = np.array([0, 1, 7, 1000, 32767])
    out = qkv.rope(u, pos, theta)
    # position 0 is the identity
    assert np.array_equal(out[0], u[0])
    # the pair (i, i + d/2) as a complex number turns by p * theta^(-2i/d)
    z = u[..., : d // 2] + 1j * u[..., d // 2:]
    f = np.array([theta ** (-2.0 * i / d) for i in range(d // 2)])
    want = z * np.exp(1j * pos[:, None, None] * f[None, None, :])
    got = out[..., : d // 2] + 1j * out[..., d // 2:]
    assert np.allclose(got, want, rtol=0, atol=1e-9)
    # pair norms are preserved
    assert np.allclose(np.abs(got), np.abs(z), rtol=0, atol=1e-12)


def test_rope_composes_and_keeps_relative_positions():
    rng = np.random.default_rng(3)
    d, theta = 128, 1.0e6
    q = rng.standard_normal((1, 1, d))
    k = rng.standard_normal((1, 1, d))
    for m, n, s in [(5, 3, 100), (0, 40000, 7), (1234, 1234, 999)]:
        a = np.sum(qkv.rope(q, [m], theta) * qkv.rope(k, [n], theta))
        b = np.sum(qkv.rope(q, [m + s], theta) * qkv.rope(k, [n + s], theta))
        assert abs(a - b) < 1e-9 * (1 + abs(a))
    # rotating by a then by b is rotating by a + b
    two = qkv.rope(qkv.rope(q, [300], theta), [45], theta)
    assert np.allclose(two, qkv.rope(q, [345], theta), rtol=0, atol=1e-9)


def test_head_split_and_value_pass_through():
    # one-hot weight rows: y column n picks hidden unit sel[n]; at position 0 every head is
    # the picked values themselves (q, k, v alike), rounded to bf16
    rng = np.random.default_rng(4)
    hq, hkv, d, h = 4, 2, 8, 20
    n = (hq + 2 * hkv) * d
    sel = rng.integers(0, h, n)
    w = np.zeros((n, h))
    w[np.arange(n), sel] = 1.0
    x = bits(rng.standard_normal((3, h)))
    (qb, kb, vb), _ = qkv.qkv_rope(x, bits(w), [0, 0, 0], hq, hkv, d, 1.0e6)
    picked = x[:, sel]
    assert np.array_equal(qb.reshape(3, -1), picked[:, : hq * d])
    assert np.array_equal(kb.reshape(3, -1), picked[:, hq * d:(hq + hkv) * d])
    assert np.array_equal(vb.reshape(3, -1), picked[:, (hq + hkv) * d:])
    # away from position 0 values stay, queries and keys turn
    (qb2, kb2, vb2), _ = qkv.qkv_rope(x, bits(w), [5, 6, 7], hq, hkv, d, 1.0e6)
    assert np.array_equal(vb2, vb) and not np.array_equal(qb2, qb)


def test_token_positions_follow_the_suffixes():
    assert qkv.token_positions([0, 3, 3, 5], [10, 4, 2]).tolist() == [7, 8, 9, 0, 1]


def test_projection_is_rounded_to_bf16_before_the_rotation():
    # Worked by hand, one query head of two dims (f_0 = 1) at position 1: x = [1, 2^-8],
    # query row 0 of W = [1, 1] gives y = 1 + 2^-8, the tie that bf16 rounds to 1.0.  The
    # rotated pair is (y cos 1, y sin 1): from the rounded y that is (0.540302..., 0.841470...)
    # -> bf16 1.078125 / 2 (0x3F0A) and 1.6796875 / 2 (0x3F57); the unrounded y would give
    # 0.542413... and 0.844758... -> 0x3F0B and 0x3F58.
    x = np.array([[0x3F80, 0x3B80]], dtype=np.uint16)           # 1.0, 2^-8
    w = np.zeros((6, 2), dtype=np.uint16)                       # rows: q0 q1 | k0 k1 | v0 v1
    w[0] = [0x3F80, 0x3F80]
    (q, k, v), _ = qkv.qkv_rope(x, w, np.array([1]), 1, 1, 2, theta=10000.0)
    assert q.reshape(-1).tolist() == [0x3F0A, 0x3F57]
    assert k.reshape(-1).tolist() == [0, 0] and v.reshape(-1).tolist() == [0, 0]
