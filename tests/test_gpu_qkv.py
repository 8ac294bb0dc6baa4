"""GPU parity of the Q/K/V producer (arckv_qkv_rope) against the oracle.

Error bound of a bf16 output (derived from the arithmetic): y's fp32 sum of H
products can be off by H 2^-24 sum_h |x_h w_h| (the standard bound for a recursive sum), and
its bf16 rounding and the oracle's differ by up to one bf16 ulp (<= 2^-7 relative); a
rotation mixes the two members of a pair, so both errors are bounded by the pair's norm of
them; the final rounding adds half an ulp (2^-8 of the value); fp32 sine / cosine of angles
reduced in fp64 add ~1e-6 of the pair's norm.  Values are not rotated.
"""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

import paper_2606_21238_amd as ak  # noqa: E402
from oracle import qkv as oqkv  # noqa: E402
from oracle.attention import bf16_to_f64  # noqa: E402
from tests.gpu_helpers import bits, compare, print_case  # noqa: E402

DEV = "cuda"
THETA = 1.0e6


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ak.lib()


def randn_bf16(shape, seed, scale=1.0):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=DEV) * scale).to(torch.bfloat16)


def run(reqs, hidden, hq, hkv, d, seed):
    """reqs: [(L, P)]: each request computes its tokens P..L-1."""
    S = [L - P for L, P in reqs]
    T = sum(S)
    cu = np.concatenate([[0], np.cumsum(S)]).astype(np.int32)
    sl = np.array([L for L, _ in reqs], dtype=np.int32)
    x = randn_bf16((T, hidden), seed)
    w = randn_bf16(((hq + 2 * hkv) * d, hidden), seed + 1, hidden ** -0.5)
    q = torch.empty((T, hq, d), dtype=torch.bfloat16, device=DEV)
    k = torch.empty((T, hkv, d), dtype=torch.bfloat16, device=DEV)
    v = torch.empty((T, hkv, d), dtype=torch.bfloat16, device=DEV)
    ws = torch.empty(4 * T * d, dtype=torch.uint8, device=DEV)          # the exact table size
    ak.qkv_rope(x, w, torch.from_numpy(cu).to(DEV), torch.from_numpy(sl).to(DEV), hq, hkv, THETA,
                q, k, v, ws)
    torch.cuda.synchronize()
    pos = oqkv.token_positions(cu, sl)
    (qb, kb, vb), (qe, ke, ve) = oqkv.qkv_rope(bits(x), bits(w), pos, hq, hkv, d, THETA)
    y = bf16_to_f64(oqkv.f64_to_bf16_bits(oqkv.project(bits(x), bits(w))))
    acc = hidden * 2.0 ** -24 * (np.abs(bf16_to_f64(bits(x))) @ np.abs(bf16_to_f64(bits(w))).T)
    return dict(x=x, w=w, q=q, k=k, v=v, cu=cu, sl=sl, pos=pos, ref=(qe, ke, ve), refbits=(qb, kb, vb), y=y,
                acc=acc)


def pair_norm(y_heads):
    half = y_heads.shape[-1] // 2
    n = np.sqrt(y_heads[..., :half] ** 2 + y_heads[..., half:] ** 2)
    return np.concatenate([n, n], axis=-1)


def check(r, hq, hkv, d):
    T = r["q"].shape[0]
    nq, nk = hq * d, hkv * d
    heads = lambda a, lo, n, c: a[:, lo:lo + n].reshape(T, c, d)
    for name, got, ref, lo, c in (("q", r["q"], r["ref"][0], 0, hq), ("k", r["k"], r["ref"][1], nq, hkv)):
        g = bf16_to_f64(bits(got))
        yn, an = pair_norm(heads(r["y"], lo, c * d, c)), pair_norm(heads(r["acc"], lo, c * d, c))
        bound = 2.0 ** -7 * yn + an + 2.0 ** -8 * np.abs(ref) + 1e-6 * yn + 1e-30
        err = np.abs(g - ref)
        assert (err <= bound).all(), f"{name}: worst excess {float((err - bound).max()):.3g}"
        assert err.mean() < 2e-3, f"{name}: mean abs {err.mean():.3g}"
    gv = bf16_to_f64(bits(r["v"]))
    rv = r["ref"][2]
    ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.maximum(np.abs(gv), np.abs(rv)), 1e-30))) - 7)
    assert (np.abs(gv - rv) <= ulp + heads(r["acc"], nq + nk, nk, hkv)).all()


@pytest.mark.parametrize("reqs,hidden,hq,hkv,d", [
    ([(1, 0)], 64, 4, 2, 64),
    ([(300, 250), (17, 0), (40000, 39990)], 512, 8, 2, 128),           # positions up to 39999
    ([(129, 1), (64, 63)], 256, 16, 2, 64),
    ([(8320, 8192), (2100, 2048)], 5120, 40, 8, 128),                  # Qwen3-14B layer shape
    ([(3, 0), (9, 6)], 128, 4, 4, 128),                                # 6 tokens: a ragged group
    ([(1300, 0), (400, 300)], 256, 5, 1, 128),     # 6 x 3.5 tiles: a half output tile, ragged tokens
    ([(600, 0)], 96, 4, 1, 64),                    # 3 stages of H (short ring), 1.5 output tiles
    ([(300, 0), (70, 0)], 32, 2, 1, 64),           # one stage of H
])
def test_qkv_rope_matches_oracle(reqs, hidden, hq, hkv, d):
    print_case(f"qkv_rope {reqs} hidden={hidden} hq={hq} hkv={hkv} d={d}")
    r = run(reqs, hidden, hq, hkv, d, seed=11 + hidden)
    check(r, hq, hkv, d)


def test_layer_path_projection_scatter_attention():
    """Projected Q/K/V through the KV scatter into a paged pool, then prefill attention over
    a cached prefix written the same way: equals the oracle's attention on the oracle's
    Q/K/V within the attention tolerance."""
    from oracle import attention as oatt
    from oracle import kvpool as okv
    hidden, hq, hkv, d = 1024, 16, 4, 128
    L, P = 700, 600
    print_case("layer path: qkv_rope -> kv_scatter -> prefill_attention")
    # the whole prompt is projected (the prefix's K/V as they were when first computed)
    full = run([(L, 0)], hidden, hq, hkv, d, seed=5)
    nblk = (L + 15) // 16 + 3
    table = np.random.default_rng(0).permutation(nblk)[: (L + 15) // 16].astype(np.int32)
    slots = (table[np.arange(L) // 16] * 16 + np.arange(L) % 16).astype(np.int32)
    kp = torch.full((nblk, hkv, 16, d), -1, dtype=torch.int16, device=DEV)
    vp = torch.full((nblk, hkv, d, 16), -1, dtype=torch.int16, device=DEV)
    ak.kv_scatter(kp, vp, full["k"], full["v"], torch.from_numpy(slots).to(DEV))
    q = full["q"][P:].contiguous()
    cu = np.array([0, L - P], dtype=np.int32)
    sl = np.array([L], dtype=np.int32)
    ap = ak.attention_plan(cu, sl, hq, hkv, d)
    out = torch.empty_like(q)
    wsa = torch.zeros(max(ap.ws_bytes, 1), dtype=torch.uint8, device=DEV)
    ak.prefill_attention(kp, vp, q, out, torch.from_numpy(table[None, :]).to(DEV), torch.from_numpy(cu).to(DEV),
                         torch.from_numpy(sl).to(DEV), torch.from_numpy(ap.work).to(DEV), ap.n_work,
                         ap.n_combine, ap.tile_cols, d ** -0.5, wsa, ap.ws_bytes)
    torch.cuda.synchronize()
    qb, kb, vb = full["refbits"]
    okp, ovp = okv.new_pool(nblk, hkv, d)
    okv.scatter(okp, ovp, kb, vb, slots)
    ref = oatt.prefill_attention(qb[P:], okp, ovp, [table], cu, sl, d ** -0.5)
    compare(bits(out), ref, "layer path")


def slot_pattern(kind, reqs, nblk, rng):
    """Slots of the computed tokens: 'prefill' places each request's positions P..L-1 through a
    random block table (8-token runs wherever a request's positions are 8-aligned), 'random'
    is a permutation of the pool's slots (no runs), 'skips' is 'prefill' with some slots -1 or
    past the pool."""
    if kind == "random":
        T = sum(L - P for L, P in reqs)
        return rng.permutation(nblk * 16)[:T].astype(np.int32)
    perm = rng.permutation(nblk)
    out, o = [], 0
    for L, P in reqs:
        n = (L + 15) // 16
        table = perm[o:o + n]
        o += n
        pos = np.arange(P, L)
        out.append(table[pos // 16] * 16 + pos % 16)
    s = np.concatenate(out).astype(np.int32)
    if kind == "skips":
        idx = rng.choice(len(s), max(1, len(s) // 20), replace=False)
        s[idx[::2]] = -1
        s[idx[1::2]] = nblk * 16 + 5
    return s


@pytest.mark.parametrize("kind", ["prefill", "random", "skips"])
@pytest.mark.parametrize("reqs,hidden,hq,hkv,d", [
    ([(2100, 2048), (300, 0), (17, 5), (40, 33)], 512, 40, 8, 128),   # Qwen3-14B heads
    ([(700, 100), (129, 1)], 256, 6, 1, 64),       # one output tile holds Q, K and V columns
    ([(520, 0), (9, 0)], 128, 5, 1, 128),          # Q and K share a tile, V a half tile
])
def test_qkv_rope_to_pool_equals_projection_then_scatter(kind, reqs, hidden, hq, hkv, d):
    """arckv_qkv_rope_to_pool against arckv_qkv_rope followed by arckv_kv_scatter (itself
    checked against the oracle above and in the scatter tests): Q and both whole pools,
    including the untouched sentinel bytes, bit for bit."""
    print_case(f"qkv_rope_to_pool {kind} {reqs} hidden={hidden} hq={hq} hkv={hkv} d={d}")
    rng = np.random.default_rng(hidden + d + len(kind))
    S = [L - P for L, P in reqs]
    T = sum(S)
    nblk = sum((L + 15) // 16 for L, _ in reqs) + 6
    cu = torch.from_numpy(np.concatenate([[0], np.cumsum(S)]).astype(np.int32)).to(DEV)
    sl = torch.from_numpy(np.array([L for L, _ in reqs], dtype=np.int32)).to(DEV)
    slots = torch.from_numpy(slot_pattern(kind, reqs, nblk, rng)).to(DEV)
    x = randn_bf16((T, hidden), 21 + hidden)
    w = randn_bf16(((hq + 2 * hkv) * d, hidden), 22 + hidden, hidden ** -0.5)
    ws = torch.empty(4 * T * d, dtype=torch.uint8, device=DEV)

    q_a = torch.empty((T, hq, d), dtype=torch.bfloat16, device=DEV)
    k_a = torch.empty((T, hkv, d), dtype=torch.bfloat16, device=DEV)
    v_a = torch.empty((T, hkv, d), dtype=torch.bfloat16, device=DEV)
    kp_a = torch.full((nblk, hkv, 16, d), -1, dtype=torch.int16, device=DEV)
    vp_a = torch.full((nblk, hkv, d, 16), -1, dtype=torch.int16, device=DEV)
    ak.qkv_rope(x, w, cu, sl, hq, hkv, THETA, q_a, k_a, v_a, ws)
    ak.kv_scatter(kp_a, vp_a, k_a, v_a, slots)

    q_b = torch.full((T, hq, d), float("nan"), dtype=torch.bfloat16, device=DEV)
    kp_b = torch.full((nblk, hkv, 16, d), -1, dtype=torch.int16, device=DEV)
    vp_b = torch.full((nblk, hkv, d, 16), -1, dtype=torch.int16, device=DEV)
    ak.qkv_rope_to_pool(x, w, cu, sl, hq, hkv, THETA, q_b, kp_b, vp_b, slots, ws)
    torch.cuda.synchronize()
    assert np.array_equal(bits(q_a), bits(q_b)), "Q differs"
    assert np.array_equal(bits(kp_a), bits(kp_b)), "K pool differs"
    assert np.array_equal(bits(vp_a), bits(vp_b)), "V pool differs"
    written = int((bits(kp_b) != 0xFFFF).any(axis=(1, 3)).sum())
    assert written > 0
