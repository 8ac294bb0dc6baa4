"""GPU parity: libarckv's HIP scatter and prefill attention against the CPU oracle.

Every case drives the library through its C ABI (via the ctypes binding) on seeded
synthetic inputs and checks: pool bytes bit-exact (scatter), block tables / slots equal to
the oracle planner's, attention within max-abs 1e-2 and mean-abs 1e-3 of the fp64 oracle
(bf16 inputs, fp32 accumulation, bf16 output).
"""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2606_21238_amd as ak  # noqa: E402
from paper_2606_21238_amd.engine import PrefillEngine  # noqa: E402
from oracle import attention as oatt  # noqa: E402
from oracle import blockhash as obh  # noqa: E402
from oracle import kvpool as okv  # noqa: E402
from oracle.planner import Planner, form_batches  # noqa: E402
from workloads import get_config  # noqa: E402
from workloads.streams import TensorBank, free_order, make_stream, steps_short, stream_docqa_hit  # noqa: E402
from tests.gpu_helpers import bits, compare, print_case, sample_rows  # noqa: E402

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ak.lib()


def randn_bf16(shape, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return torch.randn(shape, generator=g, device=DEV).to(torch.bfloat16)


# ------------------------------------------------------------------------------------------
# scatter
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("d,hkv,n", [(64, 2, 1), (64, 2, 63), (128, 8, 64), (128, 8, 65), (128, 8, 1000),
                                     (64, 1, 300)])
def test_scatter_bit_exact(d, hkv, n):
    print_case(f"scatter d={d} hkv={hkv} n={n}")
    rng = np.random.default_rng(n * 13 + d)
    nblk = (n + 15) // 16 + 7
    slots = rng.permutation(nblk * 16)[:n].astype(np.int32)
    slots[rng.integers(0, n, max(1, n // 50))] = -1            # padding slots are skipped
    k_new = randn_bf16((n, hkv, d), 1 + n)
    v_new = randn_bf16((n, hkv, d), 2 + n)
    eng_k = torch.full((nblk, hkv, 16, d), -1, dtype=torch.int16, device=DEV)
    eng_v = torch.full((nblk, hkv, d, 16), -1, dtype=torch.int16, device=DEV)
    ak.kv_scatter(eng_k, eng_v, k_new, v_new, torch.from_numpy(slots).to(DEV))
    torch.cuda.synchronize()
    kp, vp = okv.new_pool(nblk, hkv, d)
    keep = slots >= 0
    okv.scatter(kp, vp, bits(k_new)[keep], bits(v_new)[keep], slots[keep])
    assert np.array_equal(bits(eng_k), kp)
    assert np.array_equal(bits(eng_v), vp)


@pytest.mark.parametrize("d,hkv,n,start", [(64, 2, 1000, 0), (128, 8, 1000, 5), (128, 8, 3000, 3),
                                           (64, 4, 2500, 8), (128, 2, 8, 0), (128, 8, 1025, 0)])
def test_scatter_block_runs_bit_exact(d, hkv, n, start):
    """Prefill-shaped slots (requests in consecutive slots of their blocks, starting at
    `start` inside the first block), with a few skipped slots: 8-token runs take the 16-byte
    stores, broken runs the 2-byte ones; both on the small- and the large-batch grid."""
    print_case(f"scatter runs d={d} hkv={hkv} n={n} start={start}")
    rng = np.random.default_rng(n + 7 * d + start)
    nblk = (n + start + 15) // 16 + 9
    table = rng.permutation(nblk)
    j = np.arange(n) + start
    slots = (table[j // 16] * 16 + j % 16).astype(np.int32)
    slots[rng.integers(0, n, max(1, n // 300))] = -1
    k_new = randn_bf16((n, hkv, d), 3 + n)
    v_new = randn_bf16((n, hkv, d), 4 + n)
    eng_k = torch.full((nblk, hkv, 16, d), -1, dtype=torch.int16, device=DEV)
    eng_v = torch.full((nblk, hkv, d, 16), -1, dtype=torch.int16, device=DEV)
    ak.kv_scatter(eng_k, eng_v, k_new, v_new, torch.from_numpy(slots).to(DEV))
    torch.cuda.synchronize()
    kp, vp = okv.new_pool(nblk, hkv, d)
    keep = slots >= 0
    okv.scatter(kp, vp, bits(k_new)[keep], bits(v_new)[keep], slots[keep])
    assert np.array_equal(bits(eng_k), kp)
    assert np.array_equal(bits(eng_v), vp)


# ------------------------------------------------------------------------------------------
# attention on directly built batches (random placement, edge lengths)
# ------------------------------------------------------------------------------------------

def build_batch(reqs, hq, hkv, d, seed, extra_blocks=5, k_gain=None, v_gain=1.0):
    """reqs: [(L, P)].  Random placement of every request's blocks in one pool; all L tokens'
    K/V written by the library scatter; returns device tensors and oracle-side copies.
    k_gain: optional function of a token's position in its prompt (numpy array in, array out)
    scaling its K row, so that scores grow, fall or jump along the keys; v_gain scales V."""
    rng = np.random.default_rng(seed)
    nb = [(L + 15) // 16 for L, _ in reqs]
    nphys = sum(nb) + extra_blocks
    perm = rng.permutation(nphys)
    tables, o = [], 0
    for n in nb:
        tables.append(perm[o:o + n].astype(np.int32))
        o += n
    stride = max(nb)
    bt = np.full((len(reqs), stride), -1, dtype=np.int32)
    for r, t in enumerate(tables):
        bt[r, : len(t)] = t
    Ls = [L for L, _ in reqs]
    Ss = [L - P for L, P in reqs]
    cu = np.concatenate([[0], np.cumsum(Ss)]).astype(np.int32)
    k_all = randn_bf16((sum(Ls), hkv, d), seed + 1)
    v_all = randn_bf16((sum(Ls), hkv, d), seed + 2)
    if k_gain is not None:
        pos = np.concatenate([np.arange(L) for L in Ls]).astype(np.float64)
        gain = torch.from_numpy(np.asarray(k_gain(pos), dtype=np.float32)).to(DEV)
        k_all = (k_all.float() * gain[:, None, None]).to(torch.bfloat16)
    if v_gain != 1.0:
        v_all = (v_all.float() * v_gain).to(torch.bfloat16)
    q_all = randn_bf16((sum(Ss), hq, d), seed + 3)
    slots = np.concatenate([tables[r][np.arange(L) // 16] * 16 + np.arange(L) % 16
                            for r, L in enumerate(Ls)]).astype(np.int32)
    kp = torch.full((nphys, hkv, 16, d), -1, dtype=torch.int16, device=DEV)
    vp = torch.full((nphys, hkv, d, 16), -1, dtype=torch.int16, device=DEV)
    ak.kv_scatter(kp, vp, k_all, v_all, torch.from_numpy(slots).to(DEV))
    okp, ovp = okv.new_pool(nphys, hkv, d)
    okv.scatter(okp, ovp, bits(k_all), bits(v_all), slots)
    return dict(kp=kp, vp=vp, q=q_all, bt=bt, cu=cu, seq=np.array(Ls, dtype=np.int32), tables=tables,
                okp=okp, ovp=ovp, qbits=bits(q_all))


def run_attention(b, hq, hkv, d, num_cus=256, table_override=None, kp=None, vp=None, ws=None):
    ap = ak.attention_plan(b["cu"], b["seq"], hq, hkv, d, num_cus)
    bt = b["bt"] if table_override is None else table_override
    out = torch.empty_like(b["q"])
    if ws is None:
        ws = torch.zeros(max(ap.ws_bytes, 1), dtype=torch.uint8, device=DEV)
    ak.prefill_attention(b["kp"] if kp is None else kp, b["vp"] if vp is None else vp, b["q"], out,
                         torch.from_numpy(bt).to(DEV), torch.from_numpy(b["cu"]).to(DEV),
                         torch.from_numpy(b["seq"]).to(DEV), torch.from_numpy(ap.work).to(DEV),
                         ap.n_work, ap.n_combine, ap.tile_cols, d ** -0.5, ws, ap.ws_bytes)
    torch.cuda.synchronize()
    return bits(out), ap


def oracle_out(b, hq, hkv, d, rows=None):
    return oatt.prefill_attention(b["qbits"], b["okp"], b["ovp"], b["tables"], b["cu"], b["seq"],
                                  d ** -0.5, rows_per_request=rows)


SWEEP = [
    # (reqs [(L, P)], hq, hkv, d)
    ([(1, 0)], 4, 2, 64),
    ([(64, 0)], 4, 4, 64),
    ([(320, 256)], 4, 2, 64),
    ([(17, 16), (15, 0), (65, 64), (100, 48)], 8, 2, 128),
    ([(63, 0), (64, 0), (65, 0), (129, 0)], 8, 1, 128),
    ([(1040, 1024), (300, 16), (77, 0)], 32, 8, 128),
    ([(2000, 1536)], 16, 2, 64),
    ([(700, 0), (33, 32), (1, 0)], 8, 8, 128),
    ([(5000, 4990)], 8, 2, 128),                 # many pieces per tile
    # decode-like batches (one new token per request: 32-column tiles)
    ([(L, L - 1) for L in (1, 2, 17, 64, 65, 300, 1024, 2049, 4097, 777, 33, 16)], 32, 8, 128),
    ([(L, L - 2) for L in (2, 3, 40, 129, 1500, 3001)], 16, 2, 64),
    # G = 4 at d = 64; column counts on and just past each tile width (32, 128, 256 columns)
    ([(900, 892), (70, 62)], 8, 2, 64),                 # 32 columns (narrow tiles)
    ([(900, 891), (77, 68)], 8, 2, 64),                 # 36 columns: narrow tiles
    ([(700, 668), (1000, 968)], 16, 4, 64),             # 128 columns: narrow tiles
    ([(700, 667), (64, 31)], 16, 4, 64),                # 132 columns: wide tiles
    ([(512, 448), (2048, 1984), (65, 1)], 32, 8, 128),  # 256 columns: wide tiles, one tile each
    ([(513, 448), (130, 65)], 32, 8, 128),              # 260 columns: a second, 4-column tile
    # G = 5 (Qwen3-14B's 40 / 8 heads): tile edges fall inside a token's group of heads
    ([(1040, 1024), (300, 16), (77, 0)], 40, 8, 128),
    ([(4000, 3949), (130, 78), (6, 0)], 40, 8, 128),    # 255, 260 and 30 columns
    ([(700, 600), (33, 0), (1, 0)], 10, 2, 64),
    ([(L, L - 1) for L in (1, 17, 300, 4097, 65, 2000)], 40, 8, 128),   # decode (narrow tiles)
    ([(40000, 39999)], 8, 1, 64),        # 79 pieces of one tile: the combine's second batch of 64
]


@pytest.mark.parametrize("num_cus", [256, 100000])   # 100000 forces key-range splits + combine
@pytest.mark.parametrize("case", range(len(SWEEP)))
def test_attention_sweep(case, num_cus):
    reqs, hq, hkv, d = SWEEP[case]
    print_case(f"attention sweep {reqs} hq={hq} hkv={hkv} d={d} num_cus={num_cus}")
    b = build_batch(reqs, hq, hkv, d, seed=1000 + case)
    got, ap = run_attention(b, hq, hkv, d, num_cus)
    ref = oracle_out(b, hq, hkv, d)
    compare(got, ref, f"case {case}")
    if num_cus > 1000 and max(L for L, _ in reqs) > 512:   # splits are >= 512 keys
        assert (ap.work[: ap.n_work, 5] >= 0).any()


# Scores that grow, jump or spike along the keys, so that the running maximum moves after the
# first key tile of an item (the online softmax's rescale), and scores that fall (it never
# does).  With N(0, 1) inputs a 128-dim score has a standard deviation of about 1.4 in log2
# units, so gains of 4-30 move the maxima by tens to hundreds; V is scaled down to keep the
# (nearly one-hot) outputs small next to the tolerance.
RESCALE = [
    ("linear growth", lambda t: 1.0 + t / 128.0),
    ("steps every 512 keys", lambda t: 1.0 + 4.0 * np.floor(t / 512.0)),
    ("spikes on every 97th key", lambda t: np.where(t % 97 == 13, 8.0, 1.0)),
    ("moderate rises (sums past 2^8 without one large term)", lambda t: 1.0 + 0.35 * (np.floor(t / 64.0) % 12)),
    ("falling", lambda t: 30.0 / (1.0 + t / 64.0)),
]


@pytest.mark.parametrize("num_cus", [256, 100000])
@pytest.mark.parametrize("case", range(len(RESCALE)))
def test_attention_moving_maxima(case, num_cus):
    name, gain = RESCALE[case]
    for reqs, hq, hkv, d in (([(3000, 2000), (700, 0)], 32, 8, 128),               # wide tiles
                             ([(L, L - 1) for L in (5000, 2049, 300)], 32, 8, 128),  # lists (decode)
                             ([(1500, 1000)], 8, 2, 64)):
        print_case(f"moving maxima '{name}' {reqs} hq={hq} hkv={hkv} d={d} num_cus={num_cus}")
        b = build_batch(reqs, hq, hkv, d, seed=1300 + 7 * case, k_gain=gain, v_gain=0.25)
        got, _ = run_attention(b, hq, hkv, d, num_cus)
        compare(got, oracle_out(b, hq, hkv, d), f"{name}, {reqs}")


def test_attention_beyond_the_item_key_cap():
    # 70000 keys: every tile's range exceeds one item's 65536-key cap, so the plan splits it and
    # the combine merges the pieces (wide tiles on the ping-pong kernel); sampled rows
    hq, hkv, d = 16, 2, 128
    reqs = [(70000, 69800)]
    print_case(f"key cap {reqs} hq={hq} hkv={hkv} d={d}")
    b = build_batch(reqs, hq, hkv, d, seed=880)
    got, ap = run_attention(b, hq, hkv, d, 256)
    assert ap.n_combine > 0 and ap.tile_cols == 256
    rng = np.random.default_rng(8)
    rows = [sample_rows(200, rng, 24)]
    ref = oracle_out(b, hq, hkv, d, rows)
    compare(got, ref, "beyond the key cap")


def test_split_merges_reuse_one_workspace():
    # split plans of different shapes in a row on one workspace (stale partials of an earlier
    # call must not leak into a later one)
    hq, hkv, d = 32, 8, 128
    cases = [([(1040, 1024), (2100, 2068), (600, 500)], 100000),
             ([(3000, 2990), (900, 880)], 100000),
             ([(5000, 4990)], 256),
             ([(1040, 1024), (2100, 2068), (600, 500)], 100000)]
    ws = torch.zeros(64 << 20, dtype=torch.uint8, device=DEV)
    for k, (reqs, num_cus) in enumerate(cases):
        print_case(f"workspace reuse {k}: {reqs} num_cus={num_cus}")
        b = build_batch(reqs, hq, hkv, d, seed=300 + k)
        got, ap = run_attention(b, hq, hkv, d, num_cus, ws=ws)
        assert 0 < ap.ws_bytes <= ws.numel()
        compare(got, oracle_out(b, hq, hkv, d), f"reuse {k}")


def test_block_table_permutation_bitwise():
    hq, hkv, d = 16, 4, 128
    reqs = [(900, 512), (260, 0)]
    print_case(f"permutation invariance {reqs}")
    b = build_batch(reqs, hq, hkv, d, seed=77, extra_blocks=40)
    got1, _ = run_attention(b, hq, hkv, d)
    # move every block to a new physical place and rewrite the tables
    nphys = b["kp"].shape[0]
    perm = torch.from_numpy(np.random.default_rng(5).permutation(nphys)).to(DEV)
    kp2 = torch.empty_like(b["kp"])
    vp2 = torch.empty_like(b["vp"])
    kp2[perm] = b["kp"]
    vp2[perm] = b["vp"]
    pm = perm.cpu().numpy()
    bt2 = np.where(b["bt"] >= 0, pm[np.maximum(b["bt"], 0)], -1).astype(np.int32)
    got2, _ = run_attention(b, hq, hkv, d, table_override=bt2, kp=kp2, vp=vp2)
    assert np.array_equal(got1, got2)


def test_prefix_cached_equals_full_recompute():
    # the suffix rows computed with a cached prefix equal the same rows of a full recompute
    hq, hkv, d = 8, 2, 128
    L, P = 640, 448
    print_case("prefix-cached vs recompute")
    full = build_batch([(L, 0)], hq, hkv, d, seed=91)
    got_full, _ = run_attention(full, hq, hkv, d, num_cus=1)
    cached = dict(full)
    cached["q"] = full["q"][P:].contiguous()
    cached["qbits"] = full["qbits"][P:]
    cached["cu"] = np.array([0, L - P], dtype=np.int32)
    got_cached, _ = run_attention(cached, hq, hkv, d, num_cus=1)
    assert np.array_equal(got_cached, got_full[P:])
    compare(got_cached, oracle_out(cached, hq, hkv, d), "cached")


# ------------------------------------------------------------------------------------------
# the workload configurations end to end (planner + scatter + attention)
# ------------------------------------------------------------------------------------------

class Lockstep:
    """Library engine and oracle (planner + pool image) over the same request stream."""

    def __init__(self, cfg, device_bank=True):
        order = free_order(cfg.seed, cfg.num_phys)
        self.cfg = cfg
        self.eng = PrefillEngine(cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.capacity,
                                 cfg.num_phys, cfg.scratch, cfg.policy, order)
        self.orc = Planner(cfg.policy, cfg.capacity, cfg.num_phys, cfg.scratch, order)
        self.okp, self.ovp = okv.new_pool(cfg.num_phys, cfg.num_kv_heads, cfg.head_dim)
        self.bank = TensorBank(cfg, DEV)

    def batch(self, reqs, rows_fn=None, check_pool=True, native_prepare=False):
        """native_prepare: the engine's one-call path (arckv_prepare_batch) instead of
        plan() + upload()."""
        cfg = self.cfg
        toks = [r.tokens for r in reqs]
        oplan = self.orc.plan_batch([(obh.hash_blocks(t), len(t)) for t in toks])
        if native_prepare:
            db = self.eng.prepare(toks)
            plan = db.plan
        else:
            plan = self.eng.plan(toks)
            db = self.eng.upload(plan)
        assert plan.prefix_lens.tolist() == oplan.prefix_lens
        assert plan.slot_mapping.tolist() == oplan.slot_mapping
        for r, row in enumerate(oplan.block_tables):
            assert plan.block_tables[r, : len(row)].tolist() == row
        q, kn, vn = self.bank.batch_suffix(reqs, oplan.prefix_lens)
        out = torch.empty_like(q)
        self.eng.scatter(db, kn, vn)
        self.eng.attention(db, q, out)
        torch.cuda.synchronize()
        self.eng.release()
        self.orc.release_batch()
        okv.scatter(self.okp, self.ovp, bits(kn), bits(vn), oplan.slot_mapping)
        if check_pool:
            touched = sorted(okv.touched_blocks(oplan.slot_mapping))
            assert np.array_equal(bits(self.eng.k_pool[touched]), self.okp[touched])
            assert np.array_equal(bits(self.eng.v_pool[touched]), self.ovp[touched])
        rows = None if rows_fn is None else [rows_fn(r, oplan) for r in range(len(reqs))]
        ref = oatt.prefill_attention(bits(q), self.okp, self.ovp, oplan.block_tables, oplan.cu_q,
                                     oplan.seq_lens, cfg.scale, rows_per_request=rows)
        return oplan, bits(out), ref


def test_tiny_config():
    cfg = get_config("tiny")
    print_case("config tiny")
    ls = Lockstep(cfg)
    r0, r1 = make_stream(cfg)
    _, got0, ref0 = ls.batch([r0])
    compare(got0, ref0, "tiny warm")
    plan, got, ref = ls.batch([r1])
    assert plan.prefix_lens == [256] and plan.cu_q == [0, 64]
    compare(got, ref, "tiny")
    # the whole pool image matches, untouched blocks included
    assert np.array_equal(bits(ls.eng.k_pool), ls.okp)
    assert np.array_equal(bits(ls.eng.v_pool), ls.ovp)


def test_docqa_all_hit_batch():
    cfg = get_config("docqa")
    print_case("config docqa 2-hit (8 x (8192 cached + 128))")
    ls = Lockstep(cfg)
    warm, hot = stream_docqa_hit(cfg)
    rng = np.random.default_rng(2)
    ls.batch(warm, rows_fn=lambda r, p: [0, 63, 64, 4095, 8191])
    plan, got, ref = ls.batch(hot)
    assert plan.prefix_lens == [8192] * 8
    compare(got, ref, "docqa 2-hit")


def test_docqa_stream_batches():
    cfg = get_config("docqa")
    print_case("config docqa stream, 6 batches, row-sampled")
    ls = Lockstep(cfg)
    stream = make_stream(cfg, n_batches=6)
    rng = np.random.default_rng(3)
    fn = lambda r, p: sample_rows(p.cu_q[r + 1] - p.cu_q[r], rng, 24)
    for a, b in form_batches([r.n_tokens for r in stream], cfg.max_batch, cfg.capacity, cfg.scratch):
        _, got, ref = ls.batch(stream[a:b], rows_fn=fn)
        compare(got, ref, f"docqa batch {a}")


@pytest.mark.parametrize("S", [32, 48, 64])
def test_short_full_batches(S):
    """The short32 / short48 / short64 bench shapes: 16 cached lognormal histories + S new
    tokens each (128-column tiles at S = 32, 256-column tiles above)."""
    cfg = get_config("short")
    print_case(f"config short{S} (16 x (history + {S})), row-sampled, native prepare")
    ls = Lockstep(cfg)
    warm, steps = steps_short(cfg, 2, S)
    rng = np.random.default_rng(6 + S)
    for w in warm:
        ls.batch(w, rows_fn=lambda r, p: [0, int(p.cu_q[r + 1] - p.cu_q[r]) - 1], native_prepare=True)
    for k, b in enumerate(steps):
        plan, got, ref = ls.batch(b, rows_fn=lambda r, p: sample_rows(S, rng, 8), native_prepare=True)
        assert all(s == S for s in np.diff(plan.cu_q))
        compare(got, ref, f"short{S} step {k}")


def test_decode_full_batch():
    """The decode bench shape: 64 cached lognormal histories + 1 new token each (128-column
    tiles, split key ranges), every row checked."""
    cfg = get_config("decode")
    print_case("config decode (64 x (history + 1)), all rows, native prepare")
    ls = Lockstep(cfg)
    warm, steps = steps_short(cfg, 2, 1, batch=cfg.max_batch, n_sessions=cfg.max_batch)
    for w in warm:
        ls.batch(w, rows_fn=lambda r, p: [int(p.cu_q[r + 1] - p.cu_q[r]) - 1], native_prepare=True)
    for k, b in enumerate(steps):
        plan, got, ref = ls.batch(b, native_prepare=True)
        assert len(b) == 64 and all(s == 1 for s in np.diff(plan.cu_q))
        compare(got, ref, f"decode step {k}")


def test_list_plan_with_full_lists_over_several_rounds():
    """Narrow batch of 600 one-token requests over short histories: the list plan packs 8 items
    into every list and needs more lists than CUs (several rounds of persistent work-groups);
    one history longer than an item's key cap is split into pieces.  Every row checked."""
    hq, hkv, d = 16, 4, 128
    rng = np.random.default_rng(91)
    L = rng.integers(2, 300, 600)
    L[17] = 70000                                   # beyond one item's 65536-key cap
    reqs = [(int(x), int(x) - 1) for x in L]
    print_case(f"list plan: {len(reqs)} one-token requests, hq={hq} hkv={hkv} d={d}")
    b = build_batch(reqs, hq, hkv, d, seed=92)
    got, ap = run_attention(b, hq, hkv, d, 256)
    lists = ap.work[: ap.n_work].reshape(-1, 8, 8)
    assert ap.tile_cols == 128 and len(lists) > 256
    assert ((lists[:, :, 0] >= 0).sum(axis=1) == 8).sum() > 100 and ap.n_combine >= 1
    compare(got, oracle_out(b, hq, hkv, d), "full lists")


def test_longctx_sampled_rows():
    cfg = get_config("longctx")
    print_case("config longctx (4 x (32768 cached + 2048)), row-sampled")
    ls = Lockstep(cfg)
    warm, hot = make_stream(cfg)
    rng = np.random.default_rng(4)
    ls.batch(warm, rows_fn=lambda r, p: [0, 32767], check_pool=True)
    plan, got, ref = ls.batch(hot, rows_fn=lambda r, p: sample_rows(2048, rng, 16))
    assert plan.prefix_lens == [32768] * 4
    compare(got, ref, "longctx")


def test_empty_work_is_a_noop():
    b = build_batch([(32, 0)], 4, 2, 64, seed=3)
    out = torch.zeros_like(b["q"])
    ak.prefill_attention(b["kp"], b["vp"], b["q"], out, torch.from_numpy(b["bt"]).to(DEV),
                         torch.from_numpy(b["cu"]).to(DEV), torch.from_numpy(b["seq"]).to(DEV),
                         torch.zeros((1, 8), dtype=torch.int32, device=DEV), 0, 0, 256, 0.125)
    torch.cuda.synchronize()
    assert int(out.abs().sum()) == 0


def test_timed_entry_point_matches_and_records_events():
    """arckv_prefill_attention_timed computes the same bytes and records its three events."""
    cfg = get_config("docqa")
    print_case("timed entry point vs plain entry point (docqa hit batch)")
    ls = Lockstep(cfg)
    warm, hot = stream_docqa_hit(cfg)
    ls.batch(warm, rows_fn=lambda r, p: [0], check_pool=False)
    toks = [r.tokens for r in hot]
    plan = ls.eng.plan(toks)
    db = ls.eng.upload(plan)
    q, _, _ = ls.bank.batch_suffix(hot, plan.prefix_lens)
    out1, out2 = torch.empty_like(q), torch.empty_like(q)
    ls.eng.attention(db, q, out1)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    for e in evs:
        e.record()
    torch.cuda.synchronize()
    ls.eng.attention(db, q, out2, events=evs)
    torch.cuda.synchronize()
    ls.eng.release()
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    assert evs[0].elapsed_time(evs[1]) > 0 and evs[1].elapsed_time(evs[2]) >= 0
