"""arckv_prepare_batch (hash + plan + attention work plan in one native call) against the same
library calls made one by one on a twin cache (CPU only): identical plans, work items,
decision logs and cache state; a packed buffer below the bound leaves the cache unchanged."""

import numpy as np
import pytest

import paper_2606_21238_amd as ak
from paper_2606_21238_amd import _lib
from workloads import get_config
from workloads.streams import Source, make_request, KIND_DOC


def twin(policy, c, nphys, scratch, order, window=1):
    a = ak.BlockCache(policy, c, nphys, scratch, order, victim_window=window)
    b = ak.BlockCache(policy, c, nphys, scratch, order, victim_window=window)
    a.set_log(1 << 20)
    b.set_log(1 << 20)
    return a, b


def separate(cache, toks, hq, hkv, d, num_cus):
    hs = ak.hash_blocks_batch(toks)
    stride = max((len(t) + 15) // 16 for t in toks)
    plan = cache.plan_batch([(h, len(t)) for h, t in zip(hs, toks)], bt_stride=stride)
    return plan, ak.attention_plan(plan.cu_q, plan.seq_lens, hq, hkv, d, num_cus)


@pytest.mark.parametrize("policy,hq,hkv,d,num_cus,window", [
    ("arc", 32, 8, 128, 256, 1), ("lru", 8, 2, 64, 80, 1), ("dbl", 40, 8, 128, 256, 1),
    ("arc", 4, 4, 64, 1000, 4),
])
def test_prepare_equals_the_calls_in_sequence(policy, hq, hkv, d, num_cus, window):
    cfg = get_config("tiny")
    rng = np.random.default_rng(9)
    c, scratch = 60, 8
    nphys = c + scratch + 3
    a, b = twin(policy, c, nphys, scratch, rng.permutation(nphys), window)
    docs = [make_request(cfg, [(Source(KIND_DOC, k, 400), 0, 400)]).tokens for k in range(10)]
    packed = np.empty(16, dtype=np.int32)          # grows on the first ENOSPC
    n_batches = 0
    for _ in range(80):
        toks = []
        for _ in range(int(rng.integers(1, 5))):
            k = int(rng.integers(0, 10))
            n = int(rng.integers(1, 400))
            extra = rng.integers(0, 128256, int(rng.integers(0, 60))).astype(np.int32)
            toks.append(np.concatenate([docs[k][:n], extra]).astype(np.int32))
        if sum(len(t) // 16 for t in toks) > c or sum(1 for t in toks if len(t) % 16) > scratch:
            continue
        pb = a.prepare_batch(toks, hq, hkv, d, num_cus, packed)
        packed = pb.packed
        plan, ap = separate(b, toks, hq, hkv, d, num_cus)
        got = pb.plan
        for f in ("block_tables", "cu_q", "seq_lens", "prefix_lens", "hit_blocks", "slot_mapping"):
            assert np.array_equal(getattr(got, f), getattr(plan, f)), f
        assert (got.max_q_len, got.max_seq_len) == (plan.max_q_len, plan.max_seq_len)
        nw = ap.n_work + ap.n_combine
        assert (pb.attn.n_work, pb.attn.n_combine, pb.attn.ws_bytes, pb.attn.tile_cols) == \
            (ap.n_work, ap.n_combine, ap.ws_bytes, ap.tile_cols)
        assert np.array_equal(pb.attn.work[:nw], ap.work[:nw])
        # the packed layout: tables | cu_q | seq_lens | slots | work, nothing after
        i = pb.info
        assert i["off_cu_q"] == i["n_reqs"] * i["bt_stride"] and i["off_work"] == i["off_slots"] + i["n_slots"]
        assert i["n_packed"] == i["off_work"] + nw * ak.WORK_INTS
        a.release_batch()
        b.release_batch()
        n_batches += 1
    assert n_batches > 40
    assert a.log() == b.log()
    assert a.stats() == b.stats()
    for li in (ak.LIST_T1, ak.LIST_T2, ak.LIST_B1, ak.LIST_B2):
        ka, pa = a.snapshot(li)
        kb, pb_ = b.snapshot(li)
        assert np.array_equal(ka, kb) and np.array_equal(pa, pb_)


def test_too_small_buffer_reports_the_bound_and_changes_nothing():
    cache = ak.BlockCache("arc", 64, 80, 8)
    toks = [np.arange(100, dtype=np.int32), np.arange(50, dtype=np.int32) + 7]
    before = cache.stats()
    st, info, _, _ = cache.prepare_native(toks, 32, 8, 128, 256, np.empty(8, dtype=np.int32))
    assert st == _lib.ENOSPC and info["n_packed"] > 8
    assert cache.stats() == before and before["in_flight"] == 0
    st, info2, _, _ = cache.prepare_native(toks, 32, 8, 128, 256, np.empty(info["n_packed"], dtype=np.int32))
    assert st == _lib.OK and info2["n_packed"] <= info["n_packed"]
    assert cache.stats()["in_flight"] == 1
    # a second batch before release is refused like plan_batch, with nothing changed
    st, _, _, _ = cache.prepare_native(toks, 32, 8, 128, 256, np.empty(info["n_packed"], dtype=np.int32))
    assert st == _lib.ESTATE
    cache.release_batch()


def test_packed_bound_covers_every_possible_work_plan():
    # the bound depends only on prompt lengths; the work plan depends on how much was cached
    # (S <= L): any S must fit
    rng = np.random.default_rng(4)
    cache = ak.BlockCache("lru", 1 << 16, (1 << 16) + 64, 64)
    for _ in range(300):
        n = int(rng.integers(1, 65))
        lens = rng.integers(1, rng.choice([40, 600, 20000]), n)
        hq, hkv = [(32, 8), (40, 8), (8, 1), (16, 16), (64, 8)][int(rng.integers(0, 5))]
        num_cus = int(rng.choice([1, 7, 256, 1000]))
        toks = [np.zeros(int(x), dtype=np.int32) for x in lens]
        st, info, _, _ = cache.prepare_native(toks, hq, hkv, 128, num_cus, None)
        assert st == _lib.ENOSPC
        bound = info["n_packed"]
        S = np.array([int(rng.integers(1, x + 1)) for x in lens])
        if rng.random() < 0.3:
            S = np.minimum(S, 1)
        cu = np.concatenate([[0], np.cumsum(S)]).astype(np.int32)
        ap = ak.attention_plan(cu, lens.astype(np.int32), hq, hkv, 128, num_cus)
        stride = int(max((lens + 15) // 16))
        used = n * stride + 2 * n + 1 + int(S.sum()) + ak.WORK_INTS * (ap.n_work + ap.n_combine)
        assert used <= bound, (used, bound, n, num_cus)


def test_prepare_from_kept_hashes_equals_prepare_from_tokens():
    rng = np.random.default_rng(12)
    a = ak.BlockCache("arc", 200, 240, 16)
    b = ak.BlockCache("arc", 200, 240, 16)
    a.set_log(1 << 16)
    b.set_log(1 << 16)
    base = [rng.integers(0, 128256, int(n)).astype(np.int32) for n in (300, 700, 31, 16)]
    kept = [ak.hash_blocks(t) for t in base]
    packed = np.empty(1 << 16, dtype=np.int32)
    for step in range(30):
        pick = [int(x) for x in rng.choice(4, int(rng.integers(1, 4)), replace=False)]
        toks = [base[i] for i in pick]
        pa = a.prepare_batch(toks, 32, 8, 128, 256, packed)
        pb = np.empty(1 << 16, dtype=np.int32)
        st, d, pl, hb = b.prepare_native(None, 32, 8, 128, 256, pb,
                                         hashes=[kept[i] for i in pick], n_tokens=[len(t) for t in toks])
        assert st == _lib.OK
        assert d == pa.info
        assert np.array_equal(pb[:d["n_packed"]], pa.packed[:d["n_packed"]])
        assert np.array_equal(pl, pa.plan.prefix_lens) and np.array_equal(hb, pa.plan.hit_blocks)
        a.release_batch()
        b.release_batch()
    assert a.log() == b.log()


def test_kept_hashes_may_be_lists_of_large_ints_and_must_cover_the_blocks():
    # hashes above 2^63 passed as plain Python ints reach the library exactly, and a request
    # whose hash array is shorter than its full blocks is refused before any state changes
    toks = [np.arange(40, dtype=np.int32) + 7, np.arange(70, dtype=np.int32) * 3]
    hs = [ak.hash_blocks(t) for t in toks]
    big = [[int(x) | (1 << 63) for x in h] for h in hs]     # every identity >= 2^63
    packed = np.zeros(1 << 16, dtype=np.int32)
    a = ak.BlockCache("arc", 64, 80, 4)
    b = ak.BlockCache("arc", 64, 80, 4)
    ra = a.prepare_native(None, 8, 2, 64, 16, packed.copy(), hashes=[np.array(h, dtype=np.uint64) for h in big],
                          n_tokens=[40, 70])
    rb = b.prepare_native(None, 8, 2, 64, 16, packed.copy(), hashes=big, n_tokens=[40, 70])
    assert ra[0] == rb[0] == 0 and ra[1] == rb[1]
    assert (ra[2] == rb[2]).all() and (ra[3] == rb[3]).all()
    a.release_batch()
    b.release_batch()
    ka, pa = a.snapshot(ak.LIST_T1)
    kb, pb = b.snapshot(ak.LIST_T1)
    assert (ka == kb).all() and (pa == pb).all() and int(big[1][-1]) in ka.tolist()
    with pytest.raises(ValueError):
        b.prepare_native(None, 8, 2, 64, 16, packed.copy(), hashes=[big[0], big[1][:2]], n_tokens=[40, 70])
    kc, pc = b.snapshot(ak.LIST_T1)
    assert (kc == kb).all() and (pc == pb).all()
