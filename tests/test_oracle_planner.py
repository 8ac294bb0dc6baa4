"""Pins of the oracle's batch planner and KV pool (CPU only)."""

import numpy as np
import pytest

from oracle import blockhash as bh
from oracle import kvpool
from oracle.arc import CASE_I, CASE_IVB
from oracle.planner import Planner, PlanError, form_batches
from workloads import get_config
from workloads.streams import (Source, make_request, stream_tiny, free_order, KIND_DOC,
                               KIND_QUESTION)


def reqs_of(requests):
    return [(bh.hash_blocks(r.tokens), r.n_tokens) for r in requests]


def test_tiny_config_expectation():
    # Warm request (256 doc tokens) then the same document + 64 new tokens:
    # 16 misses all in T1, then k = 16, P = 256, S = 64; the four new blocks take
    # free-list entries 16..19 in tail-first order; the 16 hits move to T2.
    cfg = get_config("tiny")
    order = free_order(cfg.seed, cfg.num_phys)
    pl = Planner("arc", cfg.capacity, cfg.num_phys, cfg.scratch, order)
    r0, r1 = stream_tiny(cfg)
    p0 = pl.plan_batch(reqs_of([r0]))
    pl.release_batch()
    log0 = pl.cache.log[p0.events_begin:p0.events_end]
    assert [e.case for e in log0] == [CASE_IVB] * 16
    assert p0.hit_blocks == [0] and p0.prefix_lens == [0] and p0.cu_q == [0, 256]
    assert p0.block_tables[0] == [int(order[15 - i]) for i in range(16)]
    assert len(pl.cache.T1) == 16 and len(pl.cache.T2) == 0

    p1 = pl.plan_batch(reqs_of([r1]))
    pl.release_batch()
    assert p1.hit_blocks == [16] and p1.prefix_lens == [256] and p1.cu_q == [0, 64]
    row = p1.block_tables[0]
    assert row[:16] == p0.block_tables[0]
    assert row[16:] == [int(order[19]), int(order[18]), int(order[17]), int(order[16])]
    log1 = pl.cache.log[p1.events_begin:p1.events_end]
    assert [e.case for e in log1] == [CASE_IVB] * 4 + [CASE_I] * 16
    assert (len(pl.cache.T1), len(pl.cache.T2), pl.cache.p) == (4, 16, 0.0)
    assert p1.slot_mapping == [row[j // 16] * 16 + j % 16 for j in range(256, 320)]
    t = pl.totals
    assert t.prefix_hit_tokens == 256 and t.prompt_tokens == 576


def _doc_req(cfg, doc, n_doc, qi=None, n_q=0):
    segs = [(Source(KIND_DOC, doc, n_doc), 0, n_doc)]
    if n_q:
        segs.append((Source(KIND_QUESTION, qi, n_q), 0, n_q))
    return make_request(cfg, segs)


def test_intra_batch_reuse_partial_tail_and_full_hit():
    cfg = get_config("tiny")
    pl = Planner("arc", 64, 80, 16)
    a = _doc_req(cfg, 5, 100)                 # 6 full blocks + 4-token tail
    b = _doc_req(cfg, 5, 96)                  # the same 6 full blocks, no tail
    plan = pl.plan_batch(reqs_of([a, b]))
    assert plan.hit_blocks == [0, 5]          # b hits a's blocks; whole prompt cached -> recompute last
    assert plan.prefix_lens == [0, 80] and plan.cu_q == [0, 100, 116]
    ra, rb = plan.block_tables
    assert len(ra) == 7 and len(rb) == 6 and ra[:6] == rb
    assert ra[6] in range(64, 80)             # tail from the scratch region
    pl.release_batch()
    assert list(pl.scratch)[-1] == ra[6]      # returned to the scratch FIFO tail


def test_errors_and_call_order():
    cfg = get_config("tiny")
    pl = Planner("arc", 8, 16, 4)
    big = _doc_req(cfg, 1, 16 * 9)
    with pytest.raises(PlanError) as e:
        pl.plan_batch(reqs_of([big]))
    assert e.value.code == "ENOSPC"
    with pytest.raises(PlanError) as e:
        pl.release_batch()
    assert e.value.code == "ESTATE"
    r = _doc_req(cfg, 2, 40)
    with pytest.raises(PlanError) as e:
        pl.plan_batch([(bh.hash_blocks(r.tokens)[:1], r.n_tokens)])
    assert e.value.code == "EINVAL"
    pl.plan_batch(reqs_of([r]))
    with pytest.raises(PlanError) as e:
        pl.plan_batch(reqs_of([r]))
    assert e.value.code == "ESTATE"
    pl.release_batch()
    tails = [_doc_req(cfg, 10 + i, 17) for i in range(5)]
    with pytest.raises(PlanError) as e:
        pl.plan_batch(reqs_of(tails))         # 5 partial tails, 4 scratch blocks
    assert e.value.code == "ENOSPC"


def test_form_batches():
    assert form_batches([160, 160, 160], 8, 20, 4) == [(0, 2), (2, 3)]
    assert form_batches([16] * 5, 2, 100, 4) == [(0, 2), (2, 4), (4, 5)]
    assert form_batches([17] * 3, 8, 100, 2) == [(0, 2), (2, 3)]
    with pytest.raises(PlanError):
        form_batches([16 * 30], 8, 20, 4)


def test_orphan_block_keeps_its_physical_block():
    # c = 4, head-first-free eviction pattern: warm doc blocks 0..2, push block 0 out,
    # then re-reference the doc: block 0 misses (k = 0), blocks 1 and 2 are resident orphans.
    cfg = get_config("tiny")
    pl = Planner("lru", 4, 8, 4)
    d = _doc_req(cfg, 3, 48)
    p = pl.plan_batch(reqs_of([d]))
    pl.release_batch()
    first = p.block_tables[0]
    h = bh.hash_blocks(d.tokens)
    # LRU order after tail-first references: [h2, h1, h0]; touch h1, h2 so h0 is LRU
    x = _doc_req(cfg, 4, 16)
    pl.plan_batch([(bh.hash_blocks(x.tokens), 16)])
    pl.release_batch()
    pl.cache.reference(h[1]); pl.cache.reference(h[2])
    y = _doc_req(cfg, 6, 16)
    pl.plan_batch([(bh.hash_blocks(y.tokens), 16)])   # evicts h0
    pl.release_batch()
    assert not pl.cache.resident(h[0]) and pl.cache.resident(h[1]) and pl.cache.resident(h[2])
    p2 = pl.plan_batch(reqs_of([d]))
    pl.release_batch()
    assert p2.hit_blocks == [0]
    assert p2.block_tables[0][1:] == first[1:]           # orphans keep their blocks
    assert p2.slot_mapping[16:] == [first[j // 16] * 16 + j % 16 for j in range(16, 48)]


def test_pool_gather_reproduces_every_visible_token():
    # Scatter pin: run a small eviction-heavy stream through planner + scatter; after each
    # batch, gathering each request through its block table returns its K/V bit-exactly.
    cfg = get_config("tiny")
    rng = np.random.default_rng(7)
    hkv, d = 2, 8
    pl = Planner("arc", 24, 40, 8, order := rng.permutation(40))
    kp, vp = kvpool.new_pool(40, hkv, d)

    def src_kv(doc, n):                        # deterministic per (doc, position)
        g = np.random.default_rng(1000 + doc)
        k = g.integers(0, 1 << 16, (96, hkv, d), dtype=np.uint16)
        v = g.integers(0, 1 << 16, (96, hkv, d), dtype=np.uint16)
        return k[:n], v[:n]

    for step in range(40):
        docs = rng.integers(0, 6, size=rng.integers(1, 3))
        lens = rng.integers(1, 90, size=len(docs))
        reqs = [_doc_req(cfg, int(dd), int(n)) for dd, n in zip(docs, lens)]
        if sum(r.n_tokens // 16 for r in reqs) > 24:
            continue
        plan = pl.plan_batch(reqs_of(reqs))
        knew = np.concatenate([src_kv(int(dd), int(n))[0][p:] for dd, n, p in
                               zip(docs, lens, plan.prefix_lens)])
        vnew = np.concatenate([src_kv(int(dd), int(n))[1][p:] for dd, n, p in
                               zip(docs, lens, plan.prefix_lens)])
        kvpool.scatter(kp, vp, knew, vnew, plan.slot_mapping)
        for r, (dd, n) in enumerate(zip(docs, lens)):
            k, v = kvpool.gather(kp, vp, plan.block_tables[r], int(n))
            ek, ev = src_kv(int(dd), int(n))
            assert np.array_equal(k, ek) and np.array_equal(v, ev)
        pl.release_batch()
        pl.cache.check_invariants()
    assert pl.totals.prefix_hit_tokens > 0
    assert pl.totals.case_counts[CASE_I] > 0


def _planner_cases():
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "planner_cases.json")))
    out = []
    for case in g["cases"]:
        for var in case.get("variants", [{"intra_batch_reuse": case.get("intra_batch_reuse", True)}]):
            out.append(pytest.param(case, var, id=f"{case['name']}-reuse{int(var['intra_batch_reuse'])}"))
    return out


@pytest.mark.parametrize("case,var", _planner_cases())
def test_hand_derived_plans(case, var):
    """Hand-derived plans (tests/golden/planner_cases.json): prefix pages pinned before the
    tail-first references, the scratch FIFO's order, and a B2 ghost hit counting as a page made
    in the batch when intra-batch reuse is off."""
    from oracle.arc import CASE_NAMES
    pl = Planner(case["policy"], case["capacity"], case["num_phys"], case["scratch"],
                 intra_batch_reuse=var["intra_batch_reuse"])
    for bi, b in enumerate(case["batches"]):
        n0 = len(pl.cache.log)
        plan = pl.plan_batch([(list(h), n) for h, n in b["reqs"]])
        assert plan.block_tables == b["tables"], bi
        want_hits = var["last_hit_blocks"] if (bi == len(case["batches"]) - 1 and "last_hit_blocks" in var) \
            else b["hit_blocks"]
        assert plan.hit_blocks == want_hits, bi
        evs = pl.cache.log[n0:]
        if "cases" in b:
            assert [CASE_NAMES[e.case] for e in evs] == b["cases"]
        if "dropped" in b:
            assert [e.dropped for e in evs] == b["dropped"]
        pl.release_batch()
    T1, T2, B1, B2, p = pl.cache.snapshot()
    f = case["final"]
    assert (list(T1), list(T2), list(B1), list(B2), p) == (f["T1"], f["T2"], f["B1"], f["B2"], f["p"])
