"""Pins of the length-aware victim window (oracle, CPU only).

The rule (a reading of Sec. 6's call to weigh prompt length beside recency and frequency):
an eviction from a resident list takes the deepest of its W least recently used unpinned
pages, the less recent one on ties; W = 1 is the plain policy, whose traces are pinned
elsewhere.  Checked here against hand-derived traces, a brute-force list simulation of LRU
with an unbounded window, pins, and the ARC invariants.
"""

import numpy as np

from oracle.arc import ARC, CASE_I, CASE_II, CASE_IVA_T1DEL, CASE_IVB, FROM_T1
from oracle.lru import LRU

A, B, C, D = 101, 102, 103, 104


def test_lru_window_two_evicts_the_deeper_of_the_two_oldest():
    # c = 3; depths A 0, B 5, C 1.  D needs a page: W = 1 takes A (LRU-most), W = 2 takes
    # B (deeper of A, B).  Then A hits only under W = 2.
    for w, victim, a_hits in ((1, A, False), (2, B, True)):
        lru = LRU(3, range(10), window=w)
        for k, d in ((A, 0), (B, 5), (C, 1)):
            lru.reference(k, depth=d)
        ev = lru.reference(D, depth=2)
        assert (ev.evicted, ev.evicted_from) == (victim, FROM_T1)
        assert lru.resident(A) == a_hits
        assert list(lru.L) == [k for k in (A, B, C, D) if k != victim]


def test_arc_window_in_replace_and_in_the_t1_drop():
    # REPLACE: c = 3; A0 B1 C5 fill T1; A again goes to T2; D misses with |T1| = 2 > p = 0,
    # so T1 gives a page: W = 1 takes B (LRU-most), W = 2 takes C (depth 5 over B's 1).
    # A later C is then a Case I hit (W = 1) or a B1 ghost hit that raises p to 1 (W = 2).
    for w, victim, c_case, p_after in ((1, B, CASE_I, 0.0), (2, C, CASE_II, 1.0)):
        arc = ARC(3, range(10), window=w)
        for k, d in ((A, 0), (B, 1), (C, 5), (A, 0)):
            arc.reference(k, depth=d)
        ev = arc.reference(D, depth=2)
        assert ev.case == CASE_IVB and (ev.evicted, ev.evicted_from) == (victim, FROM_T1)
        assert list(arc.B1) == [victim]
        ev = arc.reference(C, depth=5)
        assert ev.case == c_case and ev.p_after == p_after
    # IV-A with |T1| = c drops a T1 page without a ghost: c = 2, A0 B4, then C: W = 2 drops B
    for w, dropped in ((1, A), (2, B)):
        arc = ARC(2, range(10), window=w)
        arc.reference(A, depth=0)
        arc.reference(B, depth=4)
        ev = arc.reference(C, depth=1)
        assert ev.case == CASE_IVA_T1DEL and (ev.dropped, ev.dropped_from) == (dropped, FROM_T1)
        assert not arc.B1


def test_window_skips_pinned_pages():
    # T1 = [B(1), C(5)] with C pinned: W = 2 looks at unpinned pages only and takes B
    arc = ARC(3, range(10), window=2)
    for k, d in ((A, 0), (B, 1), (C, 5), (A, 0)):
        arc.reference(k, depth=d)
    arc.pin(C)
    ev = arc.reference(D, depth=2)
    assert ev.evicted == B and arc.resident(C)
    arc.unpin_all()
    lru = LRU(2, range(10), window=8)
    lru.reference(A, depth=9)
    lru.reference(B, depth=1)
    lru.pin(A)
    assert lru.reference(C, depth=0).evicted == B


def test_unbounded_window_lru_matches_a_brute_force_list():
    # W >= c: LRU evicts the deepest resident page (least recent among equals).  Brute force:
    # a plain list in recency order, scanned for the maximum depth.
    rng = np.random.default_rng(7)
    c = 6
    lru = LRU(c, range(100), window=c)
    order, depth = [], {}
    for _ in range(400):
        k = int(rng.integers(0, 15))
        d = k % 5                       # a key keeps its depth, as a chained hash does
        ev = lru.reference(k, depth=d)
        if k in order:
            order.remove(k)
            assert ev.evicted == 0
        elif len(order) == c:
            v = max(order, key=lambda x: (depth[x], -order.index(x)))
            order.remove(v)
            assert ev.evicted == v
        order.append(k)
        depth[k] = d
        assert list(lru.L) == order


def test_arc_invariants_hold_with_windows():
    rng = np.random.default_rng(3)
    for w in (2, 5, 64):
        for adaptive in (True, False):
            arc = ARC(12, range(100), adaptive=adaptive, window=w)
            for _ in range(2000):
                k = int(rng.zipf(1.3)) % 60
                arc.reference(k, depth=k % 17)
                arc.check_invariants()
                assert 0.0 <= arc.p <= 12


def test_planner_hands_each_block_its_depth():
    # LRU, c = 3, head-first references: a 3-block prompt leaves x0, x1, x2 (depths 0, 1, 2) in
    # LRU -> MRU order.  A new block then evicts the LRU-most page x0 with W = 1 and the deepest,
    # x2, with W = 3.
    from oracle import blockhash as obh
    from oracle.planner import Planner
    x = np.arange(48 + 1, dtype=np.int32)
    y = np.arange(16 + 1, dtype=np.int32) + 5000
    hx = obh.hash_blocks(x)
    for w, gone in ((1, 0), (3, 2)):
        pl = Planner("lru", 3, 8, 4, ref_order="head_first", victim_window=w)
        pl.plan_batch([(hx, len(x))])
        pl.release_batch()
        assert list(pl.cache.L) == list(hx)
        pl.plan_batch([(obh.hash_blocks(y), len(y))])
        pl.release_batch()
        assert pl.cache.log[-1].evicted == hx[gone]
