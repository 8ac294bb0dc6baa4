"""Pins of the fixed-target policy FRC_p and of planning without intra-batch reuse (oracle,
CPU only), by hand-derived traces and by reduction to the pinned DBL."""

import numpy as np

from oracle.arc import ARC, CASE_I, CASE_II, CASE_IVB, FROM_T1, FROM_T2
from oracle.planner import Planner

A, B, C = 11, 12, 13


def test_frc_at_zero_against_arc_on_a_ghost_hit():
    # c = 2, trace A B A C B.  Both start with p = 0: C evicts B from T1 (|T1| = 1 > 0).
    # B is then a B1 ghost hit: ARC raises p to 1 and REPLACE takes A from T2 (|T1| = 1 is
    # not > 1); FRC keeps p = 0 and takes C from T1.
    want = {
        "arc": ((A, FROM_T2), 1.0, ([C], [B], [], [A])),
        "frc0": ((C, FROM_T1), 0.0, ([], [A, B], [C], [])),
    }
    for name, adaptive in (("arc", True), ("frc0", False)):
        cache = ARC(2, range(8), adaptive=adaptive, fixed_p=None if adaptive else 0.0)
        cases = [cache.reference(k).case for k in (A, B, A, C)]
        assert cases == [CASE_IVB, CASE_IVB, CASE_I, CASE_IVB]
        ev = cache.reference(B)
        (victim, frm), p, lists = want[name]
        assert ev.case == CASE_II and (ev.evicted, ev.evicted_from) == (victim, frm)
        assert cache.p == p
        assert tuple(map(list, cache.snapshot()[:4])) == lists


def test_frc_at_half_c_is_dbl():
    rng = np.random.default_rng(2)
    for c in (5, 8, 13):
        dbl = ARC(c, range(100), adaptive=False)
        frc = ARC(c, range(100), adaptive=False, fixed_p=c / 2)
        for _ in range(1500):
            k = int(rng.zipf(1.2)) % 40
            assert dbl.reference(k) == frc.reference(k)
        for f in (2, 3):
            frc = ARC(c, range(100), adaptive=False, fixed_p=c / f)
            for _ in range(300):
                frc.reference(int(rng.integers(0, 30)))
                frc.check_invariants()
                assert frc.p == c / f


def test_no_intra_batch_reuse_recomputes_a_prefix_made_in_the_same_batch():
    # a cold batch with the same 32-token prompt twice (two full blocks)
    toks = list(range(32))
    from oracle import blockhash as obh
    h = obh.hash_blocks(np.array(toks, dtype=np.int32))
    for reuse, k2 in ((True, 1), (False, 0)):
        pl = Planner("arc", 8, 16, 4, intra_batch_reuse=reuse)
        plan = pl.plan_batch([(h, 32), (h, 32)])
        # with reuse the whole prompt is cached for the second request: its last block is
        # recomputed (k = 1, P = 16); without, the blocks are this batch's own: k = 0
        assert plan.hit_blocks == [0, k2] and plan.prefix_lens == [0, 16 * k2]
        # either way both requests map their blocks to the same physical blocks
        assert plan.block_tables[0] == plan.block_tables[1]
        pl.release_batch()
        # in the next batch the blocks are old: reused in both modes
        plan = pl.plan_batch([(h, 32)])
        assert plan.hit_blocks == [1]
        pl.release_batch()


def test_a_page_back_from_a_ghost_list_counts_as_made_in_the_batch():
    # c = 2, one full block + a partial tail per request:
    #   [B] -> T1 = [B]; [D] -> T1 = [B, D]; [D] again -> D to T2; [E]: |T1| + |B1| = 1 < c
    #   with 2 pages resident, so REPLACE (|T1| = 1 > p = 0) moves B to B1.
    # Then one batch [B + 3 tokens], [B + 5 tokens]: the first references B as a B1 ghost hit
    # (Case II), which brings it back in this batch.  With reuse the second request hits it
    # (k = 1); without, its prefix stops there (k = 0).
    from oracle import blockhash as obh
    blk = {name: np.arange(16, dtype=np.int32) + 100 * i for i, name in enumerate("BDE")}

    def req(name, tail):
        t = np.concatenate([blk[name], np.arange(tail, dtype=np.int32) + 9000 + tail])
        return obh.hash_blocks(t), len(t)

    for reuse, want in ((True, [0, 1]), (False, [0, 0])):
        pl = Planner("arc", 2, 8, 4, intra_batch_reuse=reuse)
        for name in "BDDE":
            pl.plan_batch([req(name, 3)])
            pl.release_batch()
        hb = obh.hash_blocks(blk["B"])[0]
        assert hb in pl.cache.B1 and not pl.cache.resident(hb)
        plan = pl.plan_batch([req("B", 3), req("B", 5)])
        assert plan.hit_blocks == want
        assert pl.cache.log[-2].case == CASE_II      # the first request's reference of B
        pl.release_batch()
