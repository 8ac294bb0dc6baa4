"""Pins of the oracle's ARC and LRU policies (CPU only).

ARC: hand-derived traces (tests/golden/arc_traces.json), the published
invariants, the paper's qualitative claims (Sec. 3: promotion on a hit, ghost
hits steer p, flush resistance, fixed |T1|+|T2|), and the optimality bound
(no online policy beats Belady's MIN, computed by brute force).
LRU: an independent naive list implementation and the inclusion property.
"""

import json
import os
import random

import pytest
from hypothesis import given, settings, strategies as st

from oracle.arc import ARC, CASE_NAMES, CASE_I, CASE_II, CASE_III, FROM_NONE, FROM_T1, FROM_T2
from oracle.lru import LRU

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "arc_traces.json")
TRACES = json.load(open(GOLDEN))["traces"]


def key(ch):
    return ord(ch)


def names(keys):
    return "".join(chr(k) for k in keys)


def run_arc(refs, c):
    a = ARC(c, range(1000, 1000 + c))
    hits = 0
    for ch in refs:
        ev = a.reference(key(ch))
        hits += ev.case == CASE_I
        a.check_invariants()
    return a, hits


DBL_TRACES = json.load(open(GOLDEN))["dbl_traces"]


@pytest.mark.parametrize("tr", DBL_TRACES, ids=lambda t: f"dbl_c{t['c']}_{t['refs']}")
def test_dbl_hand_derived_trace(tr):
    a = ARC(tr["c"], range(1000, 1000 + tr["c"]), adaptive=False)
    hits = 0
    for ch in tr["refs"]:
        ev = a.reference(key(ch))
        hits += ev.case == CASE_I
        a.check_invariants()
    assert [CASE_NAMES[e.case] for e in a.log] == tr["cases"]
    assert [chr(e.evicted) if e.evicted_from != FROM_NONE else "" for e in a.log] == tr["evicted"]
    assert [e.p_after for e in a.log] == [float(x) for x in tr["p"]]
    assert hits == tr["hits"]
    T1, T2, B1, B2, p = a.snapshot()
    assert (names(T1), names(T2), names(B1), names(B2), p) == (tr["T1"], tr["T2"], tr["B1"], tr["B2"], tr["p_final"])


def test_dbl_keeps_p_at_half_capacity_and_the_invariants():
    rng = random.Random(4)
    for c in (1, 2, 5, 16):
        a = ARC(c, range(100000), adaptive=False)
        for _ in range(3000):
            a.reference(rng.randrange(3 * c))
            a.check_invariants()
            assert a.p == c / 2
        assert any(e.case in (CASE_II, CASE_III) for e in a.log)    # ghost hits happened


@pytest.mark.parametrize("tr", TRACES, ids=lambda t: f"c{t['c']}_{t['refs']}")
def test_arc_hand_derived_trace(tr):
    a, hits = run_arc(tr["refs"], tr["c"])
    assert [CASE_NAMES[e.case] for e in a.log] == tr["cases"]
    assert [chr(e.evicted) if e.evicted_from != FROM_NONE else "" for e in a.log] == tr["evicted"]
    if "dropped" in tr:
        assert [chr(e.dropped) if e.dropped_from != FROM_NONE else "" for e in a.log] == tr["dropped"]
    assert [e.p_after for e in a.log] == [float(x) for x in tr["p"]]
    assert hits == tr["hits"]
    T1, T2, B1, B2, p = a.snapshot()
    assert (names(T1), names(T2), names(B1), names(B2)) == (tr["T1"], tr["T2"], tr["B1"], tr["B2"])
    assert p == tr["p_final"]


def test_lru_hand_derived_trace():
    tr = TRACES[0]
    lru = LRU(tr["c"], range(tr["c"]))
    hits = sum(lru.reference(key(ch)).case == 6 for ch in tr["refs"])
    assert hits == tr["lru_hits"]
    assert names(lru.snapshot()[0]) == tr["lru_final"]


def test_physical_blocks_are_reused_by_the_inserting_page():
    a = ARC(2, [7, 9])
    assert a.reference(1).phys == 7
    assert a.reference(2).phys == 9
    ev = a.reference(3)             # |T1| = c: IV-A drops 1 (LRU of T1, no ghost); its block goes to 3
    assert CASE_NAMES[ev.case] == "IVA_T1DEL" and ev.dropped == 1 and ev.phys == 7
    assert a.reference(2).case == CASE_I
    ev = a.reference(4)             # |T1| = 1 > p = 0: REPLACE moves 3 to B1; 4 takes its block
    assert ev.evicted == 3 and ev.evicted_from == FROM_T1 and ev.phys == 7 and 3 in a.B1
    resident_phys = sorted(list(a.T1.values()) + list(a.T2.values()))
    assert resident_phys == [7, 9]


# ---------------------------------------------------------------------------------------------
# invariants and qualitative properties
# ---------------------------------------------------------------------------------------------

@settings(max_examples=150, deadline=None)
@given(c=st.integers(1, 9), refs=st.lists(st.integers(0, 25), min_size=0, max_size=300))
def test_arc_invariants_random(c, refs):
    a = ARC(c, range(c))
    for x in refs:
        p0 = a.p
        ev = a.reference(x)
        a.check_invariants()
        if ev.case == CASE_II:
            assert ev.p_after >= p0             # B1 ghost hit: invest more in T1 (Sec. 3)
        elif ev.case == CASE_III:
            assert ev.p_after <= p0             # B2 ghost hit: invest more in T2
        else:
            assert ev.p_after == p0
        # physical blocks of resident pages stay a set of distinct pool blocks
        ph = list(a.T1.values()) + list(a.T2.values())
        assert len(set(ph)) == len(ph)


@settings(max_examples=60, deadline=None)
@given(c=st.integers(2, 8), refs=st.lists(st.integers(0, 20), min_size=1, max_size=200),
       seed=st.integers(0, 10**6))
def test_arc_with_pins_never_evicts_a_pinned_page(c, refs, seed):
    rng = random.Random(seed)
    a = ARC(c, range(c))
    for x in refs:
        # pin a random subset of residents, leaving at least one unpinned
        res = list(a.T1) + list(a.T2)
        a.unpin_all()
        if len(res) >= 2:
            for k in rng.sample(res, rng.randint(0, len(res) - 1)):
                if k != x:
                    a.pin(k)
        pinned = set(a.pinned)
        ev = a.reference(x)
        assert ev.evicted_from == FROM_NONE or ev.evicted not in pinned
        assert ev.dropped_from == FROM_NONE or ev.dropped not in pinned
        a.check_invariants()


def belady_hits(refs, c):
    """Optimal offline demand paging (evict the page reused farthest in the future)."""
    cache, hits = set(), 0
    for i, x in enumerate(refs):
        if x in cache:
            hits += 1
            continue
        if len(cache) == c:
            def next_use(y):
                for j in range(i + 1, len(refs)):
                    if refs[j] == y:
                        return j
                return 1 << 30
            cache.remove(max(cache, key=next_use))
        cache.add(x)
    return hits


@settings(max_examples=150, deadline=None)
@given(c=st.integers(1, 6), refs=st.lists(st.integers(0, 12), min_size=0, max_size=60))
def test_arc_and_lru_never_beat_belady(c, refs):
    a = ARC(c, range(c))
    lru = LRU(c, range(c))
    ah = sum(a.reference(x).case == CASE_I for x in refs)
    lh = sum(lru.reference(x).case == 6 for x in refs)
    opt = belady_hits(refs, c)
    assert ah <= opt and lh <= opt


def test_pure_scan_never_hits():
    a = ARC(8, range(8))
    assert all(a.reference(x).case != CASE_I for x in range(1000))


def test_cycle_within_capacity_hits_after_first_pass():
    c = 10
    for n in (1, 5, 10):
        a = ARC(c, range(c))
        cases = [a.reference(x % n).case for x in range(5 * n)]
        assert all(cs != CASE_I for cs in cases[:n])
        assert all(cs == CASE_I for cs in cases[n:])


def test_flush_resistance():
    # A frequently used working set lives in T2; a long scan of never-seen blocks
    # (no ghost hits) then clears T1 but keeps most of T2 (Sec. 3).
    c = 32
    a = ARC(c, range(c))
    hot = list(range(24))
    for _ in range(3):
        for x in hot:
            a.reference(x)
    p0 = a.p
    for x in range(10**6, 10**6 + 5000):
        a.reference(x)
    assert a.p == p0                              # no ghost hit during the scan -> p unchanged
    # T1 grows only while |T1| <= p; once |T1| > p every REPLACE takes from T1,
    # so T2 loses pages only until T1 holds floor(p) + 1 of them.
    assert len(a.T1) + len(a.T2) == c
    assert set(a.T2) <= set(hot)
    assert len(a.T2) >= min(len(hot), c - int(p0) - 1)
    assert set(a.T2) == set(hot)                  # here |T1| = 8 > p = 0 when the cache fills


def test_lru_flushes_under_the_same_scan():
    c = 32
    lru = LRU(c, range(c))
    for _ in range(3):
        for x in range(24):
            lru.reference(x)
    for x in range(10**6, 10**6 + 5000):
        lru.reference(x)
    assert not (set(lru.L) & set(range(24)))


def naive_lru_hits(refs, c):
    lst, hits = [], 0
    for x in refs:
        if x in lst:
            hits += 1
            lst.remove(x)
        elif len(lst) == c:
            lst.pop(0)
        lst.append(x)
    return hits, lst


@settings(max_examples=150, deadline=None)
@given(c=st.integers(1, 8), refs=st.lists(st.integers(0, 15), max_size=200))
def test_lru_matches_naive_list_and_inclusion(c, refs):
    lru = LRU(c, range(c))
    hits = sum(lru.reference(x).case == 6 for x in refs)
    nh, lst = naive_lru_hits(refs, c)
    assert hits == nh and list(lru.L) == lst
    assert naive_lru_hits(refs, c + 1)[0] >= hits   # stack property of LRU


def test_ghost_hits_move_to_t2_and_t1_hit_promotes():
    a = ARC(3, range(3))
    for x in (1, 2, 3):
        a.reference(x)
    assert a.reference(2).case == CASE_I and 2 in a.T2 and 2 not in a.T1
    a.reference(4)                                # evicts 1 -> B1
    assert 1 in a.B1
    ev = a.reference(1)
    assert ev.case == CASE_II and 1 in a.T2 and ev.evicted_from in (FROM_T1, FROM_T2)
