"""ARC(c) over KV blocks (oracle).  TEST INFRASTRUCTURE ONLY.

The paper's evictor (Sec. 3, the two bullet points and Fig. 2) keeps

* T1: resident blocks seen once recently, T2: resident blocks seen at least
  twice (a hit promotes a block from T1 to T2);
* B1, B2: ghost lists holding only the identity of blocks evicted from T1, T2;
* p: the adaptive target size of T1.  A ghost hit in B1 means a larger T1
  would have hit, so p grows; a ghost hit in B2 shrinks it.  |T1| + |T2| is
  fixed at the capacity c once the cache has filled.

The paper defers the exact adaptation and learning rate to the ARC paper of
Megiddo and Modha (FAST 2003).  The four cases and REPLACE below restate that
published algorithm in this project's words:

Case I    x in T1 or T2: hit; move x to the MRU end of T2.
Case II   x in B1: p <- min(p + d1, c), d1 = 1 if |B1| >= |B2| else |B2|/|B1|;
          REPLACE; move x to T2 (MRU).
Case III  x in B2: p <- max(p - d2, 0), d2 = 1 if |B2| >= |B1| else |B1|/|B2|;
          REPLACE; move x to T2 (MRU).
Case IV   x in no list.
  IV-A    |T1| + |B1| == c: if |T1| < c drop the LRU entry of B1 then REPLACE,
          else drop the LRU page of T1 (no ghost).
  IV-B    |T1| + |B1| <  c: if the four lists hold >= c entries, drop the LRU
          entry of B2 when they hold 2c, then REPLACE.
          Then x goes to the MRU end of T1.
REPLACE   if T1 is non-empty and (|T1| > p, or x in B2 and |T1| == p) move the
          LRU page of T1 to the MRU end of B1, else the LRU page of T2 to B2.

Readings fixed by this project where the paper is silent:

* p is real-valued and updated in IEEE binary64; |T1| is compared with p
  exactly.
* A page used by the running batch is *pinned* and never chosen as a victim:
  REPLACE (and the IV-A T1 drop) take the LRU-most unpinned page of the list
  the rule selects; if that list has none they take the LRU-most unpinned page
  of the other list, and that page goes to the ghost list of the list it left.
* Physical placement: a page created by a miss takes the physical block of
  the page evicted by the same reference, else the head of a FIFO free list.

DBL (Sec. 4, the evaluated variant with a fixed 1:1 split between the recency and the
frequency queue) is the same policy with the adaptation switched off: p stays at c/2 and
ghost hits (Cases II and III) only move x and call REPLACE.  This is the fixed-target form
FRC_p of the ARC paper with p = c/2.

Length-aware victims (Sec. 6 names prompt length as a further eviction factor beside
recency and frequency; the rule is this project's reading, not the paper's): with a victim
window W > 1, every eviction from a resident list (REPLACE and the IV-A T1 drop) takes,
among the W least recently used unpinned pages of that list, the page at the greatest
depth (its block index in the prompt that referenced it), the less recent one on ties.
Which list loses a page, the ghost lists and p follow the rules above unchanged; W = 1 is
the plain policy.  Losing the block at depth k makes the next request on that chain
recompute blocks k onwards, so among recently similar pages the deepest is the cheapest loss.

Every reference is appended to a decision log (``Event``) so that another
implementation can be compared decision by decision.
"""

from __future__ import annotations

from collections import OrderedDict, deque
from dataclasses import dataclass

# case codes (shared numbering with the C ABI, which is an interface, not code)
CASE_I, CASE_II, CASE_III, CASE_IVA, CASE_IVA_T1DEL, CASE_IVB, LRU_HIT, LRU_MISS = range(8)
CASE_NAMES = ["I", "II", "III", "IVA", "IVA_T1DEL", "IVB", "LRU_HIT", "LRU_MISS"]
FROM_NONE, FROM_T1, FROM_T2, FROM_B1, FROM_B2 = range(5)
NO_HASH = 0


def window_victim(lst, pinned, depth, window: int):
    """The page an eviction takes from ``lst`` (keys in LRU -> MRU order): the deepest of the
    ``window`` least recently used unpinned pages, the less recent on ties (window 1: the
    LRU-most unpinned page); None if every page is pinned."""
    best, seen = None, 0
    for key in lst:
        if key in pinned:
            continue
        if best is None or depth.get(key, 0) > depth.get(best, 0):
            best = key
        seen += 1
        if seen == window:
            break
    return best


@dataclass(frozen=True)
class Event:
    """One policy reference, as the decision log records it."""
    key: int            # block identity referenced
    case: int           # CASE_*
    evicted: int        # identity of the page evicted by this reference (0 if none)
    evicted_from: int   # FROM_T1 / FROM_T2 / FROM_NONE
    dropped: int        # ghost (or IV-A T1 page) dropped from the history (0 if none)
    dropped_from: int   # FROM_B1 / FROM_B2 / FROM_T1 / FROM_NONE
    phys: int           # physical block of x after the reference
    p_after: float      # adaptive target after the reference


class ARC:
    """ARC(c) with pins and physical block placement (adaptive=False: DBL, p fixed at c/2)."""

    def __init__(self, capacity: int, free_blocks, adaptive: bool = True, window: int = 1,
                 fixed_p: float | None = None):
        """adaptive=False: the fixed-target form, p = fixed_p (c/2 when None: DBL)."""
        if capacity < 1 or window < 1:
            raise ValueError("capacity and window must be >= 1")
        self.c = int(capacity)
        self.adaptive = adaptive
        self.window = int(window)
        self.depth: dict[int, int] = {}       # block index of each key in its prompt
        self.p = 0.0 if adaptive else (self.c / 2.0 if fixed_p is None else float(fixed_p))
        if not 0.0 <= self.p <= self.c:
            raise ValueError("fixed p must lie in [0, c]")
        # OrderedDicts in LRU -> MRU order; resident lists map key -> physical block.
        self.T1: OrderedDict[int, int] = OrderedDict()
        self.T2: OrderedDict[int, int] = OrderedDict()
        self.B1: OrderedDict[int, None] = OrderedDict()
        self.B2: OrderedDict[int, None] = OrderedDict()
        self.free = deque(int(b) for b in free_blocks)
        self.pinned: set[int] = set()
        self.log: list[Event] = []

    # -- queries -------------------------------------------------------------
    def resident(self, key: int) -> bool:
        return key in self.T1 or key in self.T2

    def phys_of(self, key: int) -> int:
        return self.T1[key] if key in self.T1 else self.T2[key]

    def snapshot(self):
        return (list(self.T1), list(self.T2), list(self.B1), list(self.B2), self.p)

    def pin(self, key: int) -> None:
        assert self.resident(key)
        self.pinned.add(key)

    def unpin_all(self) -> None:
        self.pinned.clear()

    # -- helpers -------------------------------------------------------------
    def _lru_unpinned(self, lst: OrderedDict):
        return window_victim(lst, self.pinned, self.depth, self.window)

    def _replace(self, x_in_b2: bool):
        """Evict one resident page to its ghost list; return (key, from, phys)."""
        n1 = len(self.T1)
        prefer_t1 = n1 > 0 and (n1 > self.p or (x_in_b2 and n1 == self.p))
        order = [(self.T1, self.B1, FROM_T1), (self.T2, self.B2, FROM_T2)]
        if not prefer_t1:
            order.reverse()
        for src, ghost, tag in order:
            victim = self._lru_unpinned(src)
            if victim is not None:
                phys = src.pop(victim)
                ghost[victim] = None
                return victim, tag, phys
        raise RuntimeError("REPLACE found no unpinned resident page")

    # -- one reference ---------------------------------------------------------
    def reference(self, x: int, depth: int = 0) -> Event:
        c = self.c
        evicted, evicted_from = NO_HASH, FROM_NONE
        dropped, dropped_from = NO_HASH, FROM_NONE
        if x in self.T1 or x in self.T2:                       # Case I
            phys = self.T1.pop(x) if x in self.T1 else self.T2.pop(x)
            self.T2[x] = phys
            case = CASE_I
        elif x in self.B1:                                     # Case II
            if self.adaptive:
                d1 = 1.0 if len(self.B1) >= len(self.B2) else len(self.B2) / len(self.B1)
                self.p = min(self.p + d1, float(c))
            evicted, evicted_from, phys = self._replace(False)
            del self.B1[x]
            self.T2[x] = phys
            case = CASE_II
        elif x in self.B2:                                     # Case III
            if self.adaptive:
                d2 = 1.0 if len(self.B2) >= len(self.B1) else len(self.B1) / len(self.B2)
                self.p = max(self.p - d2, 0.0)
            evicted, evicted_from, phys = self._replace(True)
            del self.B2[x]
            self.T2[x] = phys
            case = CASE_III
        else:                                                  # Case IV
            if len(self.T1) + len(self.B1) == c:
                if len(self.T1) < c:                           # IV-A
                    dropped = next(iter(self.B1))
                    del self.B1[dropped]
                    dropped_from = FROM_B1
                    evicted, evicted_from, phys = self._replace(False)
                    case = CASE_IVA
                else:                                          # IV-A, T1 full
                    victim = self._lru_unpinned(self.T1)
                    if victim is None:
                        raise RuntimeError("IV-A: every T1 page is pinned")
                    phys = self.T1.pop(victim)
                    dropped, dropped_from = victim, FROM_T1
                    case = CASE_IVA_T1DEL
            else:                                              # IV-B
                total = len(self.T1) + len(self.T2) + len(self.B1) + len(self.B2)
                if total >= c:
                    if total == 2 * c:
                        dropped = next(iter(self.B2))
                        del self.B2[dropped]
                        dropped_from = FROM_B2
                    evicted, evicted_from, phys = self._replace(False)
                else:
                    if not self.free:
                        raise RuntimeError("free list exhausted")
                    phys = self.free.popleft()
                case = CASE_IVB
            self.T1[x] = phys
        self.depth[x] = int(depth)
        ev = Event(x, case, evicted, evicted_from, dropped, dropped_from, phys, self.p)
        self.log.append(ev)
        return ev

    def check_invariants(self) -> None:
        """The published ARC invariants (counts) plus 0 <= p <= c and disjointness."""
        c = self.c
        n1, n2, m1, m2 = len(self.T1), len(self.T2), len(self.B1), len(self.B2)
        keys = [set(self.T1), set(self.T2), set(self.B1), set(self.B2)]
        for i in range(4):
            for j in range(i + 1, 4):
                assert not (keys[i] & keys[j]), "lists not disjoint"
        assert n1 + n2 <= c
        assert n1 + m1 <= c
        assert n1 + n2 + m1 + m2 <= 2 * c
        assert 0.0 <= self.p <= c
        if n1 + n2 + m1 + m2 < c:
            assert m1 == 0 and m2 == 0
        else:
            assert n1 + n2 == c
