"""LRU over KV blocks (oracle).  TEST INFRASTRUCTURE ONLY.

The baseline the paper improves on: the serving engine evicts the
least-recently-used block when the cache is full (Sec. 1, Sec. 2 "cache
replacement", Sec. 4).  Same interface, pins and physical placement as
``oracle.arc.ARC`` so that the planner can run either.
"""

from __future__ import annotations

from collections import OrderedDict, deque

from .arc import Event, LRU_HIT, LRU_MISS, FROM_NONE, FROM_T1, NO_HASH, window_victim


class LRU:
    """window > 1: length-aware victims, as for ``oracle.arc.ARC``."""

    def __init__(self, capacity: int, free_blocks, window: int = 1):
        if capacity < 1 or window < 1:
            raise ValueError("capacity and window must be >= 1")
        self.c = int(capacity)
        self.window = int(window)
        self.depth: dict[int, int] = {}
        self.p = 0.0
        self.L: OrderedDict[int, int] = OrderedDict()    # LRU -> MRU, key -> phys
        self.free = deque(int(b) for b in free_blocks)
        self.pinned: set[int] = set()
        self.log: list[Event] = []

    def resident(self, key: int) -> bool:
        return key in self.L

    def phys_of(self, key: int) -> int:
        return self.L[key]

    def snapshot(self):
        return (list(self.L), [], [], [], 0.0)

    def pin(self, key: int) -> None:
        assert key in self.L
        self.pinned.add(key)

    def unpin_all(self) -> None:
        self.pinned.clear()

    def reference(self, x: int, depth: int = 0) -> Event:
        if x in self.L:
            self.L.move_to_end(x)
            ev = Event(x, LRU_HIT, NO_HASH, FROM_NONE, NO_HASH, FROM_NONE, self.L[x], 0.0)
        else:
            evicted, evicted_from = NO_HASH, FROM_NONE
            if len(self.L) == self.c:
                victim = window_victim(self.L, self.pinned, self.depth, self.window)
                if victim is None:
                    raise RuntimeError("LRU found no unpinned page")
                phys = self.L.pop(victim)
                evicted, evicted_from = victim, FROM_T1
            else:
                if not self.free:
                    raise RuntimeError("free list exhausted")
                phys = self.free.popleft()
            self.L[x] = phys
            ev = Event(x, LRU_MISS, evicted, evicted_from, NO_HASH, FROM_NONE, phys, 0.0)
        self.depth[x] = int(depth)
        self.log.append(ev)
        return ev

    def check_invariants(self) -> None:
        assert len(self.L) <= self.c
