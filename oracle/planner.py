"""Batch planning over the block cache (oracle).  TEST INFRASTRUCTURE ONLY.

What one batch of prefill requests needs before the GPU runs (Sec. 2 "LLM
Serving": prefix caching reuses the KV of a shared prefix across requests;
paged attention keeps KV in fixed-size blocks handed out by a paging-style
allocator; Sec. 3: a miss is processed by the engine, which regenerates the
block; Sec. 4 "Batch Inference": several requests are planned together).

Readings fixed by this project where the paper is silent:

* Request order.  Requests of a batch are planned one after another; a later
  request may hit blocks an earlier request of the same batch created (the
  scatter of the whole batch is ordered before its attention).  With
  ``intra_batch_reuse=False`` the prefix lookup stops at a block that a reference
  of the current batch made resident (a miss or a ghost hit); it is then
  referenced like any resident block (an orphan, recomputed).
* Prefix lookup.  k = number of leading full blocks whose identity is resident
  (in T1 or T2 for ARC).  If that covers the whole prompt (16 k == L) the last
  block is recomputed (k -> k - 1) so that at least one query produces the
  next-token logit (Sec. 4 generates one token per request).  P = 16 k cached
  tokens, S = L - P computed tokens.
* Pins.  The k prefix pages are pinned first, then every full block of the
  request is referenced once in tail-first order (last block first) and
  pinned; pins last until the batch is released, so no block a planned request
  reads can be evicted by a later request of the same batch.
* Orphans.  A block resident beyond the first miss is a Case I hit for the
  policy; its physical block is kept and its KV is rewritten with equal bytes.
* Partial tail.  A last block with fewer than 16 tokens has no identity; it
  takes a block from a separate scratch FIFO and returns it on release.
* Placement.  The pool's blocks, in the given initial order, are split into a
  page region (the first ``num_phys - scratch``) and the scratch FIFO (the rest).
* Depth.  Each reference carries the block's index in its prompt, which a
  length-aware victim window (``oracle.arc``) weighs.
* Batch formation.  Consecutive requests, at most ``max_batch``, while the sum
  of their full blocks stays within the capacity c and their partial tails
  within the scratch blocks; this guarantees that a pin-aware victim exists.

Outputs per batch (all integers): block table rows (physical block of every
logical block, full and partial), cu_q (prefix sums of S), seq_lens (L),
prefix_lens (P), hit_blocks (k) and the slot of every computed token,
slot = table[j // 16] * 16 + j % 16 for j in [P, L).
"""

from __future__ import annotations

from collections import deque
from dataclasses import dataclass, field

from .arc import ARC, CASE_I, LRU_HIT
from .lru import LRU

BLOCK_TOKENS = 16


class PlanError(Exception):
    """Planner refused a batch; ``code`` mirrors the library's status codes."""

    def __init__(self, code: str, msg: str):
        super().__init__(f"{code}: {msg}")
        self.code = code


@dataclass
class Plan:
    block_tables: list[list[int]]
    cu_q: list[int]
    seq_lens: list[int]
    prefix_lens: list[int]
    hit_blocks: list[int]
    slot_mapping: list[int]
    events_begin: int = 0
    events_end: int = 0


@dataclass
class Totals:
    requests: int = 0
    prompt_tokens: int = 0
    prefix_hit_tokens: int = 0
    computed_tokens: int = 0
    case_counts: list[int] = field(default_factory=lambda: [0] * 8)


def form_batches(n_tokens_list, max_batch: int, capacity: int, scratch_blocks: int):
    """Split a request stream into batches (list of (start, end) index pairs)."""
    out = []
    i, n = 0, len(n_tokens_list)
    while i < n:
        blocks, tails, j = 0, 0, i
        while j < n and j - i < max_batch:
            nf = n_tokens_list[j] // BLOCK_TOKENS
            tl = 1 if n_tokens_list[j] % BLOCK_TOKENS else 0
            if blocks + nf > capacity or tails + tl > scratch_blocks:
                break
            blocks += nf
            tails += tl
            j += 1
        if j == i:
            raise PlanError("ENOSPC", f"request {i} alone exceeds capacity or scratch")
        out.append((i, j))
        i = j
    return out


class Planner:
    def __init__(self, policy: str, capacity: int, num_phys: int, scratch_blocks: int,
                 initial_order=None, ref_order: str = "tail_first", victim_window: int = 1,
                 intra_batch_reuse: bool = True, frc_p: float = 0.0):
        order = list(range(num_phys)) if initial_order is None else [int(b) for b in initial_order]
        if sorted(order) != list(range(num_phys)):
            raise PlanError("EINVAL", "initial order is not a permutation of the pool")
        n_pages = num_phys - scratch_blocks
        if scratch_blocks < 0 or n_pages < capacity:
            raise PlanError("EINVAL", "pool too small for capacity + scratch")
        pages = order[:n_pages]
        self.scratch = deque(order[n_pages:])
        if policy == "arc":
            self.cache = ARC(capacity, pages, window=victim_window)
        elif policy == "dbl":
            self.cache = ARC(capacity, pages, adaptive=False, window=victim_window)
        elif policy == "frc":
            if not 0.0 <= frc_p <= capacity:
                raise PlanError("EINVAL", "frc_p outside [0, c]")
            self.cache = ARC(capacity, pages, adaptive=False, window=victim_window, fixed_p=frc_p)
        elif policy == "lru":
            self.cache = LRU(capacity, pages, window=victim_window)
        else:
            raise PlanError("EINVAL", f"unknown policy {policy}")
        if ref_order not in ("tail_first", "head_first"):
            raise PlanError("EINVAL", "ref_order")
        self.ref_order = ref_order
        self.capacity = capacity
        self.intra_batch_reuse = intra_batch_reuse
        self.born: set[int] = set()      # keys a reference of the batch made resident
        self.in_flight = False
        self.batch_scratch: list[int] = []
        self.totals = Totals()

    def plan_batch(self, reqs) -> Plan:
        """reqs: sequence of (hashes, n_tokens) with len(hashes) == n_tokens // 16."""
        if self.in_flight:
            raise PlanError("ESTATE", "previous batch not released")
        total_blocks, tails = 0, 0
        for hashes, n_tok in reqs:
            if n_tok < 1 or len(hashes) != n_tok // BLOCK_TOKENS:
                raise PlanError("EINVAL", "request length / hash count mismatch")
            total_blocks += len(hashes)
            tails += 1 if n_tok % BLOCK_TOKENS else 0
        if total_blocks > self.capacity:
            raise PlanError("ENOSPC", "batch needs more full blocks than the capacity")
        if tails > len(self.scratch):
            raise PlanError("ENOSPC", "not enough scratch blocks for partial tails")

        cache = self.cache
        plan = Plan([], [0], [], [], [], [], events_begin=len(cache.log))
        for hashes, n_tok in reqs:
            n_full = len(hashes)
            k = 0
            while k < n_full and cache.resident(hashes[k]) and \
                    (self.intra_batch_reuse or hashes[k] not in self.born):
                k += 1
            if BLOCK_TOKENS * k == n_tok:
                k -= 1
            for i in range(k):
                cache.pin(hashes[i])
            order = range(n_full - 1, -1, -1) if self.ref_order == "tail_first" else range(n_full)
            phys = [None] * n_full
            for i in order:
                ev = cache.reference(hashes[i], depth=i)
                if ev.case not in (CASE_I, LRU_HIT):      # a miss or a ghost hit
                    self.born.add(hashes[i])
                phys[i] = ev.phys
                cache.pin(hashes[i])
                self.totals.case_counts[ev.case] += 1
            row = list(phys)
            if n_tok % BLOCK_TOKENS:
                blk = self.scratch.popleft()
                self.batch_scratch.append(blk)
                row.append(blk)
            P = BLOCK_TOKENS * k
            plan.block_tables.append(row)
            plan.seq_lens.append(n_tok)
            plan.prefix_lens.append(P)
            plan.hit_blocks.append(k)
            plan.cu_q.append(plan.cu_q[-1] + n_tok - P)
            for j in range(P, n_tok):
                plan.slot_mapping.append(row[j // BLOCK_TOKENS] * BLOCK_TOKENS + j % BLOCK_TOKENS)
            self.totals.requests += 1
            self.totals.prompt_tokens += n_tok
            self.totals.prefix_hit_tokens += P
            self.totals.computed_tokens += n_tok - P
        plan.events_end = len(cache.log)
        self.in_flight = True
        return plan

    def release_batch(self) -> None:
        if not self.in_flight:
            raise PlanError("ESTATE", "no batch to release")
        self.cache.unpin_all()
        self.born.clear()
        self.scratch.extend(self.batch_scratch)
        self.batch_scratch = []
        self.in_flight = False
