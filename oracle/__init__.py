"""CPU oracle for prefix-cached paged prefill attention under an ARC/LRU KV-block cache.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously-correct
reference of what the GPU library computes.  Only the test-suite, the smoke
check in ``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import
it.  It shares no code with the library (``paper_2606_21238_amd``): neither
imports the other; both take their inputs from the seeded generators in
``workloads`` (which hold none of the method's arithmetic).

Contents, each module citing the passage of the paper it follows:

* ``blockhash`` -- chained 64-bit block identities (FNV-1a over parent hash and
  16 token ids).  The paper makes eviction block-granular (end of Sec. 3) and
  relies on prefix caching (Sec. 2, "LLM Serving"); it does not define the hash,
  so the hash is this project's reading, pinned against the published FNV
  test vectors.
* ``arc`` -- ARC(c) over KV blocks: resident lists T1/T2, ghost lists B1/B2,
  adaptive target p (Sec. 3 and Fig. 2; adaptation rules of the cited ARC
  paper by Megiddo and Modha, restated).  Pin-aware victim choice for blocks in
  use by the running batch.
* ``lru`` -- the LRU baseline the paper compares against (Sec. 2, Sec. 4).
* ``planner`` -- per-batch prefix lookup, policy references, physical block
  placement, block tables and slot mappings (Sec. 2: blocks handed out by a
  paging allocator; Sec. 3: a miss is recomputed by the engine, which writes the
  block's KV again).
* ``kvpool`` -- the paged pool image, the KV scatter, and the gather through a
  block table.
* ``attention`` -- fp64 causal softmax attention of the uncached suffix over
  the gathered contiguous K/V (Sec. 2: prefill processes the prompt; with a
  cached prefix only the uncached tokens are computed).
* ``qkv`` -- the producer of the computed tokens' Q/K/V: projection of their
  hidden states and rotary position embedding (Sec. 4 serves Qwen3-14B; the
  layer details are this project's reading of the public model configuration).

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
against values fixed by the mathematics or by hand-derived traces; none is
"parity unpinned".
"""

from . import blockhash, arc, lru, planner, kvpool, attention, qkv  # noqa: F401

__all__ = ["blockhash", "arc", "lru", "planner", "kvpool", "attention", "qkv"]
