"""Paged KV pool image, scatter and gather (oracle).  TEST INFRASTRUCTURE ONLY.

Paged attention keeps K/V in fixed-size blocks reached through a per-request
block table (Sec. 2, "LLM Serving"); the tokens a miss recomputes are written
into their blocks (Sec. 3: the engine recomputes a missed block and writes its
KV again).  Element values are bf16 bit patterns held as uint16, so every
operation here is an exact copy.

Pool layout (version 1, an interface shared with the library by definition):

* K pool: ``[num_blocks][num_kv_heads][16][head_dim]`` -- token-major in a block.
* V pool: ``[num_blocks][num_kv_heads][head_dim][16]`` -- dim-major in a block.

Token j of a request lives in physical block ``table[j // 16]`` at offset
``j % 16``; its "slot" is ``table[j // 16] * 16 + j % 16``.
"""

from __future__ import annotations

import numpy as np

BLOCK_TOKENS = 16


def new_pool(num_blocks: int, num_kv_heads: int, head_dim: int, fill: int = 0xFFFF):
    k = np.full((num_blocks, num_kv_heads, BLOCK_TOKENS, head_dim), fill, dtype=np.uint16)
    v = np.full((num_blocks, num_kv_heads, head_dim, BLOCK_TOKENS), fill, dtype=np.uint16)
    return k, v


def scatter(k_pool, v_pool, k_new, v_new, slots) -> None:
    """Write token t's K/V rows ([Hkv, D] bf16 bits) into slot ``slots[t]`` (in place).

    blk = slot // 16, off = slot % 16; K goes to k_pool[blk, :, off, :], V to
    v_pool[blk, :, :, off] (numpy fancy-index assignment, one element per token and head)."""
    k_new = np.asarray(k_new, dtype=np.uint16)
    v_new = np.asarray(v_new, dtype=np.uint16)
    slots = np.asarray(slots, dtype=np.int64)
    if slots.size == 0:
        return
    blk, off = slots // BLOCK_TOKENS, slots % BLOCK_TOKENS
    k_pool[blk, :, off, :] = k_new
    # advanced indices (blk, off) separated by slices put the token axis first: [T, Hkv, D]
    v_pool[blk, :, :, off] = v_new


def gather(k_pool, v_pool, table_row, n_tokens: int):
    """Contiguous K, V ([n_tokens, Hkv, D] bf16 bits) of one request through its block table:
    token j comes from physical block table_row[j // 16] at offset j % 16."""
    j = np.arange(n_tokens)
    blk = np.asarray(table_row, dtype=np.int64)[j // BLOCK_TOKENS]
    off = j % BLOCK_TOKENS
    k = k_pool[blk, :, off, :]
    v = v_pool[blk, :, :, off]
    return np.ascontiguousarray(k), np.ascontiguousarray(v)


def touched_blocks(slots) -> set[int]:
    return {int(s) // BLOCK_TOKENS for s in slots}
