"""Chained block identities (oracle).  TEST INFRASTRUCTURE ONLY.

The paper caches and evicts KV at the granularity of fixed 16-token blocks
(Sec. 3, last paragraph; Sec. 4 "Inference Configuration") and reuses the KV
of a shared prefix across requests (Sec. 2, "LLM Serving").  A block can only be
reused if every token before it is the same, so a block's identity must cover
its own tokens and, through its parent, all earlier ones.  The paper does not
name a hash; this project's reading is:

    h_{-1} = root (0 by default)
    h_i    = FNV1a64( le64(h_{i-1}) || le32(tok[16 i]) || ... || le32(tok[16 i + 15]) )

for every *full* block i; a trailing partial block gets no identity.
FNV-1a-64: offset basis 0xcbf29ce484222325, prime 0x100000001b3, for each byte
``h ^= b; h *= prime (mod 2**64)``.
"""

from __future__ import annotations

import numpy as np

BLOCK_TOKENS = 16
FNV_OFFSET = 0xCBF29CE484222325
FNV_PRIME = 0x100000001B3
MASK64 = (1 << 64) - 1


def fnv1a64(data: bytes, h: int = FNV_OFFSET) -> int:
    """FNV-1a, 64-bit, byte at a time (the published definition)."""
    for b in data:
        h ^= b
        h = (h * FNV_PRIME) & MASK64
    return h


def block_bytes(parent: int, tokens) -> bytes:
    """The byte string hashed for one block: parent hash, then 16 token ids, little-endian."""
    assert len(tokens) == BLOCK_TOKENS
    out = int(parent & MASK64).to_bytes(8, "little")
    for t in tokens:
        out += int(np.int32(t)).to_bytes(4, "little", signed=True)
    return out


def hash_blocks(tokens, root: int = 0) -> list[int]:
    """Chained identities of the full blocks of one token sequence (pure Python)."""
    tokens = [int(t) for t in tokens]
    n_full = len(tokens) // BLOCK_TOKENS
    out = []
    h = root & MASK64
    for i in range(n_full):
        h = fnv1a64(block_bytes(h, tokens[BLOCK_TOKENS * i: BLOCK_TOKENS * (i + 1)]))
        out.append(h)
    return out


def hash_blocks_many(seqs, root: int = 0) -> list[list[int]]:
    """Same definition, evaluated for many sequences at once.

    The recurrence is sequential in the bytes of one sequence, so the only
    vectorisation is across sequences: every byte step updates one uint64 lane
    per sequence (numpy uint64 multiply wraps modulo 2**64).  Sequences shorter
    than the longest simply stop updating.
    """
    seqs = [np.asarray(s, dtype=np.int32) for s in seqs]
    if not seqs:
        return []
    nfull = np.array([len(s) // BLOCK_TOKENS for s in seqs], dtype=np.int64)
    maxb = int(nfull.max()) if len(nfull) else 0
    n = len(seqs)
    tok = np.zeros((n, maxb * BLOCK_TOKENS), dtype=np.int32)
    for r, s in enumerate(seqs):
        tok[r, : nfull[r] * BLOCK_TOKENS] = s[: nfull[r] * BLOCK_TOKENS]
    tok_bytes = tok.view(np.uint8).reshape(n, maxb, BLOCK_TOKENS * 4)  # little-endian host
    prime = np.uint64(FNV_PRIME)
    parent = np.full(n, np.uint64(root & MASK64), dtype=np.uint64)
    out = np.zeros((n, maxb), dtype=np.uint64)
    with np.errstate(over="ignore"):
        for i in range(maxb):
            h = np.full(n, np.uint64(FNV_OFFSET), dtype=np.uint64)
            for byte in range(8):
                b = (parent >> np.uint64(8 * byte)) & np.uint64(0xFF)
                h = (h ^ b) * prime
            for byte in range(BLOCK_TOKENS * 4):
                h = (h ^ tok_bytes[:, i, byte].astype(np.uint64)) * prime
            live = nfull > i
            out[live, i] = h[live]
            parent = np.where(live, h, parent)
    return [[int(x) for x in out[r, : nfull[r]]] for r in range(n)]
