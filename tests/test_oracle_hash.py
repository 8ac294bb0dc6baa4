"""Pins of the oracle's chained block hash (CPU only)."""

import os
import struct

import numpy as np
import pytest

from oracle import blockhash as bh

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fnv1a64_vectors.txt")


def _vectors():
    out = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            s, h = line.rsplit(" ", 1)
            out.append((s.strip('"').encode(), int(h, 16)))
    return out


@pytest.mark.parametrize("data,expect", _vectors())
def test_fnv1a64_published_vectors(data, expect):
    assert bh.fnv1a64(data) == expect


def test_block_bytes_layout_matches_struct_packing():
    # The hashed message is the parent as little-endian u64 then 16 little-endian i32 ids;
    # struct packing is an independent route to the same byte string.
    toks = list(range(-3, 13))
    parent = 0x0123456789ABCDEF
    assert bh.block_bytes(parent, toks) == struct.pack("<Q16i", parent, *toks)


def test_chain_first_block_and_partial_tail():
    toks = np.arange(40, dtype=np.int32)
    hs = bh.hash_blocks(toks)
    assert len(hs) == 2                         # 40 tokens -> 2 full blocks, tail of 8 not hashed
    h0 = bh.fnv1a64(struct.pack("<Q16i", 0, *range(16)))
    h1 = bh.fnv1a64(struct.pack("<Q16i", h0, *range(16, 32)))
    assert hs == [h0, h1]
    assert bh.hash_blocks(toks[:15]) == []


def test_chain_prefix_property():
    rng = np.random.default_rng(0)
    a = rng.integers(0, 128256, 16 * 9).astype(np.int32)
    b = a.copy()
    b[16 * 4 + 3] += 1                          # change one token of block 4
    ha, hb = bh.hash_blocks(a), bh.hash_blocks(b)
    assert ha[:4] == hb[:4]                     # earlier blocks keep their identity
    assert all(x != y for x, y in zip(ha[4:], hb[4:]))   # the change propagates down the chain
    c = a.copy()
    c[:16] = a[16:32]
    c[16:32] = a[:16]                           # same block contents in another order -> new ids
    assert bh.hash_blocks(c)[1] != ha[1]


def test_root_changes_every_identity():
    a = np.arange(64, dtype=np.int32)
    assert all(x != y for x, y in zip(bh.hash_blocks(a, root=0), bh.hash_blocks(a, root=7)))


def test_vectorised_equals_scalar():
    rng = np.random.default_rng(1)
    seqs = [rng.integers(0, 128256, n).astype(np.int32) for n in (0, 15, 16, 17, 100, 333)]
    assert bh.hash_blocks_many(seqs) == [bh.hash_blocks(s) for s in seqs]
    assert bh.hash_blocks_many(seqs, root=99) == [bh.hash_blocks(s, root=99) for s in seqs]
