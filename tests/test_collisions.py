"""Check mode: block identity collisions are caught by the planner (CPU only).

Block identities are 64-bit chained hashes (FNV-1a-64); two different token blocks behind one
identity would make the cache hand one prompt's KV to another.  In check mode every resident
page also keeps the block's digest (an independent chained hash) and every plan verifies the
digests of the blocks it is about to reuse or share, before it changes anything.  A test-only
override masks the identities so that collisions happen on demand.
"""

from __future__ import annotations

import numpy as np
import pytest

import paper_2606_21238_amd as ak
from paper_2606_21238_amd import _lib

M64 = (1 << 64) - 1


def splitmix_final(z: int) -> int:
    """The splitmix64 finaliser, from its published definition (Steele, Lea and Flood 2014)."""
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def digests_by_hand(tokens, root=0):
    d = splitmix_final(root ^ 0xD1B54A32D192ED03)
    out = []
    for b in range(len(tokens) // 16):
        for t in tokens[16 * b:16 * b + 16]:
            d = splitmix_final((d + 0x9E3779B97F4A7C15 + (int(t) & 0xFFFFFFFF)) & M64)
        out.append(d)
    return out


def all_lists(cache):
    return [tuple(map(tuple, cache.snapshot(li))) for li in (ak.LIST_T1, ak.LIST_T2, ak.LIST_B1, ak.LIST_B2)]


def plan(cache, prompts, digests=True):
    reqs = [(ak.hash_blocks(t), len(t), ak.digest_blocks(t) if digests else None) for t in prompts]
    return cache.plan_batch(reqs)


def test_digest_is_the_splitmix_chain():
    rng = np.random.default_rng(3)
    for n, root in ((16, 0), (53, 0), (80, 12345), (15, 0), (0, 0)):
        t = rng.integers(-2**31, 2**31, n, dtype=np.int64).astype(np.int32)
        got = ak.digest_blocks(t, root)
        assert [int(v) for v in got] == digests_by_hand(t, root)
        assert len(got) == n // 16                       # the partial tail is not digested


def test_digest_chains_over_the_prefix_and_differs_from_the_identity():
    t = np.arange(64, dtype=np.int32)
    d = ak.digest_blocks(t)
    u = t.copy()
    u[20] += 1                                           # block 1
    e = ak.digest_blocks(u)
    assert d[0] == e[0] and (d[1:] != e[1:]).all()       # blocks >= 1 change, block 0 does not
    assert (ak.digest_blocks(t, root=1) != d).all()
    assert not set(map(int, d)) & set(map(int, ak.hash_blocks(t)))


def test_mask_forces_identity_collisions_and_restores():
    t = np.arange(48, dtype=np.int32)
    normal = ak.hash_blocks(t)
    with ak.forced_identity_mask(0):
        assert (ak.hash_blocks(t) == 0).all()
        assert all((h == 0).all() for h in ak.hash_blocks_batch([t, t + 1]))
    with ak.forced_identity_mask(0xFF):
        assert (ak.hash_blocks(t) == (normal & np.uint64(0xFF))).all()    # the chain runs unmasked
    assert (ak.hash_blocks(t) == normal).all()


def test_collision_with_a_resident_page_is_refused_before_any_state_change():
    a = np.arange(20, dtype=np.int32)            # one full block + a tail
    b = np.arange(20, dtype=np.int32) + 1000     # a different first block
    with ak.forced_identity_mask(0):             # every identity is 0: a and b collide
        cache = ak.BlockCache("arc", 8, 12, 4, check_blocks=True)
        plan(cache, [a])
        cache.release_batch()
        before = (cache.stats(), all_lists(cache))
        with pytest.raises(_lib.ArckvError) as e:
            plan(cache, [b])
        assert e.value.status == _lib.ECOLLISION
        assert "0000000000000000" in str(e.value) and "differs from the resident page" in str(e.value)
        assert (cache.stats(), all_lists(cache)) == before and before[0]["in_flight"] == 0
        # the same prompt again is a verified hit, not a collision
        p = plan(cache, [a])
        assert p.hit_blocks[0] == 1 and p.prefix_lens[0] == 16
        cache.release_batch()


def test_without_check_mode_the_collision_reuses_the_wrong_kv():
    # what the check prevents: b's first block is "found" and a's KV would serve it
    a = np.arange(20, dtype=np.int32)
    b = np.arange(20, dtype=np.int32) + 1000
    with ak.forced_identity_mask(0):
        cache = ak.BlockCache("arc", 8, 12, 4)
        pa = plan(cache, [a])
        cache.release_batch()
        pb = plan(cache, [b])                    # digests are ignored without check mode
        assert pb.hit_blocks[0] == 1 and pb.block_tables[0, 0] == pa.block_tables[0, 0]
        cache.release_batch()


def test_collision_inside_one_batch_and_inside_one_prompt():
    a = np.arange(20, dtype=np.int32)
    b = np.arange(20, dtype=np.int32) + 1000
    with ak.forced_identity_mask(0):
        cache = ak.BlockCache("lru", 8, 12, 4, check_blocks=True)
        with pytest.raises(_lib.ArckvError) as e:
            plan(cache, [a, b])
        assert e.value.status == _lib.ECOLLISION
        assert "request 0 block 0 and request 1 block 0" in str(e.value)
        with pytest.raises(_lib.ArckvError) as e:
            plan(cache, [np.arange(32, dtype=np.int32)])    # blocks 0 and 1 share identity 0
        assert e.value.status == _lib.ECOLLISION
        assert cache.stats()["references"] == 0 and cache.stats()["in_flight"] == 0
        # the same block twice in one batch is no collision
        plan(cache, [a, a.copy()])
        cache.release_batch()


def test_many_prompts_under_a_narrow_mask_every_reuse_is_verified():
    # 64 identities, prompts drawn from 8 bases: every plan either succeeds with only verified
    # reuse or reports ECOLLISION and leaves the cache as it was
    rng = np.random.default_rng(7)
    bases = [rng.integers(0, 1000, 48, dtype=np.int64).astype(np.int32) for _ in range(8)]
    with ak.forced_identity_mask(0x3F):         # 64 identities for 24 distinct blocks
        cache = ak.BlockCache("arc", 12, 16, 4, check_blocks=True)
        owner = {}                               # physical block -> digest of the KV it holds
        n_ok = n_coll = n_hit = 0
        for _ in range(400):
            pr = [bases[int(rng.integers(0, 8))][: int(rng.integers(16, 49))] for _ in range(int(rng.integers(1, 3)))]
            before = (cache.stats(), all_lists(cache))
            try:
                p = plan(cache, pr)
            except _lib.ArckvError as e:
                assert e.status == _lib.ECOLLISION
                assert (cache.stats(), all_lists(cache)) == before
                n_coll += 1
                continue
            n_ok += 1
            for r, t in enumerate(pr):
                dg = ak.digest_blocks(t)
                for i in range(len(dg)):
                    phys = int(p.block_tables[r, i])
                    if i < p.hit_blocks[r]:
                        assert owner[phys] == int(dg[i])   # reused KV is this block's KV
                        n_hit += 1
                    owner[phys] = int(dg[i])
            cache.release_batch()
        assert n_ok > 50 and n_coll > 20 and n_hit > 50


def test_prepare_batch_checks_in_check_mode_only_on_the_token_path():
    a = np.arange(20, dtype=np.int32)
    b = np.arange(20, dtype=np.int32) + 1000
    packed = np.empty(1 << 16, dtype=np.int32)
    with ak.forced_identity_mask(0):
        cache = ak.BlockCache("arc", 8, 12, 4, check_blocks=True)
        st, _, _, _ = cache.prepare_native([a], 8, 2, 128, 256, packed)
        assert st == _lib.OK
        cache.release_batch()
        st, _, _, _ = cache.prepare_native([b], 8, 2, 128, 256, packed)
        assert st == _lib.ECOLLISION and cache.stats()["in_flight"] == 0
        # the hashed path carries no digests: it is not checked
        st, _, _, hb = cache.prepare_native(None, 8, 2, 128, 256, packed, hashes=[ak.hash_blocks(b)],
                                            n_tokens=[len(b)])
        assert st == _lib.OK and hb[0] == 1
        cache.release_batch()


def test_unchecked_pages_adopt_the_first_checked_digest():
    a = np.arange(20, dtype=np.int32)
    b = np.arange(20, dtype=np.int32) + 1000
    with ak.forced_identity_mask(0):
        cache = ak.BlockCache("arc", 8, 12, 4, check_blocks=True)
        plan(cache, [a], digests=False)          # page stored with no digest
        cache.release_batch()
        plan(cache, [a])                         # unverifiable hit: the page takes a's digest
        cache.release_batch()
        with pytest.raises(_lib.ArckvError) as e:
            plan(cache, [b])
        assert e.value.status == _lib.ECOLLISION


def test_check_flag_is_validated():
    cfg = _lib.CacheCfg(_lib.POLICY["arc"], _lib.REF_ORDER["tail_first"], 8, 12, 4, None, 1, 0, 0.0, 2)
    h = _lib.vp()
    assert ak.lib().arckv_cache_create(cfg, h) == _lib.EINVAL
