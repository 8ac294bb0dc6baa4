"""Checkpoint / resume of the host cache (arckv_cache_save / arckv_cache_restore), CPU only.

A replay stopped after some batches, saved, restored into a new cache and continued makes the
same decisions, placements and plans as the uninterrupted replay, for every policy and option;
images round-trip byte for byte; malformed or inconsistent images are refused.
"""

import numpy as np
import pytest

import paper_2606_21238_amd as ak
from paper_2606_21238_amd import _lib
from oracle.planner import form_batches
from workloads import get_config
from workloads.streams import free_order, sized, stream_multiturn, stream_trace

LISTS = (ak.LIST_T1, ak.LIST_T2, ak.LIST_B1, ak.LIST_B2)


def lists(cache):
    return [tuple(map(tuple, cache.snapshot(li))) for li in LISTS]


def plan_fields(p):
    return (p.block_tables.tolist(), p.cu_q.tolist(), p.seq_lens.tolist(), p.prefix_lens.tolist(),
            p.hit_blocks.tolist(), p.slot_mapping.tolist())


def stream(name, n):
    base = get_config(name)
    reqs, cap = stream_trace(base, n) if name == "trace" else stream_multiturn(base)
    cfg = sized(base, cap)
    lens = [r.n_tokens for r in reqs]
    batches = form_batches(lens, cfg.max_batch, cfg.capacity, cfg.scratch)
    hashes = ak.hash_blocks_batch([r.tokens for r in reqs])
    digests = [ak.digest_blocks(r.tokens) for r in reqs]
    return cfg, lens, batches, hashes, digests


def make(cfg, policy, **kw):
    return ak.BlockCache(policy, cfg.capacity, cfg.num_phys, cfg.scratch, free_order(cfg.seed, cfg.num_phys), **kw)


def run(cache, batches, lens, hashes, digests, check):
    out = []
    for a, b in batches:
        reqs = [(hashes[j], lens[j], digests[j] if check else None) for j in range(a, b)]
        out.append(plan_fields(cache.plan_batch(reqs)))
        cache.release_batch()
    return out


@pytest.mark.parametrize("policy,kw", [
    ("arc", {}),
    ("lru", {}),
    ("dbl", {}),
    ("frc", {"frc_p": 1000.5}),
    ("arc", {"victim_window": 8}),
    ("arc", {"intra_batch_reuse": False, "ref_order": "head_first"}),
    ("arc", {"check_blocks": True}),
])
def test_resumed_replay_equals_the_uninterrupted_one(policy, kw):
    cfg, lens, batches, hashes, digests = stream("multiturn", 0)
    check = kw.get("check_blocks", False)
    stop = len(batches) // 2
    full = make(cfg, policy, **kw)
    full.set_log(sum(len(h) for h in hashes) + 1)
    ref = run(full, batches, lens, hashes, digests, check)
    n_first = sum(len(hashes[j]) for a, b in batches[:stop] for j in range(a, b))

    first = make(cfg, policy, **kw)
    run(first, batches[:stop], lens, hashes, digests, check)
    image = first.save()
    resumed = ak.BlockCache.restore(image)
    assert resumed.stats() == first.stats() and lists(resumed) == lists(first)
    assert resumed.save() == image                           # round trip, byte for byte
    resumed.set_log(sum(len(h) for h in hashes) + 1)
    got = run(resumed, batches[stop:], lens, hashes, digests, check)
    assert got == ref[stop:]
    assert resumed.log() == full.log()[n_first:]
    assert resumed.stats() == full.stats() and lists(resumed) == lists(full)


def test_trace_resumes_past_the_full_cache():
    """The trace window runs until the cache evicts; stop there and go on."""
    cfg, lens, batches, hashes, digests = stream("trace", 900)
    full = make(cfg, "arc")
    ref = run(full, batches, lens, hashes, digests, False)
    stop = 2 * len(batches) // 3
    first = make(cfg, "arc")
    run(first, batches[:stop], lens, hashes, digests, False)
    assert first.stats()["case_counts"][ak.CASE_IVB] > 0 and first.stats()["b1"] > 0
    resumed = ak.BlockCache.restore(first.save())
    assert run(resumed, batches[stop:], lens, hashes, digests, False) == ref[stop:]
    assert resumed.stats() == full.stats() and lists(resumed) == lists(full)


def test_save_refuses_a_batch_in_flight_and_small_buffers():
    cache = ak.BlockCache("arc", 8, 12, 4)
    cache.plan_batch([(ak.hash_blocks(np.arange(40, dtype=np.int32)), 40)])
    with pytest.raises(_lib.ArckvError) as e:
        cache.save()
    assert e.value.status == _lib.ESTATE
    cache.release_batch()
    n = _lib.i64()
    L = ak.lib()
    assert L.arckv_cache_save(cache._h, None, 0, n) == _lib.OK and n.value > 0
    import ctypes
    buf = ctypes.create_string_buffer(16)
    assert L.arckv_cache_save(cache._h, buf, 16, n) == _lib.ENOSPC and n.value > 16


def test_restore_refuses_malformed_images():
    cache = ak.BlockCache("arc", 8, 12, 4)
    for t in (np.arange(40), np.arange(40) + 100, np.arange(20) + 7):
        cache.plan_batch([(ak.hash_blocks(t.astype(np.int32)), len(t))])
        cache.release_batch()
    image = bytearray(cache.save())
    words = np.frombuffer(bytes(image), dtype=np.uint64).copy()
    ak.BlockCache.restore(bytes(image))                     # the image itself is fine

    def refused(w):
        with pytest.raises(_lib.ArckvError) as e:
            ak.BlockCache.restore(w.tobytes() if isinstance(w, np.ndarray) else w)
        assert e.value.status == _lib.EINVAL

    refused(bytes(image[:-8]))                              # truncated
    refused(bytes(image) + bytes(8))                        # trailing word
    w = words.copy(); w[0] ^= 1; refused(w)                 # magic
    w = words.copy(); w[1] = 2; refused(w)                  # version
    w = words.copy(); w[10] = np.array([99.0]).view(np.uint64)[0]; refused(w)       # p > c
    # a resident page whose physical block is also on the free list
    t1_size_at = 2 + 8 + 1 + 5 + 8
    n_t1 = int(words[t1_size_at])
    assert n_t1 > 0
    phys0 = int(words[t1_size_at + 2])
    free_at = t1_size_at + 1 + 4 * n_t1
    for _ in range(3):                                      # skip T2, B1, B2
        free_at += 1 + 4 * int(words[free_at])
    n_free = int(words[free_at])
    assert n_free > 0
    w = words.copy(); w[free_at + 1] = phys0; refused(w)
