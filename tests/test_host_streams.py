"""Host phase of the multi-turn and trace-replay workloads, library vs oracle, bit-exact.

Every request of the stream is hashed (library: C++ hasher; oracle: its own FNV-1a), grouped
into batches (library batch formation vs oracle's), planned and released by the library cache
and by the oracle planner with the same policy and seeded free list.  Compared per batch: block
tables, cu_q, sequence lengths, hit blocks, slot mappings; over the whole stream: every policy
decision (case, evicted / dropped identity and list, physical block, p after the reference),
the final T1 / T2 / B1 / B2 contents, p, and the token totals.  ARC, DBL and LRU all run, so
the reported hit rates of the policies are each the oracle's.
"""

import numpy as np
import pytest

import paper_2606_21238_amd as ak
from oracle import blockhash as obh
from oracle.planner import Planner, form_batches
from workloads import get_config
from workloads.streams import free_order, sized, stream_multiturn, stream_trace

LIST_IDS = (ak.LIST_T1, ak.LIST_T2, ak.LIST_B1, ak.LIST_B2)


def oracle_hashes(reqs, chunk=512):
    out = []
    for i in range(0, len(reqs), chunk):
        out += obh.hash_blocks_many([r.tokens for r in reqs[i:i + chunk]])
    return out


def replay(cfg, reqs, policy, orc_hashes, window=1):
    """Drive library and oracle over the whole stream; returns (library cache, oracle planner)."""
    lens = [r.n_tokens for r in reqs]
    batches = form_batches(lens, cfg.max_batch, cfg.capacity, cfg.scratch)
    i, lib_batches = 0, []
    while i < len(lens):
        n = ak.next_batch(lens[i:i + 4 * cfg.max_batch], cfg.max_batch, cfg.capacity, cfg.scratch)
        lib_batches.append((i, i + n))
        i += n
    assert lib_batches == batches
    order = free_order(cfg.seed, cfg.num_phys)
    lib = ak.BlockCache(policy, cfg.capacity, cfg.num_phys, cfg.scratch, order, victim_window=window)
    lib.set_log(sum(len(h) for h in orc_hashes) + 1)
    orc = Planner(policy, cfg.capacity, cfg.num_phys, cfg.scratch, order, victim_window=window)
    lib_hashes = ak.hash_blocks_batch([r.tokens for r in reqs])
    for a, b in batches:
        p = lib.plan_batch([(lib_hashes[j], lens[j]) for j in range(a, b)])
        q = orc.plan_batch([(orc_hashes[j], lens[j]) for j in range(a, b)])
        assert p.hit_blocks.tolist() == q.hit_blocks
        assert p.prefix_lens.tolist() == q.prefix_lens
        assert p.seq_lens.tolist() == q.seq_lens
        assert p.cu_q.tolist() == q.cu_q
        assert p.slot_mapping.tolist() == q.slot_mapping
        for r, row in enumerate(q.block_tables):
            assert p.block_tables[r, : len(row)].tolist() == row
            assert (p.block_tables[r, len(row):] == -1).all()
        lib.release_batch()
        orc.release_batch()
    return lib, orc


def check_decisions(lib, orc):
    got = lib.log_array()
    want = orc.cache.log
    assert len(got) == len(want) == lib.log_count()
    for field, attr in (("key", "key"), ("kase", "case"), ("evicted", "evicted"),
                        ("evicted_from", "evicted_from"), ("dropped", "dropped"),
                        ("dropped_from", "dropped_from"), ("phys_block", "phys"), ("p_after", "p_after")):
        col = np.array([getattr(e, attr) for e in want], dtype=got.dtype[field])
        bad = np.flatnonzero(got[field] != col)
        assert bad.size == 0, f"{field} differs first at decision {bad[0]}: {got[bad[0]]} vs {want[bad[0]]}"
    snap = orc.cache.snapshot()
    for li, keys in zip(LIST_IDS, snap[:4]):
        k, _ = lib.snapshot(li)
        assert [int(x) for x in k] == list(keys)
    st = lib.stats()
    assert st["p"] == snap[4]
    t = orc.totals
    assert (st["requests"], st["prompt_tokens"], st["prefix_hit_tokens"], st["computed_tokens"]) == \
        (t.requests, t.prompt_tokens, t.prefix_hit_tokens, t.computed_tokens)
    assert st["case_counts"] == t.case_counts
    orc.cache.check_invariants()
    return t.prefix_hit_tokens / t.prompt_tokens


@pytest.fixture(scope="module")
def multiturn():
    base = get_config("multiturn")
    reqs, cap = stream_multiturn(base)
    return sized(base, cap), reqs, oracle_hashes(reqs)


@pytest.mark.parametrize("policy,window", [("arc", 1), ("lru", 1), ("dbl", 1), ("arc", 16), ("lru", 16)])
def test_multiturn_stream_bit_exact(multiturn, policy, window):
    cfg, reqs, hashes = multiturn
    assert len(reqs) == 1024
    lib, orc = replay(cfg, reqs, policy, hashes, window)
    rate = check_decisions(lib, orc)
    print(f"multiturn {policy}: capacity {cfg.capacity} blocks, token hit rate {rate:.4f}")
    # sessions come back, so a large share of the prompt tokens is served from the cache
    assert 0.2 < rate < 1.0


def trace_case(n_requests):
    base = get_config("trace")
    reqs, cap = stream_trace(base, n_requests)
    return sized(base, cap), reqs, oracle_hashes(reqs)


@pytest.fixture(scope="module")
def trace_head():
    return trace_case(2000)


@pytest.mark.parametrize("policy", ["arc", "lru", "dbl"])
def test_trace_first_2000_bit_exact(trace_head, policy):
    cfg, reqs, hashes = trace_head
    lib, orc = replay(cfg, reqs, policy, hashes)
    rate = check_decisions(lib, orc)
    print(f"trace[:2000] {policy}: capacity {cfg.capacity} blocks, token hit rate {rate:.4f}")
    assert 0.1 < rate < 1.0


@pytest.mark.slow
def test_trace_full_replay_bit_exact():
    """All 10,000 requests, the two policies bench reports (about two minutes of oracle time;
    DBL runs on the first 2,000 above)."""
    cfg, reqs, hashes = trace_case(None)
    assert len(reqs) == 10000
    for policy in ("arc", "lru"):
        lib, orc = replay(cfg, reqs, policy, hashes)
        check_decisions(lib, orc)
