"""Native host side (hash, ARC/LRU cache, planner) against the oracle, bit-exact (CPU only).

Both sides take the same seeded inputs (token streams from ``workloads``); the library
hashes with its own C++ hasher, the oracle with its own Python one.  Compared: hashes,
block tables, cu_q, lengths, hit blocks, slot mappings, every policy decision (case,
evicted / dropped identities and lists, physical block, p), final list contents and p.
"""

import numpy as np
import pytest

import paper_2606_21238_amd as ak
from oracle import blockhash as obh
from oracle.planner import Planner, PlanError, form_batches
from workloads import get_config
from workloads.streams import (Source, make_request, free_order, make_stream, stream_docqa_hit,
                               KIND_DOC)


def test_hash_matches_oracle():
    rng = np.random.default_rng(11)
    seqs = [rng.integers(0, 128256, n).astype(np.int32) for n in (0, 1, 15, 16, 17, 160, 1000)]
    for s in seqs:
        assert [int(x) for x in ak.hash_blocks(s)] == obh.hash_blocks(s)
        assert [int(x) for x in ak.hash_blocks(s, root=12345)] == obh.hash_blocks(s, root=12345)
    neg = np.array([-1, -(2 ** 31)] + [7] * 14, dtype=np.int32)
    assert [int(x) for x in ak.hash_blocks(neg)] == obh.hash_blocks(neg)
    # the multi-sequence entry point (lock-step chains) gives the same identities
    many = seqs + [neg] + [rng.integers(0, 128256, n).astype(np.int32) for n in range(0, 400, 37)]
    got = ak.hash_blocks_batch(many, root=5)
    assert [[int(x) for x in g] for g in got] == [obh.hash_blocks(s, root=5) for s in many]


class Pair:
    """Library cache and oracle planner driven in lockstep."""

    def __init__(self, policy, c, nphys, scratch, order=None, ref_order="tail_first", window=1,
                 reuse=True, frc_p=0.0):
        self.lib = ak.BlockCache(policy, c, nphys, scratch, order, ref_order, window, reuse, frc_p)
        self.lib.set_log(1 << 20)
        self.orc = Planner(policy, c, nphys, scratch, order, ref_order, window, reuse, frc_p)
        self.n_events = 0

    def run(self, token_lists):
        lib_reqs = [(ak.hash_blocks(t), len(t)) for t in token_lists]
        orc_reqs = [(obh.hash_blocks(t), len(t)) for t in token_lists]
        p = self.lib.plan_batch(lib_reqs)
        q = self.orc.plan_batch(orc_reqs)
        n = len(token_lists)
        assert p.hit_blocks.tolist() == q.hit_blocks
        assert p.prefix_lens.tolist() == q.prefix_lens
        assert p.seq_lens.tolist() == q.seq_lens
        assert p.cu_q.tolist() == q.cu_q
        assert p.slot_mapping.tolist() == q.slot_mapping
        for r in range(n):
            row = q.block_tables[r]
            assert p.block_tables[r, : len(row)].tolist() == row
            assert (p.block_tables[r, len(row):] == -1).all()
        self.lib.release_batch()
        self.orc.release_batch()
        return p, q

    def check_log_and_state(self):
        got = self.lib.log()
        want = self.orc.cache.log
        assert len(got) == len(want)
        for g, e in zip(got, want):
            assert g == (e.key, e.case, e.evicted, e.evicted_from, e.dropped, e.dropped_from, e.phys,
                         e.p_after), (g, e)
        snap = self.orc.cache.snapshot()
        for li, keys in zip((ak.LIST_T1, ak.LIST_T2, ak.LIST_B1, ak.LIST_B2), snap[:4]):
            k, ph = self.lib.snapshot(li)
            assert [int(x) for x in k] == list(keys)
        st = self.lib.stats()
        assert st["p"] == snap[4]
        t = self.orc.totals
        assert (st["requests"], st["prompt_tokens"], st["prefix_hit_tokens"], st["computed_tokens"]) == \
            (t.requests, t.prompt_tokens, t.prefix_hit_tokens, t.computed_tokens)
        assert st["case_counts"] == t.case_counts


@pytest.mark.parametrize("policy", ["arc", "lru", "dbl", "frc"])
@pytest.mark.parametrize("ref_order", ["tail_first", "head_first"])
@pytest.mark.parametrize("seed,window,reuse", [(0, 1, True), (1, 1, True), (2, 1, False), (3, 2, True),
                                               (4, 7, False)])
def test_random_streams_bit_exact(policy, ref_order, seed, window, reuse):
    """window > 1: length-aware victims; reuse False: no intra-batch prefix reuse; frc: a
    fixed target p drawn per case.  The same decisions on both sides."""
    cfg = get_config("tiny")
    rng = np.random.default_rng(100 + seed)
    c, scratch = int(rng.integers(8, 40)), 8
    nphys = c + scratch + int(rng.integers(0, 5))
    frc_p = float(rng.integers(0, 2 * c + 1)) / 2     # multiples of 1/2 in [0, c]
    pair = Pair(policy, c, nphys, scratch, rng.permutation(nphys), ref_order, window, reuse, frc_p)
    docs = [make_request(cfg, [(Source(KIND_DOC, d, 200), 0, 200)]).tokens for d in range(12)]
    pops = 1.0 / np.arange(1, 13) ** 1.1
    pops /= pops.sum()
    for step in range(120):
        nreq = int(rng.integers(1, 4))
        toks = []
        for _ in range(nreq):
            d = int(rng.choice(12, p=pops))
            n = int(rng.integers(1, 200))
            extra = rng.integers(0, 128256, int(rng.integers(0, 40))).astype(np.int32)
            toks.append(np.concatenate([docs[d][:n], extra]))
        if sum(len(t) // 16 for t in toks) > c or sum(1 for t in toks if len(t) % 16) > scratch:
            continue
        pair.run(toks)
    pair.check_log_and_state()
    assert pair.orc.totals.prefix_hit_tokens > 0


def _golden_traces():
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "arc_traces.json")))
    return [("arc", t) for t in g["traces"]] + [("dbl", t) for t in g["dbl_traces"]]


@pytest.mark.parametrize("policy,tr", _golden_traces(), ids=lambda v: v if isinstance(v, str) else v["refs"])
def test_library_replays_the_hand_derived_traces(policy, tr):
    """The library's cache against the hand-derived ARC and DBL traces themselves (not the
    oracle): one single-block request per batch is exactly one policy reference of its key,
    so the decision log must list the fixture's cases, evicted and dropped pages and p."""
    c = tr["c"]
    cache = ak.BlockCache(policy, c, c + 1, 1)
    cache.set_log(1 << 10)
    for ch in tr["refs"]:
        cache.plan_batch([(np.array([ord(ch)], dtype=np.uint64), 16)])
        cache.release_batch()
    log = cache.log()
    case_names = ["I", "II", "III", "IVA", "IVA_T1DEL", "IVB"]
    assert [case_names[e[1]] for e in log] == tr["cases"]
    assert ["" if e[3] == 0 else chr(e[2]) for e in log] == tr["evicted"]
    if "dropped" in tr:
        assert ["" if e[5] == 0 else chr(e[4]) for e in log] == tr["dropped"]
    assert [e[7] for e in log] == [float(x) for x in tr["p"]]
    lists = [("".join(chr(k) for k in cache.snapshot(li)[0])) for li in
             (ak.LIST_T1, ak.LIST_T2, ak.LIST_B1, ak.LIST_B2)]
    assert lists == [tr["T1"], tr["T2"], tr["B1"], tr["B2"]]
    assert cache.stats()["p"] == tr["p_final"]


def _planner_cases():
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "planner_cases.json")))
    return [pytest.param(c, v, id=f"{c['name']}-reuse{int(v['intra_batch_reuse'])}") for c in g["cases"]
            for v in c.get("variants", [{"intra_batch_reuse": c.get("intra_batch_reuse", True)}])]


@pytest.mark.parametrize("case,var", _planner_cases())
def test_library_hand_derived_plans(case, var):
    """The library's planner against the hand-derived plans themselves (prefix pins, scratch
    FIFO, a B2 ghost hit as a page made in the batch)."""
    case_names = ["I", "II", "III", "IVA", "IVA_T1DEL", "IVB"]
    cache = ak.BlockCache(case["policy"], case["capacity"], case["num_phys"], case["scratch"],
                          intra_batch_reuse=var["intra_batch_reuse"])
    cache.set_log(1 << 10)
    for bi, b in enumerate(case["batches"]):
        n0 = len(cache.log())
        plan = cache.plan_batch([(np.array(h, dtype=np.uint64), n) for h, n in b["reqs"]])
        for r, row in enumerate(b["tables"]):
            assert plan.block_tables[r, : len(row)].tolist() == row, bi
        want = var["last_hit_blocks"] if (bi == len(case["batches"]) - 1 and "last_hit_blocks" in var) \
            else b["hit_blocks"]
        assert plan.hit_blocks.tolist() == want, bi
        evs = cache.log()[n0:]
        if "cases" in b:
            assert [case_names[e[1]] for e in evs] == b["cases"]
        if "dropped" in b:
            assert [e[4] for e in evs] == b["dropped"]
        cache.release_batch()
    f = case["final"]
    lists = [[int(k) for k in cache.snapshot(li)[0]] for li in (ak.LIST_T1, ak.LIST_T2, ak.LIST_B1, ak.LIST_B2)]
    assert lists == [f["T1"], f["T2"], f["B1"], f["B2"]]
    assert cache.stats()["p"] == f["p"]


def test_tiny_config_host_phase():
    cfg = get_config("tiny")
    order = free_order(cfg.seed, cfg.num_phys)
    pair = Pair("arc", cfg.capacity, cfg.num_phys, cfg.scratch, order)
    r0, r1 = make_stream(cfg)
    pair.run([r0.tokens])
    p, _ = pair.run([r1.tokens])
    assert p.hit_blocks.tolist() == [16] and p.cu_q.tolist() == [0, 64]
    pair.check_log_and_state()


def test_docqa_stream_host_phase_and_batching():
    cfg = get_config("docqa")
    order = free_order(cfg.seed, cfg.num_phys)
    stream = make_stream(cfg, n_batches=24)
    lens = [r.n_tokens for r in stream]
    batches = form_batches(lens, cfg.max_batch, cfg.capacity, cfg.scratch)
    # the library's batch formation agrees with the oracle's
    i, lib_batches = 0, []
    while i < len(lens):
        n = ak.next_batch(lens[i:], cfg.max_batch, cfg.capacity, cfg.scratch)
        lib_batches.append((i, i + n))
        i += n
    assert lib_batches == batches
    pair = Pair("arc", cfg.capacity, cfg.num_phys, cfg.scratch, order)
    hits = 0
    for a, b in batches:
        p, _ = pair.run([r.tokens for r in stream[a:b]])
        hits += int(p.prefix_lens.sum())
    pair.check_log_and_state()
    assert hits > 0
    warm, hot = stream_docqa_hit(cfg)
    pair2 = Pair("arc", cfg.capacity, cfg.num_phys, cfg.scratch, order)
    pair2.run([r.tokens for r in warm])
    p, _ = pair2.run([r.tokens for r in hot])
    assert p.prefix_lens.tolist() == [8192] * 8 and p.cu_q[-1] == 8 * 128
    pair2.check_log_and_state()


def test_longctx_host_phase():
    cfg = get_config("longctx")
    order = free_order(cfg.seed, cfg.num_phys)
    warm, hot = make_stream(cfg)
    pair = Pair("arc", cfg.capacity, cfg.num_phys, cfg.scratch, order)
    pair.run([r.tokens for r in warm])
    p, _ = pair.run([r.tokens for r in hot])
    assert p.prefix_lens.tolist() == [32768] * 4 and p.cu_q.tolist() == [0, 2048, 4096, 6144, 8192]
    pair.check_log_and_state()


def test_error_statuses_match_the_oracle():
    cfg = get_config("tiny")
    lib = ak.BlockCache("arc", 8, 16, 4)
    orc = Planner("arc", 8, 16, 4)
    big = make_request(cfg, [(Source(KIND_DOC, 1, 144), 0, 144)]).tokens
    with pytest.raises(ak.ArckvError) as e1:
        lib.plan_batch([(ak.hash_blocks(big), len(big))])
    with pytest.raises(PlanError) as e2:
        orc.plan_batch([(obh.hash_blocks(big), len(big))])
    assert e1.value.code == e2.value.code == "ENOSPC"
    with pytest.raises(ak.ArckvError) as e1:
        lib.release_batch()
    assert e1.value.code == "ESTATE"
    small = big[:40]
    with pytest.raises(ak.ArckvError) as e1:
        lib.plan_batch([(ak.hash_blocks(small)[:1], len(small))])
    assert e1.value.code == "EINVAL"
    lib.plan_batch([(ak.hash_blocks(small), len(small))])
    with pytest.raises(ak.ArckvError) as e1:
        lib.plan_batch([(ak.hash_blocks(small), len(small))])
    assert e1.value.code == "ESTATE"
    lib.release_batch()
    assert lib.stats()["in_flight"] == 0
    with pytest.raises(ak.ArckvError):
        ak.BlockCache("arc", 10, 12, 4)              # pool too small for c + scratch
    with pytest.raises(ak.ArckvError):
        ak.BlockCache("arc", 4, 8, 2, initial_order=[0, 1, 2, 3, 4, 5, 6, 6])
    with pytest.raises(ak.ArckvError):
        ak.BlockCache("frc", 4, 8, 2, frc_p=4.5)      # p outside [0, c]
    for bad_window in (-1, 4097):
        with pytest.raises(ak.ArckvError) as e2:
            ak.BlockCache("lru", 4, 8, 2, victim_window=bad_window)
        assert e2.value.code == "EINVAL"


ITEM_COST = 4   # the list planner's cost of one item, in key tiles (kItemCost)


def attention_plan_coverage(cu_q, seq_lens, hq, hkv, d, num_cus):
    ap = ak.attention_plan(cu_q, seq_lens, hq, hkv, d, num_cus)
    g = hq // hkv
    tc = ap.tile_cols
    max_cols = max(int(cu_q[r + 1] - cu_q[r]) * g for r in range(len(seq_lens)))
    assert tc == (128 if max_cols <= 128 else 256)
    items = ap.work[: ap.n_work]
    comb = ap.work[ap.n_work: ap.n_work + ap.n_combine]
    lists = tc == 128               # narrow plans: one list of 8 entries per work-group
    if lists:
        assert ap.n_work % 8 == 0
        for lst in items.reshape(-1, 8, 8):
            live = lst[:, 0] >= 0
            assert live[0] and not (live[1:] & ~live[:-1]).any()    # live items, then padding
    cover, n_live, n_slots, max_piece = {}, 0, 0, 0
    for it in items:
        req, kvh, cs, a, b, slot = (int(x) for x in it[:6])
        if req < 0:
            continue
        n_live += 1
        n_slots += slot >= 0
        assert a % 64 == 0 and b > a
        max_piece = max(max_piece, (b - a + 63) // 64)
        cover.setdefault((req, kvh, cs), []).append((a, b, slot))
    n_tiles, total_tiles, min_pieces = 0, 0, 0
    for r in range(len(seq_lens)):
        S = cu_q[r + 1] - cu_q[r]
        P = seq_lens[r] - S
        for cs in range(0, S * g, tc):
            last = min(cs + tc, S * g) - 1
            kv_end = P + last // g + 1
            n_tiles += hkv
            total_tiles += hkv * (-(-kv_end // 64))
            min_pieces += hkv * max(1, -(-(-(-kv_end // 64)) // 1024))
            for h in range(hkv):
                ranges = sorted(cover.pop((r, h, cs)))
                assert ranges[0][0] == 0 and ranges[-1][1] == kv_end
                assert all(x[1] == y[0] for x, y in zip(ranges, ranges[1:]))
                if len(ranges) == 1:
                    assert ranges[0][2] == -1
                else:
                    slots = [x[2] for x in ranges]
                    assert slots == list(range(slots[0], slots[0] + len(slots)))
                    sizes = [(x[1] - x[0] + 63) // 64 for x in ranges]
                    if lists:   # cuts leave no piece under 4 key tiles
                        assert min(sizes) >= 4
                    else:       # pieces of whole key tiles, as equal as whole tiles allow
                        assert max(sizes) - min(sizes) <= 1
                    assert any(list(c[:5]) == [r, h, cs, slots[0], len(slots)] for c in comb)
    assert not cover
    base = n_tiles
    share = max(8, -(-total_tiles // num_cus))
    if lists:
        # at most one list per CU unless the 8-entry lists force more; equal cost per list
        # (key tiles + ITEM_COST per item) up to what a budget cut can leave unused
        n_lists = ap.n_work // 8
        n_target = max(num_cus, -(-min_pieces // 8))
        assert n_lists <= n_target
        costs, full = [], False
        for lst in items.reshape(-1, 8, 8):
            live = lst[lst[:, 0] >= 0]
            full |= len(live) == 8
            costs.append(int(((live[:, 4] - live[:, 3] + 63) // 64).sum()) + ITEM_COST * len(live))
        # a list closes with at most 2 * 4 - 1 key tiles + one item's cost unused
        fair = -(-(total_tiles + ITEM_COST * min_pieces) // n_target)
        assert full or max(costs) <= max(fair + 8 + ITEM_COST, max_piece + ITEM_COST)
    elif base < num_cus:
        assert n_live <= num_cus          # split into one round: at most one item per CU
    else:
        assert max_piece <= max(share, 1)  # several rounds: no piece beyond one CU's share
    if n_slots:
        slot_bytes = tc * (d + 1) * 4
        assert ap.ws_bytes == n_slots * slot_bytes
    else:
        assert ap.ws_bytes == 0
    return ap


def test_attention_plan_covers_every_tile_once():
    attention_plan_coverage([0, 64], [320], 4, 2, 64, 256)
    ap = attention_plan_coverage(np.cumsum([0] + [128] * 8).tolist(), [8320] * 8, 32, 8, 128, 256)
    assert ap.n_combine == 128 and ap.ws_bytes > 0         # short suffixes: split key ranges
    ap = attention_plan_coverage([0, 16], [32784], 32, 8, 128, 256)
    assert ap.n_combine == 8 and ap.n_work // 8 <= 256      # one list per CU at most
    ap = attention_plan_coverage([0, 2048, 4096, 6144, 8192], [34816] * 4, 64, 8, 128, 256)
    assert ap.n_combine == 0                                # plenty of tiles: no split
    rng = np.random.default_rng(3)
    S = rng.integers(1, 700, 10)
    L = S + 16 * rng.integers(0, 300, 10)
    attention_plan_coverage(np.concatenate([[0], np.cumsum(S)]).tolist(), L.tolist(), 32, 8, 128, 256)
    attention_plan_coverage([0, 1], [1], 8, 1, 128, 256)
    # G = 5 (40 / 8 heads): tiles of 256 columns end inside a token's group of heads
    attention_plan_coverage(np.concatenate([[0], np.cumsum(S)]).tolist(), L.tolist(), 40, 8, 128, 256)
    attention_plan_coverage([0, 51, 103], [4000, 103], 40, 8, 128, 256)


def test_list_plans_cover_and_balance():
    """Narrow batches (at most 128 columns per request): per-work-group lists of 8 entries,
    about equal cost per list, no cut piece under 4 key tiles."""
    rng = np.random.default_rng(11)
    hist = np.clip(np.exp(rng.normal(7.5, 0.8, 256)), 256, 16384).astype(np.int64) // 16 * 16
    for S, n, hq, hkv, cus in ((32, 16, 32, 8, 256), (1, 64, 32, 8, 256), (16, 16, 32, 8, 256),
                               (1, 64, 32, 8, 100000), (25, 9, 40, 8, 256), (1, 3, 8, 1, 4),
                               (64, 5, 16, 8, 256), (128, 2, 8, 8, 256)):
        L = (hist[:n] + S).tolist()
        cu = (np.arange(n + 1) * S).tolist()
        ap = attention_plan_coverage(cu, L, hq, hkv, 128, cus)
        assert ap.tile_cols == 128
    # many tiny requests: the 8-entry lists, not the CU count, bound the lists
    n = 700
    ap = attention_plan_coverage(list(range(n + 1)), [40] * n, 32, 8, 128, 256)
    assert ap.n_work // 8 == -(-n * 8 // 8) and ap.n_combine == 0
    # a history longer than one item's key cap (65536 keys) is cut even when nothing else is
    ap = attention_plan_coverage([0, 1], [200000], 8, 1, 128, 4)
    w = ap.work[: ap.n_work]
    assert (w[w[:, 0] >= 0, 4] - w[w[:, 0] >= 0, 3] <= 65536).all()


def test_attention_plan_caps_the_keys_of_one_item():
    """No work item covers more than 65536 keys (the attention kernel keeps an item's block-table
    slice in LDS): long key ranges are split even where the tiles alone would fill the CUs."""
    for cu, L, hq, hkv, cus in (([0, 2048, 4096], [140000, 100000], 64, 8, 256),   # plenty of tiles
                                ([0, 16], [300000], 32, 8, 256),                    # one short suffix
                                ([0, 1, 2], [70000, 65600], 8, 1, 4)):               # decode-like
        ap = attention_plan_coverage(cu, L, hq, hkv, 128, cus)
        w = ap.work[: ap.n_work]
        live = w[:, 0] >= 0
        assert (w[live, 4] - w[live, 3] <= 65536).all()
        assert ap.n_combine > 0


def test_attention_plan_places_a_group_on_one_xcd():
    cu = np.cumsum([0] + [2048] * 4).tolist()
    ap = ak.attention_plan(cu, [34816] * 4, 64, 8, 128, 256)
    xcd_of = {}
    for i, it in enumerate(ap.work[: ap.n_work]):
        if it[0] < 0:
            continue
        key = (int(it[0]), int(it[1]))
        assert xcd_of.setdefault(key, i % 8) == i % 8


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_attention_plan_order_is_xcd_phased_and_longest_first(seed):
    # Work-group i of a launch runs on XCD i % 8.  The order the planner emits keeps every
    # (request, KV head) group on one XCD when there are at least 8 groups, lists each XCD's
    # items longest first (items within ~10 % of each other may come in any order), pads with
    # idle slots (request -1) only to keep that phase, and never ends on an idle slot.
    rng = np.random.default_rng(seed)
    n = int(rng.integers(6, 40))
    S = rng.integers(1, [40, 300, 3000, 600][seed], n)
    L = S + 16 * rng.integers(0, 600, n)
    hkv = [8, 2, 8, 1][seed]
    hq = hkv * [4, 8, 4, 5][seed]
    ap = ak.attention_plan(np.concatenate([[0], np.cumsum(S)]), L, hq, hkv, 128, 256)
    assert ap.tile_cols == 256          # (narrow batches use per-work-group lists instead)
    items = ap.work[: ap.n_work]
    assert ap.n_work == 0 or items[-1][0] >= 0
    groups = {(int(it[0]), int(it[1])) for it in items if it[0] >= 0}
    xcd_of, last_cost = {}, [None] * 8
    for i, it in enumerate(items):
        req, kvh, _, a, b = (int(x) for x in it[:5])
        if req < 0:
            continue
        x = i % 8
        if len(groups) >= 8:
            assert xcd_of.setdefault((req, kvh), x) == x
        cost = b - a
        if last_cost[x] is not None:
            assert cost <= last_cost[x] * 1.1 + 1
        last_cost[x] = cost
