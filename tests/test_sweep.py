"""Windowed-Zipf document-QA streams and the cache-size sweep (host only).

* The stream generator keeps the recipe of Sec. 4's document QA workloads: 3,072 requests,
  windows of 512, Zipf(1.0) over item ranks inside a window, the rank -> item map drawn
  afresh for every window.
* The sweep's per-request hit tokens and per-batch |T1|, |T2|, p come from the library;
  they equal the oracle planner's over the same stream for ARC, DBL and LRU.
* Independent pins: a cache that holds every distinct block reaches the compulsory-miss
  bound (brute force over a set of seen identities) under every policy; DBL's p never moves
  from c/2; an empty cache starts with everything in T1.
"""

import numpy as np
import pytest

from oracle import blockhash as obh
from oracle.planner import Planner, form_batches
import paper_2606_21238_amd as ak
from paper_2606_21238_amd import sweep
from workloads import get_config
from workloads.streams import stream_wzqa, wzqa_items, wzqa_ranks, zipf_probs


@pytest.mark.parametrize("name", ["wzqa_long", "wzqa_short"])
def test_windowed_zipf_recipe(name):
    cfg = get_config(name)
    e = cfg.extra
    ranks = wzqa_ranks(cfg)
    n_items = e["n_docs"] * e["questions_per_doc"]
    assert len(ranks) == e["n_requests"] == 3072 and e["window"] == 512 and e["zipf_s"] == 1.0
    windows = np.array([w for w, _, _ in ranks])
    assert (windows == np.arange(3072) // 512).all()
    # one rank maps to one item inside a window; the map changes between windows
    top = []
    for w in range(6):
        m = {}
        for ww, rk, it in ranks:
            if ww == w:
                assert m.setdefault(rk, it) == it
        top.append(m[0])
    assert len(set(top)) >= 5
    # rank frequencies over the whole stream follow Zipf(1): within 5 sigma for the top ranks
    rk = np.array([r for _, r, _ in ranks])
    p = zipf_probs(n_items, 1.0)
    for r in range(4):
        n = int((rk == r).sum())
        mu, sd = 3072 * p[r], np.sqrt(3072 * p[r] * (1 - p[r]))
        assert abs(n - mu) < 5 * sd, (r, n, mu)
    # requests are document + question of their item; items of one document share it
    items = wzqa_items(cfg)
    reqs = stream_wzqa(cfg, 64)
    assert wzqa_ranks(cfg, 64) == ranks[:64]
    for (w, r, it), req in zip(ranks[:64], reqs):
        d, qi, dl, ql = items[it]
        assert req.n_tokens == dl + ql
        assert e["doc_min"] <= dl <= e["doc_max"] and e["question_min"] <= ql <= e["question_max"]
    same_doc = [(a, b) for a in range(64) for b in range(a) if items[ranks[a][2]][0] == items[ranks[b][2]][0]]
    for a, b in same_doc[:5]:
        dl = items[ranks[a][2]][2]
        assert (reqs[a].tokens[:dl] == reqs[b].tokens[:dl]).all()


def oracle_replay(hashes, lens, policy, c, scratch):
    """Oracle planner over the stream: per-request hit tokens, per-batch (|T1|, |T2|, p)."""
    orc = Planner(policy, c, c + scratch, scratch)
    hit, series = [], []
    for a, b in form_batches(lens, 1, c, scratch):
        plan = orc.plan_batch([(hashes[j], lens[j]) for j in range(a, b)])
        hit += plan.prefix_lens
        orc.release_batch()
        if policy == "lru":
            series.append((len(orc.cache.L), 0, 0.0))
        else:
            series.append((len(orc.cache.T1), len(orc.cache.T2), orc.cache.p))
    return np.array(hit), series


@pytest.mark.parametrize("name,n_req,size", [("wzqa_short", 3072, 10000), ("wzqa_long", 384, 20000)])
def test_sweep_replay_equals_oracle(name, n_req, size):
    cfg = get_config(name)
    reqs = stream_wzqa(cfg, n_req)
    lens = [r.n_tokens for r in reqs]
    orc_hashes = obh.hash_blocks_many([r.tokens for r in reqs])
    lib_hashes = ak.hash_blocks_batch([r.tokens for r in reqs])
    c = size // 16
    rates = {}
    for policy in ("arc", "dbl", "lru"):
        got = sweep.replay(lib_hashes, lens, policy, c, cfg.scratch)
        want_hit, want_series = oracle_replay(orc_hashes, lens, policy, c, cfg.scratch)
        assert (got.hit_tokens == want_hit).all()
        assert got.batch_end.tolist() == list(range(1, n_req + 1))
        assert list(zip(got.t1.tolist(), got.t2.tolist(), got.p.tolist())) == want_series
        rates[policy] = got.hit_rate()
    # the recency/frequency split pays off on this stream; adaptation on top of it as well
    assert rates["arc"] > rates["lru"] and rates["arc"] >= rates["dbl"]


def compulsory_hit_tokens(hashes, lens):
    """Hit tokens with an unbounded cache: the leading blocks of a request already seen, one
    block fewer when that covers the whole (block-aligned) prompt."""
    seen, out = set(), []
    for h, L in zip(hashes, lens):
        k = 0
        while k < len(h) and h[k] in seen:
            k += 1
        if 16 * k == L:
            k -= 1
        out.append(16 * max(k, 0))
        seen.update(h)
    return np.array(out)


def test_unbounded_cache_reaches_the_compulsory_bound():
    cfg = get_config("wzqa_short")
    reqs = stream_wzqa(cfg, 1024)
    lens = [r.n_tokens for r in reqs]
    orc_hashes = obh.hash_blocks_many([r.tokens for r in reqs])
    want = compulsory_hit_tokens(orc_hashes, lens)
    c = len({x for h in orc_hashes for x in h})
    lib_hashes = ak.hash_blocks_batch([r.tokens for r in reqs])
    for policy in ("arc", "dbl", "lru"):
        got = sweep.replay(lib_hashes, lens, policy, c, cfg.scratch)
        assert (got.hit_tokens == want).all(), policy


def test_dbl_target_fixed_and_empty_cache_starts_in_t1():
    cfg = get_config("wzqa_long")
    reqs = stream_wzqa(cfg, 256)
    lens = [r.n_tokens for r in reqs]
    hashes = ak.hash_blocks_batch([r.tokens for r in reqs])
    c = 20000 // 16
    dbl = sweep.replay(hashes, lens, "dbl", c, cfg.scratch)
    assert (dbl.p == c / 2).all()
    arc = sweep.replay(hashes, lens, "arc", c, cfg.scratch)
    assert arc.t1_ratio()[0] == 1.0 and arc.t2[0] == 0
    assert ((arc.p >= 0) & (arc.p <= c)).all()
    assert ((arc.t1 + arc.t2) <= c).all()


def test_sweep_cli_table(capsys):
    assert sweep.main(["--workload", "wzqa_short", "--sizes", "5000,80000", "--requests", "512"]) == 0
    out = capsys.readouterr().out
    assert "| 5000 |" in out and "| 80000 |" in out and "512 requests" in out
