"""GPU parity over request streams: multi-turn conversations and the trace replay.

The library engine (C++ cache and planner, HIP scatter and attention) and the oracle planner
run in lockstep over consecutive batches of one stream.  Every batch: block tables, slots and
prefix lengths equal to the oracle's (bit-exact).  Every checked batch, for every request: the
pool, read back through the request's block table with the oracle's gather, holds exactly the
K/V rows of all L prompt tokens (so hit blocks kept their bytes through the evictions and reuse
before them, and the suffix was scattered where the table says), and sampled suffix rows of the
attention output are within tolerance of the oracle's fp64 attention over those rows.
"""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

import paper_2606_21238_amd as ak  # noqa: E402
from paper_2606_21238_amd.engine import PrefillEngine  # noqa: E402
from oracle import attention as oatt  # noqa: E402
from oracle import blockhash as obh  # noqa: E402
from oracle import kvpool as okv  # noqa: E402
from oracle.planner import Planner, form_batches  # noqa: E402
from workloads import get_config  # noqa: E402
from workloads.streams import TensorBank, free_order, sized, stream_multiturn, stream_trace  # noqa: E402
from tests.gpu_helpers import bits, compare, print_case, sample_rows  # noqa: E402

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ak.lib()


class StreamRun:
    def __init__(self, cfg, max_sources):
        order = free_order(cfg.seed, cfg.num_phys)
        self.cfg = cfg
        self.eng = PrefillEngine(cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.capacity,
                                 cfg.num_phys, cfg.scratch, cfg.policy, order)
        self.orc = Planner(cfg.policy, cfg.capacity, cfg.num_phys, cfg.scratch, order)
        self.bank = TensorBank(cfg, DEV, max_sources=max_sources)
        self.hit_tokens = 0
        self.rows_checked = 0

    def batch(self, reqs, rng=None, side=None, busy=None):
        """side: run the engine's whole step (copy, scatter, attention) on this stream, after
        queueing `busy()` (long work) on torch's default stream."""
        cfg = self.cfg
        toks = [r.tokens for r in reqs]
        oplan = self.orc.plan_batch(list(zip(obh.hash_blocks_many(toks), map(len, toks))))
        q, kn, vn = self.bank.batch_suffix(reqs, oplan.prefix_lens)
        if side is None:
            db = self.eng.prepare(toks)          # hash + plan + work plan in one native call
            plan = db.plan
            out = torch.empty_like(q)
            self.eng.scatter(db, kn, vn)
            self.eng.attention(db, q, out)
        else:
            side.wait_stream(torch.cuda.current_stream())      # q / k / v were made on the default stream
            busy()
            plan, out = self.eng.step(toks, lambda p: (q, kn, vn), stream=side, release=False)
            side.synchronize()
        torch.cuda.synchronize()
        assert plan.prefix_lens.tolist() == oplan.prefix_lens
        assert plan.slot_mapping.tolist() == oplan.slot_mapping
        assert plan.cu_q.tolist() == oplan.cu_q
        for r, row in enumerate(oplan.block_tables):
            assert plan.block_tables[r, : len(row)].tolist() == row
        self.hit_tokens += sum(oplan.prefix_lens)
        if rng is not None:
            for r, req in enumerate(reqs):
                L, P = req.n_tokens, oplan.prefix_lens[r]
                q0, q1 = oplan.cu_q[r], oplan.cu_q[r + 1]
                table = np.asarray(oplan.block_tables[r], dtype=np.int64)
                idx = torch.from_numpy(table).to(DEV)
                mk, mv = bits(self.eng.k_pool[idx]), bits(self.eng.v_pool[idx])
                k, v = okv.gather(mk, mv, np.arange(len(table)), L)
                _, k_src, v_src = self.bank.rows(req, 0, L)
                assert np.array_equal(k, bits(k_src)), f"K of request {r} (L={L}, P={P})"
                assert np.array_equal(v, bits(v_src)), f"V of request {r} (L={L}, P={P})"
                rows = sample_rows(q1 - q0, rng, 6)
                ref = oatt.request_attention(bits(q[q0:q1]), k, v, P, cfg.scale, rows=rows)
                compare(bits(out[q0:q1]), ref, f"request {r} (L={L}, P={P})")
                self.rows_checked += len(rows)
        self.eng.release()
        self.orc.release_batch()


def run_stream(cfg, reqs, check_every, max_sources, seed):
    run = StreamRun(cfg, max_sources)
    rng = np.random.default_rng(seed)
    batches = form_batches([r.n_tokens for r in reqs], cfg.max_batch, cfg.capacity, cfg.scratch)
    for i, (a, b) in enumerate(batches):
        run.batch(reqs[a:b], rng if i % check_every == check_every - 1 else None)
    assert run.rows_checked > 0
    return run, len(batches)


def test_multiturn_stream():
    base = get_config("multiturn")
    reqs, cap = stream_multiturn(base)
    cfg = sized(base, cap)
    print_case(f"config multiturn: {len(reqs)} requests, capacity {cap} blocks, checks 1 batch in 4")
    run, n = run_stream(cfg, reqs, 4, 96, seed=31)
    print(f"multiturn: {n} batches, hit tokens {run.hit_tokens}, rows checked {run.rows_checked}", flush=True)
    assert run.hit_tokens > 0


def test_trace_replay_window():
    base = get_config("trace")
    reqs, cap = stream_trace(base, 1280)
    cfg = sized(base, cap)
    print_case(f"config trace: first {len(reqs)} requests, capacity {cap} blocks, checks 1 batch in 5")
    run, n = run_stream(cfg, reqs, 5, 48, seed=51)
    print(f"trace: {n} batches, hit tokens {run.hit_tokens}, rows checked {run.rows_checked}", flush=True)
    # the window runs past the point where the cache is full, so evicted blocks are reused
    assert run.orc.cache.log and any(e.evicted_from for e in run.orc.cache.log)


def test_step_on_a_side_stream_while_the_default_stream_is_busy():
    """The engine's step on a non-default stream: the metadata copy must be ordered before the
    kernels on that stream, not on torch's default stream, which here is held busy by a chain
    of large matmuls queued just before each step (a copy queued behind them would let the
    kernels read the block tables and slots of a batch four ring turns earlier)."""
    base = get_config("multiturn")
    reqs, cap = stream_multiturn(base)
    cfg = sized(base, cap)
    print_case(f"config multiturn on a side stream: first 10 batches, every batch checked")
    run = StreamRun(cfg, 96)
    side = torch.cuda.Stream()
    m = torch.randn(4096, 4096, device=DEV)

    def busy():
        for _ in range(6):
            torch.mm(m, m)

    rng = np.random.default_rng(17)
    batches = form_batches([r.n_tokens for r in reqs], cfg.max_batch, cfg.capacity, cfg.scratch)[:10]
    for a, b in batches:
        run.batch(reqs[a:b], rng, side=side, busy=busy)
    print(f"side stream: {len(batches)} batches, rows checked {run.rows_checked}", flush=True)
    assert run.rows_checked > 0 and run.hit_tokens > 0
