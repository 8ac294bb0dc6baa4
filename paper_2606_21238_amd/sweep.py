"""Cache-size sweeps of the host block cache: hit-rate curves and T1-ratio series.

Sec. 4 compares ARC, DBL (the two queues at a fixed 1:1 split) and LRU by KV-cache hit
rate over several cache sizes, and follows the share of the cache held by the recency
queue T1 over the run (Fig. 7).  This module replays a seeded request stream through the
library's cache -- chained block hashing, batch formation and batch planning all in the
native library -- once per (policy, cache size), and reports

* the token hit rate: prefix-hit tokens / prompt tokens, over the requests after an
  optional warm-up (Sec. 4 warms the trace replay up before it measures);
* the T1 ratio |T1| / (|T1| + |T2|) after every batch, for ARC and DBL, summarised as
  quantiles and a down-sampled series; and ARC's target p / c beside it.

A policy may carry a victim window, ``arc@16``: length-aware eviction (Sec. 6 future work),
the deepest of the 16 least recently used unpinned pages of the list a policy evicts from.
``frc:0.25`` is the fixed-target policy FRC_p with p = 0.25 c (``dbl`` is ``frc:0.5``).

Usage::

    python -m paper_2606_21238_amd.sweep --workload wzqa_long
    python -m paper_2606_21238_amd.sweep --workload trace --policies arc,dbl,lru --json out.json
"""

from __future__ import annotations

import argparse
import json
import sys
import time
from dataclasses import dataclass, field

import numpy as np

from . import BLOCK_TOKENS, BlockCache, hash_blocks_batch, next_batch

POLICIES = ("arc", "dbl", "lru")


@dataclass
class Replay:
    policy: str
    capacity_blocks: int
    hit_tokens: np.ndarray             # int64 [n_requests]: prefix-hit tokens per request
    prompt_tokens: np.ndarray          # int64 [n_requests]
    batch_end: np.ndarray              # int64 [n_batches]: index after each batch's last request
    t1: np.ndarray                     # int64 [n_batches]: |T1| after each batch
    t2: np.ndarray                     # int64 [n_batches]: |T2| after each batch
    p: np.ndarray                      # float64 [n_batches]: target p after each batch
    stats: dict = field(default_factory=dict)

    def hit_rate(self, warmup: int = 0) -> float:
        den = int(self.prompt_tokens[warmup:].sum())
        return float(self.hit_tokens[warmup:].sum()) / den if den else 0.0

    def t1_ratio(self) -> np.ndarray:
        """|T1| / (|T1| + |T2|) after every batch (1.0 while the cache is empty)."""
        tot = self.t1 + self.t2
        return np.where(tot > 0, self.t1 / np.maximum(tot, 1), 1.0)


def parse_policy(name: str):
    """'arc' -> ('arc', 1, 0.0); 'lru@16' -> ('lru', 16, 0.0) (victim window);
    'frc:0.25@4' -> ('frc', 4, 0.25) (p as a fraction of c)."""
    base, _, w = name.partition("@")
    base, _, frac = base.partition(":")
    if base not in POLICIES + ("frc",) or (base == "frc") != bool(frac):
        raise ValueError(f"unknown policy {name!r}")
    return base, int(w) if w else 1, float(frac) if frac else 0.0


def replay(hashes, lens, policy: str, capacity: int, scratch: int, max_batch: int = 1,
           initial_order=None, ref_order: str = "tail_first") -> Replay:
    """Plans and releases every batch of the stream on a fresh cache of `capacity` pages and
    `capacity + scratch` physical blocks; hashes[j] are request j's chained block identities.
    `policy` may carry a victim window (``arc@16``)."""
    lens = np.asarray(lens, dtype=np.int64)
    n = len(lens)
    base, window, frac = parse_policy(policy)
    cache = BlockCache(base, capacity, capacity + scratch, scratch, initial_order, ref_order, window,
                       frc_p=frac * capacity)
    hit = np.zeros(n, dtype=np.int64)
    ends, t1, t2, p = [], [], [], []
    i = 0
    try:
        while i < n:
            b = next_batch(lens[i:i + 4 * max_batch], max_batch, capacity, scratch)
            if b == 0:
                raise ValueError(f"request {i} ({int(lens[i])} tokens) does not fit a cache of "
                                 f"{capacity} blocks with {scratch} scratch blocks")
            plan = cache.plan_batch([(hashes[j], int(lens[j])) for j in range(i, i + b)])
            hit[i:i + b] = plan.prefix_lens
            cache.release_batch()
            st = cache.stats()
            ends.append(i + b)
            t1.append(st["t1"])
            t2.append(st["t2"])
            p.append(st["p"])
            i += b
        stats = cache.stats()
    finally:
        cache.close()
    return Replay(policy, capacity, hit, lens.copy(), np.array(ends, dtype=np.int64),
                  np.array(t1, dtype=np.int64), np.array(t2, dtype=np.int64),
                  np.array(p, dtype=np.float64), stats)


# ---------------------------------------------------------------------------------------------
# workloads
# ---------------------------------------------------------------------------------------------

def load_workload(name: str, n_requests: int | None = None):
    """(config, requests, warm-up requests, default cache sizes in tokens) of a named stream."""
    from workloads import get_config
    from workloads import streams as ws

    cfg = get_config(name)
    e = cfg.extra
    if name in ("wzqa_long", "wzqa_short"):
        return cfg, ws.stream_wzqa(cfg, n_requests), 0, list(e["sizes_tokens"])
    if name == "multiturn":
        reqs, cap = ws.stream_multiturn(cfg, n_requests)
        base = cap * BLOCK_TOKENS
        return cfg, reqs, e["warmup_requests"], [int(base * f) for f in (0.25, 0.5, 1.0, 1.5, 2.0)]
    if name == "trace":
        reqs, cap = ws.stream_trace(cfg, n_requests)
        base = cap * BLOCK_TOKENS
        return cfg, reqs, e["warmup_requests"], [int(base * f) for f in (0.25, 0.5, 1.0, 1.5, 2.0)]
    if name == "docqa":
        n_batches = None if n_requests is None else -(-n_requests // cfg.max_batch)
        reqs = ws.stream_docqa(cfg, n_batches)
        base = cfg.capacity * BLOCK_TOKENS
        return cfg, reqs, e["warmup_batches"] * cfg.max_batch, [int(base * f) for f in (0.25, 0.5, 1.0, 2.0)]
    raise KeyError(f"unknown workload {name!r}")


def sweep(name: str, sizes_tokens=None, policies=POLICIES, max_batch: int = 1,
          n_requests: int | None = None, series_points: int = 48, log=None) -> dict:
    cfg, reqs, warmup, default_sizes = load_workload(name, n_requests)
    sizes_tokens = default_sizes if not sizes_tokens else list(sizes_tokens)
    lens = np.array([r.n_tokens for r in reqs], dtype=np.int64)
    t0 = time.perf_counter()
    hashes = hash_blocks_batch([r.tokens for r in reqs])
    distinct = len(np.unique(np.concatenate(hashes))) if hashes else 0
    out = {"workload": name, "requests": len(reqs), "warmup_requests": warmup, "batch": max_batch,
           "prompt_tokens": int(lens.sum()), "distinct_blocks": int(distinct),
           "hash_seconds": round(time.perf_counter() - t0, 3), "points": []}
    for size in sizes_tokens:
        c = int(size) // BLOCK_TOKENS
        row = {"cache_tokens": int(size), "capacity_blocks": c}
        for pol in policies:
            t = time.perf_counter()
            r = replay(hashes, lens, pol, c, cfg.scratch, max_batch)
            entry = {"hit_rate": round(r.hit_rate(warmup), 6), "seconds": round(time.perf_counter() - t, 3)}
            if parse_policy(pol)[0] != "lru":
                ratio = r.t1_ratio()
                q = np.quantile(ratio[r.batch_end > warmup] if warmup else ratio, [0.1, 0.5, 0.9])
                idx = np.unique(np.linspace(0, len(ratio) - 1, series_points).round().astype(int))
                entry.update(t1_ratio_p10=round(float(q[0]), 4), t1_ratio_median=round(float(q[1]), 4),
                             t1_ratio_p90=round(float(q[2]), 4),
                             series_request=[int(r.batch_end[k]) for k in idx],
                             series_t1_ratio=[round(float(ratio[k]), 4) for k in idx],
                             series_p_over_c=[round(float(r.p[k]) / c, 4) for k in idx])
            row[pol] = entry
            if log is not None:
                log(f"{name} {size:>8d} tokens {pol}: hit {entry['hit_rate']:.4f} ({entry['seconds']} s)")
        out["points"].append(row)
    return out


def format_table(res: dict, policies=POLICIES) -> str:
    head = f"| cache (tokens) | " + " | ".join(f"{p} hit" for p in policies) + \
           " | ARC - LRU | ARC T1 ratio p10/med/p90 | DBL T1 ratio med |"
    lines = [head, "|" + "---|" * (head.count("|") - 1)]
    for row in res["points"]:
        hits = [row[p]["hit_rate"] for p in policies if p in row]
        d = (row["arc"]["hit_rate"] - row["lru"]["hit_rate"]) if "arc" in row and "lru" in row else float("nan")
        a = row.get("arc", {})
        t = f"{a['t1_ratio_p10']:.2f}/{a['t1_ratio_median']:.2f}/{a['t1_ratio_p90']:.2f}" if a else "-"
        dm = f"{row['dbl']['t1_ratio_median']:.2f}" if "dbl" in row else "-"
        lines.append(f"| {row['cache_tokens']} | " + " | ".join(f"{h:.4f}" for h in hits) +
                     f" | {d:+.4f} | {t} | {dm} |")
    return "\n".join(lines)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="wzqa_long",
                    choices=["wzqa_long", "wzqa_short", "multiturn", "trace", "docqa"])
    ap.add_argument("--sizes", default="", help="comma-separated cache sizes in tokens")
    ap.add_argument("--policies", default=",".join(POLICIES))
    ap.add_argument("--batch", type=int, default=1, help="requests per batch (Sec. 4 default: 1)")
    ap.add_argument("--requests", type=int, default=None, help="use the first N requests only")
    ap.add_argument("--json", default="", help="write the full result (with series) here")
    args = ap.parse_args(argv)
    sizes = [int(s) for s in args.sizes.split(",") if s]
    pols = tuple(p for p in args.policies.split(",") if p)
    res = sweep(args.workload, sizes, pols, args.batch, args.requests,
                log=lambda m: print(m, file=sys.stderr, flush=True))
    print(f"{res['workload']}: {res['requests']} requests ({res['warmup_requests']} warm-up), "
          f"{res['prompt_tokens']} prompt tokens, {res['distinct_blocks']} distinct blocks, batch {res['batch']}")
    print(format_table(res, pols))
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
