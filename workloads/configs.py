"""The five synthetic workload configurations (shapes, sizes, seeds).

Sizes are in tokens and blocks of 16 tokens; a cache capacity c is in blocks
(cache sizes quoted in tokens divided by 16).  The physical pool holds the c
cacheable pages plus ``scratch`` blocks for partial last blocks.
"""

from __future__ import annotations

from dataclasses import dataclass, field

VOCAB = 128256          # token-id range of a Llama-3-style tokenizer (ids only feed the hash)


@dataclass(frozen=True)
class Config:
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    capacity: int                 # c, in blocks
    scratch: int                  # blocks reserved for partial tails
    num_phys: int                 # pool size in blocks (>= capacity + scratch)
    max_batch: int
    policy: str = "arc"
    extra: dict = field(default_factory=dict)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def scale(self) -> float:
        return self.head_dim ** -0.5


CONFIGS = {
    # 1: single request on a tiny GQA layer; 16-block prefix placed by a seeded
    #    permutation of a 64-block pool; 64-token uncached suffix.
    "tiny": Config("tiny", 1001, 4, 2, 64, capacity=32, scratch=32, num_phys=64, max_batch=1,
                   extra=dict(doc_tokens=256, suffix_tokens=64)),
    # 2: document QA on a Llama-3-8B-shaped layer: 8 requests per batch, each an
    #    8192-token document drawn Zipf(1.1) from 64 documents + 128-token question;
    #    capacity 25 % of all document tokens.
    "docqa": Config("docqa", 1002, 32, 8, 128, capacity=8192, scratch=8, num_phys=8200, max_batch=8,
                    extra=dict(n_docs=64, doc_tokens=8192, question_tokens=128, zipf_s=1.1,
                               n_batches=64, warmup_batches=16)),
    # 2 on a Qwen3-14B-shaped layer (public configuration: 40 q / 8 kv heads, head_dim 128,
    #    hidden 5120, rotary base 1e6), with the Q/K/V projection in the step: the same stream,
    #    documents and cache as docqa.
    "docqa14b": Config("docqa14b", 1002, 40, 8, 128, capacity=8192, scratch=8, num_phys=8200, max_batch=8,
                       extra=dict(n_docs=64, doc_tokens=8192, question_tokens=128, zipf_s=1.1,
                                  n_batches=64, warmup_batches=16, hidden=5120, rope_theta=1.0e6)),
    # 3: multi-turn conversation, 8B shape: 64 sessions, lognormal histories,
    #    uniform new turns, Zipf(1.0) session activity, capacity 40 % of the working set.
    #    (capacity 0 = derived from the generated working set)
    "multiturn": Config("multiturn", 1003, 32, 8, 128, capacity=0, scratch=16, num_phys=0, max_batch=16,
                        extra=dict(n_sessions=64, hist_mu=7.5, hist_sigma=0.8, hist_min=256,
                                   hist_max=16384, turn_min=32, turn_max=512, activity_s=1.0,
                                   n_requests=1024, warmup_requests=256, cache_frac=0.4)),
    # 4: long-context QA on a 70B-shaped layer: 4 requests, 32768-token cached
    #    document + 2048-token suffix; prefix blocks scattered over a 16384-block pool.
    "longctx": Config("longctx", 1004, 64, 8, 128, capacity=16380, scratch=4, num_phys=16384, max_batch=4,
                      extra=dict(n_docs=4, doc_tokens=32768, suffix_tokens=2048)),
    # 3-short: the same layer shape, 16 sessions per batch each adding 32-64 new tokens to a
    #    fully cached lognormal history (the key-read-bound case); pool large enough for all
    #    64 histories.
    "short": Config("short", 1003, 32, 8, 128, capacity=16384, scratch=16, num_phys=16400, max_batch=16,
                    extra=dict(hist_mu=7.5, hist_sigma=0.8, hist_min=256, hist_max=16384)),
    # decode: one new token per request over a fully cached history (the KV-read-bound end of
    #    short suffixes): 256 sessions with lognormal(7.5, 0.8) histories clipped to [256, 16384]
    #    and rounded down to whole blocks, batches of 64 sessions rotating over all 256 (about
    #    2.7 GB of K/V in the pool, so consecutive steps read different KV).
    "decode": Config("decode", 1008, 32, 8, 128, capacity=65536, scratch=64, num_phys=65600, max_batch=64,
                     extra=dict(hist_mu=7.5, hist_sigma=0.8, hist_min=256, hist_max=16384, n_sessions=256)),
    # 5: trace replay: 10,000 requests over 500 documents of U[4096, 16384] tokens,
    #    Zipf(1.1) popularity, 30 % one-off documents; capacity 20 % of the working set.
    "trace": Config("trace", 1005, 32, 8, 128, capacity=0, scratch=16, num_phys=0, max_batch=16,
                    extra=dict(n_docs=500, doc_min=4096, doc_max=16384, zipf_s=1.1, oneoff_frac=0.3,
                               question_tokens=128, n_requests=10000, warmup_requests=2000,
                               cache_frac=0.2)),
    # 6: document QA with windowed Zipf sampling (Sec. 4, document QA): 3,072 requests in
    #    windows of 512; inside a window the QA items are drawn Zipf(1.0) by rank, and the
    #    rank -> item map is reshuffled for every window.  An item is a document plus one of
    #    its questions; items of one document share the document as prefix.  Two stand-ins:
    #    long articles with many questions each, and short passages with few.
    #    (capacity 0 = set by the sweep; host-only workloads)
    "wzqa_long": Config("wzqa_long", 1006, 32, 8, 128, capacity=0, scratch=16, num_phys=0, max_batch=1,
                        extra=dict(n_docs=128, doc_min=2048, doc_max=8192, questions_per_doc=8,
                                   question_min=24, question_max=96, n_requests=3072, window=512,
                                   zipf_s=1.0, sizes_tokens=[10000, 20000, 40000, 80000, 160000])),
    "wzqa_short": Config("wzqa_short", 1007, 32, 8, 128, capacity=0, scratch=16, num_phys=0, max_batch=1,
                         extra=dict(n_docs=1024, doc_min=256, doc_max=1536, questions_per_doc=2,
                                    question_min=12, question_max=48, n_requests=3072, window=512,
                                    zipf_s=1.0, sizes_tokens=[5000, 10000, 20000, 40000, 80000])),
}


def get_config(name: str) -> Config:
    return CONFIGS[name]
