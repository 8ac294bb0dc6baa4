"""Seeded request streams and bf16 Q/K/V tensors for the workload configurations.

A *source* is a seeded token sequence with its own Q/K/V rows: a document, a
question, a conversation session, a one-off document.  A request's prompt is
a concatenation of source segments; the Q/K/V row of prompt position j is the
row of the source position it came from, so a document prefix always carries
identical K/V bytes whenever it is seen again (what prefix caching relies on).
Inputs are synthetic: token ids uniform over the vocabulary, Q/K/V i.i.d.
N(0, 1) rounded to bf16 (round-to-nearest-even).
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .configs import VOCAB, Config

KIND_DOC, KIND_QUESTION, KIND_SESSION, KIND_ONEOFF, KIND_STREAM = 0, 1, 2, 3, 4
TAG_TOKENS, TAG_Q, TAG_K, TAG_V = 0, 1, 2, 3


def derive_seed(cfg_seed: int, kind: int, index: int, tag: int) -> int:
    return int(np.random.SeedSequence([cfg_seed, kind, index, tag]).generate_state(1, np.uint64)[0]
               & np.uint64(0x7FFFFFFFFFFFFFFF))


@dataclass(frozen=True)
class Source:
    kind: int
    index: int
    length: int


@dataclass
class Request:
    segments: list            # [(Source, start, length)]
    tokens: np.ndarray        # int32 [n_tokens]

    @property
    def n_tokens(self) -> int:
        return int(self.tokens.shape[0])


_token_cache: dict = {}


def source_tokens(cfg: Config, src: Source) -> np.ndarray:
    key = (cfg.seed, src.kind, src.index, src.length)
    t = _token_cache.get(key)
    if t is None:
        rng = np.random.default_rng(derive_seed(cfg.seed, src.kind, src.index, TAG_TOKENS))
        t = rng.integers(0, VOCAB, size=src.length, dtype=np.int64).astype(np.int32)
        if len(_token_cache) > 4096:
            _token_cache.clear()
        _token_cache[key] = t
    return t


def make_request(cfg: Config, segments) -> Request:
    toks = [source_tokens(cfg, s)[a:a + n] for (s, a, n) in segments]
    return Request(list(segments), np.concatenate(toks).astype(np.int32))


def free_order(seed: int, num_phys: int) -> np.ndarray:
    """Seeded initial order of the physical blocks (a permutation of the pool)."""
    return np.random.default_rng(seed).permutation(num_phys).astype(np.int32)


def zipf_probs(n: int, s: float) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


# ---------------------------------------------------------------------------------------------
# streams
# ---------------------------------------------------------------------------------------------

def stream_tiny(cfg: Config):
    e = cfg.extra
    doc = Source(KIND_DOC, 0, e["doc_tokens"])
    q = Source(KIND_QUESTION, 0, e["suffix_tokens"])
    r0 = make_request(cfg, [(doc, 0, doc.length)])
    r1 = make_request(cfg, [(doc, 0, doc.length), (q, 0, q.length)])
    return [r0, r1]


def stream_docqa(cfg: Config, n_batches: int | None = None):
    e = cfg.extra
    n_batches = e["n_batches"] if n_batches is None else n_batches
    rng = np.random.default_rng(derive_seed(cfg.seed, KIND_STREAM, 0, 0))
    rank_to_doc = rng.permutation(e["n_docs"])
    ranks = rng.choice(e["n_docs"], size=n_batches * cfg.max_batch, p=zipf_probs(e["n_docs"], e["zipf_s"]))
    out = []
    for i, rk in enumerate(ranks):
        doc = Source(KIND_DOC, int(rank_to_doc[rk]), e["doc_tokens"])
        q = Source(KIND_QUESTION, i, e["question_tokens"])
        out.append(make_request(cfg, [(doc, 0, doc.length), (q, 0, q.length)]))
    return out


def stream_docqa_hit(cfg: Config):
    """Eight distinct documents (a warm pass, then the same documents with new questions)."""
    e = cfg.extra
    warm, hot = [], []
    for i in range(cfg.max_batch):
        doc = Source(KIND_DOC, i, e["doc_tokens"])
        warm.append(make_request(cfg, [(doc, 0, doc.length)]))
        q = Source(KIND_QUESTION, 100000 + i, e["question_tokens"])
        hot.append(make_request(cfg, [(doc, 0, doc.length), (q, 0, q.length)]))
    return warm, hot


def stream_longctx(cfg: Config):
    e = cfg.extra
    warm, hot = [], []
    for i in range(e["n_docs"]):
        doc = Source(KIND_DOC, i, e["doc_tokens"])
        q = Source(KIND_QUESTION, i, e["suffix_tokens"])
        warm.append(make_request(cfg, [(doc, 0, doc.length)]))
        hot.append(make_request(cfg, [(doc, 0, doc.length), (q, 0, q.length)]))
    return warm, hot


def make_stream(cfg: Config, **kw):
    if cfg.name == "tiny":
        return stream_tiny(cfg)
    if cfg.name == "docqa":
        return stream_docqa(cfg, **kw)
    if cfg.name == "longctx":
        return stream_longctx(cfg)
    raise KeyError(cfg.name)


# ---------------------------------------------------------------------------------------------
# tensors
# ---------------------------------------------------------------------------------------------

def _randn_bf16(shape, seed: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)


class TensorBank:
    """Per-source Q/K/V rows (bf16) on one device, generated on first use."""

    def __init__(self, cfg: Config, device="cpu", max_sources: int = 1 << 30):
        self.cfg = cfg
        self.device = device
        self.cache: dict = {}
        self.max_sources = max_sources

    def source(self, src: Source):
        key = (src.kind, src.index, src.length)
        t = self.cache.get(key)
        if t is None:
            c = self.cfg
            q = _randn_bf16((src.length, c.num_q_heads, c.head_dim),
                            derive_seed(c.seed, src.kind, src.index, TAG_Q), self.device)
            k = _randn_bf16((src.length, c.num_kv_heads, c.head_dim),
                            derive_seed(c.seed, src.kind, src.index, TAG_K), self.device)
            v = _randn_bf16((src.length, c.num_kv_heads, c.head_dim),
                            derive_seed(c.seed, src.kind, src.index, TAG_V), self.device)
            if len(self.cache) >= self.max_sources:
                self.cache.pop(next(iter(self.cache)))
            t = (q, k, v)
            self.cache[key] = t
        return t

    def rows(self, req: Request, start: int, end: int):
        """Q, K, V rows of prompt positions [start, end) of one request."""
        import torch
        qs, ks, vs = [], [], []
        pos = 0
        for (src, a, n) in req.segments:
            lo, hi = max(start, pos), min(end, pos + n)
            if lo < hi:
                q, k, v = self.source(src)
                qs.append(q[a + lo - pos: a + hi - pos])
                ks.append(k[a + lo - pos: a + hi - pos])
                vs.append(v[a + lo - pos: a + hi - pos])
            pos += n
        return torch.cat(qs), torch.cat(ks), torch.cat(vs)

    def batch_suffix(self, reqs, prefix_lens):
        """Q_new [sum S, Hq, D], K_new / V_new [sum S, Hkv, D] for the computed tokens of a batch."""
        import torch
        parts = [self.rows(r, int(p), r.n_tokens) for r, p in zip(reqs, prefix_lens)]
        return tuple(torch.cat([p[i] for p in parts]).contiguous() for i in range(3))


def bits(t) -> np.ndarray:
    """bf16 torch tensor -> uint16 numpy bit patterns (host copy)."""
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


# ---------------------------------------------------------------------------------------------
# measured step streams: warm-up batches (fill the cache) followed by timed batches that each
# carry fresh uncached tokens after cached prefixes
# ---------------------------------------------------------------------------------------------

def steps_docqa_hit(cfg: Config, n_steps: int):
    """Warm: 8 distinct documents.  Step k: the same documents + a fresh 128-token question."""
    e = cfg.extra
    docs = [Source(KIND_DOC, i, e["doc_tokens"]) for i in range(cfg.max_batch)]
    warm = [[make_request(cfg, [(d, 0, d.length)]) for d in docs]]
    steps = []
    for k in range(n_steps):
        steps.append([make_request(cfg, [(d, 0, d.length),
                                         (Source(KIND_QUESTION, 200000 + k * 16 + i, e["question_tokens"]),
                                          0, e["question_tokens"])]) for i, d in enumerate(docs)])
    return warm, steps


def steps_longctx(cfg: Config, n_steps: int):
    """Warm: 4 documents of 32768 tokens.  Step k: the same documents + a fresh 2048-token suffix."""
    e = cfg.extra
    docs = [Source(KIND_DOC, i, e["doc_tokens"]) for i in range(e["n_docs"])]
    warm = [[make_request(cfg, [(d, 0, d.length)]) for d in docs]]
    steps = []
    for k in range(n_steps):
        steps.append([make_request(cfg, [(d, 0, d.length),
                                         (Source(KIND_QUESTION, 300000 + k * 16 + i, e["suffix_tokens"]),
                                          0, e["suffix_tokens"])]) for i, d in enumerate(docs)])
    return warm, steps


def session_lengths(cfg: Config, n: int, seed_index: int = 0) -> np.ndarray:
    """Conversation histories: lognormal(mu, sigma) clipped, rounded down to whole blocks."""
    e = cfg.extra
    rng = np.random.default_rng(derive_seed(cfg.seed, KIND_STREAM, 10 + seed_index, 0))
    h = np.clip(np.round(np.exp(rng.normal(e["hist_mu"], e["hist_sigma"], n))), e["hist_min"], e["hist_max"])
    return (h.astype(np.int64) // 16) * 16


def steps_short(cfg: Config, n_steps: int, suffix: int, batch: int = 16, n_sessions: int = 64):
    """Short new turns over resident histories (the key-read-bound case).

    Warm: every session's history (block-aligned, so all of it is cached).  Step k: a batch of
    `batch` sessions, rotating through all sessions so consecutive steps read different KV,
    each with `suffix` fresh tokens after its history."""
    hist = session_lengths(cfg, n_sessions)
    srcs = [Source(KIND_SESSION, s, int(hist[s])) for s in range(n_sessions)]
    warm, cur, blocks = [], [], 0
    for s in srcs:
        if cur and (len(cur) == batch or blocks + s.length // 16 > cfg.capacity):
            warm.append(cur)
            cur, blocks = [], 0
        cur.append(make_request(cfg, [(s, 0, s.length)]))
        blocks += s.length // 16
    if cur:
        warm.append(cur)
    steps = []
    per = n_sessions // batch
    for k in range(n_steps):
        g = k % per
        steps.append([make_request(cfg, [(srcs[s], 0, srcs[s].length),
                                         (Source(KIND_QUESTION, 400000 + k * batch + j, suffix), 0, suffix)])
                      for j, s in enumerate(range(g * batch, (g + 1) * batch))])
    return warm, steps


# ---------------------------------------------------------------------------------------------
# configuration 3: multi-turn conversations; configuration 5: trace replay
# ---------------------------------------------------------------------------------------------

def stream_multiturn(cfg: Config, n_requests: int | None = None):
    """Requests of 64 conversation sessions, merged in arrival order.

    Session s starts with a history of h_s tokens, h_s = clip(round(exp(N(mu, sigma^2))),
    [hist_min, hist_max]).  Each request of the session is its whole history plus a new turn
    of U{turn_min..turn_max} tokens; the turn is then appended to the history.  A session
    whose next prompt would exceed hist_max tokens starts over with a fresh history (a new
    conversation of the same user).  Session activity w_s ~ Zipf(activity_s) over a seeded
    permutation; each session's requests arrive with exponential gaps of mean 1/w_s.
    Returns (requests, capacity in blocks = floor(cache_frac * sum_s h_s / 16)).
    """
    e = cfg.extra
    n_requests = e["n_requests"] if n_requests is None else n_requests
    n = e["n_sessions"]
    rng = np.random.default_rng(derive_seed(cfg.seed, KIND_STREAM, 3, 0))
    hist0 = np.clip(np.round(np.exp(rng.normal(e["hist_mu"], e["hist_sigma"], n))), e["hist_min"],
                    e["hist_max"]).astype(np.int64)
    perm = rng.permutation(n)
    w = np.empty(n)
    w[perm] = zipf_probs(n, e["activity_s"])
    # arrival times: per session a Poisson process of rate w_s; merge the first n_requests
    events = []
    for s in range(n):
        t = 0.0
        k = 0
        while True:
            t += rng.exponential(1.0 / w[s])
            events.append((t, s, k))
            k += 1
            if k > n_requests:
                break
    events.sort()
    events = events[:n_requests]
    turns = rng.integers(e["turn_min"], e["turn_max"] + 1, size=len(events))
    gen = np.zeros(n, dtype=np.int64)
    hist = hist0.copy()
    out = []
    max_len = e["hist_max"] + e["turn_max"]
    for (t, s, k), turn in zip(events, turns):
        if hist[s] + turn > max_len:                       # the conversation starts over
            gen[s] += 1
            hist[s] = hist0[s]
        src = Source(KIND_SESSION, int(s * 100000 + gen[s]), max_len)
        L = int(hist[s] + turn)
        out.append(make_request(cfg, [(src, 0, L)]))
        hist[s] = L
    capacity = int(e["cache_frac"] * hist0.sum() // 16)
    return out, capacity


def trace_docs(cfg: Config):
    """Lengths of the recurring documents of the trace (seeded)."""
    e = cfg.extra
    rng = np.random.default_rng(derive_seed(cfg.seed, KIND_STREAM, 5, 1))
    return rng.integers(e["doc_min"], e["doc_max"] + 1, size=e["n_docs"])


def stream_trace(cfg: Config, n_requests: int | None = None):
    """Trace replay: a recurring document drawn Zipf(s) (seeded rank permutation) with
    probability 1 - oneoff_frac, else a one-off fresh document (same length law); each request
    adds a fresh question of question_tokens tokens.
    Returns (requests, capacity = floor(cache_frac * sum of recurring document tokens / 16))."""
    e = cfg.extra
    n_requests = e["n_requests"] if n_requests is None else n_requests
    lens = trace_docs(cfg)
    rng = np.random.default_rng(derive_seed(cfg.seed, KIND_STREAM, 5, 2))
    rank_to_doc = rng.permutation(e["n_docs"])
    p = zipf_probs(e["n_docs"], e["zipf_s"])
    out = []
    n_oneoff = 0
    for i in range(n_requests):
        if rng.random() < e["oneoff_frac"]:
            L = int(rng.integers(e["doc_min"], e["doc_max"] + 1))
            doc = Source(KIND_ONEOFF, n_oneoff, L)
            n_oneoff += 1
        else:
            d = int(rank_to_doc[rng.choice(e["n_docs"], p=p)])
            doc = Source(KIND_DOC, d, int(lens[d]))
        q = Source(KIND_QUESTION, 500000 + i, e["question_tokens"])
        out.append(make_request(cfg, [(doc, 0, doc.length), (q, 0, q.length)]))
    capacity = int(e["cache_frac"] * lens.sum() // 16)
    return out, capacity


# ---------------------------------------------------------------------------------------------
# configuration 6: document QA with windowed Zipf sampling
# ---------------------------------------------------------------------------------------------

def wzqa_items(cfg: Config):
    """The QA items: (document index, question index, document length, question length).
    Document lengths U{doc_min..doc_max}, question lengths U{question_min..question_max},
    questions_per_doc items per document (seeded)."""
    e = cfg.extra
    rng = np.random.default_rng(derive_seed(cfg.seed, KIND_STREAM, 6, 1))
    doc_len = rng.integers(e["doc_min"], e["doc_max"] + 1, size=e["n_docs"])
    nq = e["questions_per_doc"]
    q_len = rng.integers(e["question_min"], e["question_max"] + 1, size=e["n_docs"] * nq)
    return [(d, d * nq + k, int(doc_len[d]), int(q_len[d * nq + k]))
            for d in range(e["n_docs"]) for k in range(nq)]


def wzqa_ranks(cfg: Config, n_requests: int | None = None):
    """Per request: (window, rank drawn, item index).  Window w = request // window; the
    ranks are i.i.d. Zipf(zipf_s) over all items; each window draws its own seeded
    permutation rank -> item, so popularity shifts at window boundaries."""
    e = cfg.extra
    n_requests = e["n_requests"] if n_requests is None else n_requests
    n_items = e["n_docs"] * e["questions_per_doc"]
    rng = np.random.default_rng(derive_seed(cfg.seed, KIND_STREAM, 6, 2))
    p = zipf_probs(n_items, e["zipf_s"])
    out = []
    n_windows = -(-n_requests // e["window"])
    for w in range(n_windows):                  # whole windows, so a shorter stream is a prefix
        rank_to_item = rng.permutation(n_items)
        for rk in rng.choice(n_items, size=e["window"], p=p):
            out.append((w, int(rk), int(rank_to_item[rk])))
    return out[:n_requests]


def stream_wzqa(cfg: Config, n_requests: int | None = None):
    """Document QA requests with windowed Zipf popularity: each request is its item's
    document followed by the item's question (token streams seeded per document and per
    question, so a repeated item repeats its whole prompt)."""
    items = wzqa_items(cfg)
    out = []
    for _, _, it in wzqa_ranks(cfg, n_requests):
        d, qi, dl, ql = items[it]
        out.append(make_request(cfg, [(Source(KIND_DOC, d, dl), 0, dl),
                                      (Source(KIND_QUESTION, qi, ql), 0, ql)]))
    return out


def sized(cfg: Config, capacity: int) -> Config:
    """The configuration with a stream-derived cache capacity and a pool of capacity + scratch."""
    import dataclasses
    return dataclasses.replace(cfg, capacity=int(capacity), num_phys=int(capacity) + cfg.scratch)
