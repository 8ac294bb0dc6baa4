// Host block cache (ARC or LRU) and the per-batch planner.
//
// ARC as the paper's evictor (Sec. 3, Fig. 2): resident lists T1 (seen once recently) and
// T2 (seen again), ghost lists B1/B2 holding identities of pages evicted from T1/T2, and an
// adaptive target p for |T1| that B1 ghost hits raise and B2 ghost hits lower.  The exact
// rules are those of the ARC paper (Megiddo and Modha) the paper defers to:
//   I   hit in T1 u T2            -> MRU of T2
//   II  x in B1: p = min(p + d1, c), d1 = 1 if |B1| >= |B2| else |B2|/|B1|; REPLACE; -> T2
//   III x in B2: p = max(p - d2, 0), d2 = 1 if |B2| >= |B1| else |B1|/|B2|; REPLACE; -> T2
//   IV  new: if |T1|+|B1| = c { |T1| < c ? (drop LRU of B1, REPLACE) : drop LRU page of T1 }
//            else if |T1|+|T2|+|B1|+|B2| >= c { drop LRU of B2 when the total is 2c; REPLACE }
//            -> MRU of T1
//   REPLACE: T1 non-empty and (|T1| > p or (x in B2 and |T1| == p)) ? T1 LRU -> B1 : T2 LRU -> B2
// p is an IEEE binary64 value; sizes are compared with it exactly.
//
// DBL (Sec. 4: the two queues at a fixed 1:1 split) is the same machine with the adaptation
// off: p starts at c/2 and Cases II/III leave it there (the fixed-target FRC_p of the ARC
// paper).
//
// Serving additions (the paper is silent on them): pages used by the batch in flight are
// pinned and skipped by victim selection (falling back to the other resident list, whose
// ghost list then receives the page); a new page takes the evicted page's physical block or
// the head of a FIFO free list; partial last blocks use a separate scratch FIFO.
//
// Check mode (a safety net; the paper identifies blocks by hash alone): every resident page
// also keeps the block's digest, an independent second hash; before a plan changes anything,
// each block of a checked request whose identity is resident must match the stored digest, and
// blocks of the batch that share an identity must share the digest.
//
// Lists are intrusive doubly linked lists over a node array (head = LRU, tail = MRU) with an
// open-addressing index from identity to node (linear probing, backward-shift deletion, no
// per-entry allocation), so every reference is O(1) apart from skipping pinned pages at the
// LRU end.
#include <algorithm>
#include <deque>
#include <unordered_map>
#include <vector>

#include "internal.hpp"

namespace {

struct Node {
  uint64_t key = 0;
  uint64_t pin_epoch = 0;
  uint64_t born_epoch = 0;  // batch in which a miss or a ghost hit (re)made it resident
  int32_t phys = -1;
  int32_t prev = -1, next = -1;
  int32_t list = ARCKV_LIST_NONE;
  int32_t depth = 0;  // block index of the page in the prompt that last referenced it
  uint64_t digest = 0;  // check mode: digest of the block whose KV the page holds (0: unknown)
};

struct List {
  int32_t head = -1, tail = -1;  // head = LRU end, tail = MRU end
  int64_t size = 0;
};

// identity -> node index; at most 2c + 1 live entries, table at least 2x that (power of two)
class NodeIndex {
 public:
  void init(int64_t max_entries) {
    size_t cap = 16;
    while (cap < static_cast<size_t>(2 * max_entries + 16)) cap <<= 1;
    tab_.assign(cap, Entry{});
    mask_ = cap - 1;
  }
  int32_t find(uint64_t key) const {
    for (size_t i = slot(key);; i = (i + 1) & mask_) {
      const Entry& e = tab_[i];
      if (e.val < 0) return -1;
      if (e.key == key) return e.val;
    }
  }
  // start fetching the cache line a later find(key) begins its probe at
  void prefetch(uint64_t key) const { __builtin_prefetch(&tab_[slot(key)]); }
  void insert(uint64_t key, int32_t val) {  // key absent
    size_t i = slot(key);
    while (tab_[i].val >= 0) i = (i + 1) & mask_;
    tab_[i] = Entry{key, val, 0};
  }
  void erase(uint64_t key) {  // key present
    size_t i = slot(key);
    while (tab_[i].key != key || tab_[i].val < 0) i = (i + 1) & mask_;
    // backward-shift: pull later entries of the probe run into the hole
    for (size_t j = (i + 1) & mask_; tab_[j].val >= 0; j = (j + 1) & mask_) {
      const size_t home = slot(tab_[j].key);
      // entry j may move to the hole i iff its home is not cyclically in (i, j]
      const bool between = i <= j ? (home > i && home <= j) : (home > i || home <= j);
      if (!between) {
        tab_[i] = tab_[j];
        i = j;
      }
    }
    tab_[i].val = -1;
  }

 private:
  // key and value side by side: a lookup touches one cache line (four entries per line)
  struct Entry {
    uint64_t key = 0;
    int32_t val = -1;
    int32_t pad = 0;
  };
  size_t slot(uint64_t key) const { return static_cast<size_t>((key * 0x9E3779B97F4A7C15ull) >> 20) & mask_; }
  std::vector<Entry> tab_;
  size_t mask_ = 0;
};

struct Victim {
  uint64_t key = 0;
  int32_t from = ARCKV_LIST_NONE;
  int32_t phys = -1;
};

}  // namespace

struct arckv_cache {
  int32_t policy = ARCKV_POLICY_ARC;
  int32_t ref_order = ARCKV_REF_TAIL_FIRST;
  int32_t window = 1;  // victim window (length-aware eviction when > 1)
  bool intra_batch_reuse = true;
  bool check_blocks = false;
  int64_t c = 0;
  int64_t num_phys = 0;
  int64_t n_scratch = 0;
  double p = 0.0;

  List lists[5];
  std::vector<Node> nodes;
  std::vector<int32_t> free_nodes;
  NodeIndex index;
  std::deque<int32_t> free_blocks;
  std::deque<int32_t> scratch_fifo;
  std::vector<int32_t> batch_scratch;

  uint64_t epoch = 1;
  bool in_flight = false;
  int32_t scan_from[5] = {-1, -1, -1, -1, -1};  // per list: see lru_unpinned
  uint64_t scan_epoch[5] = {0, 0, 0, 0, 0};

  arckv_event* log_buf = nullptr;
  int64_t log_cap = 0;
  int64_t log_n = 0;

  int64_t references = 0, requests = 0, prompt_tokens = 0, prefix_hit_tokens = 0,
          computed_tokens = 0;
  int64_t case_counts[8] = {0, 0, 0, 0, 0, 0, 0, 0};

  // ---- list primitives ----------------------------------------------------------------
  void unlink(int32_t n) {
    Node& x = nodes[n];
    if ((x.list == ARCKV_LIST_T1 || x.list == ARCKV_LIST_T2) && scan_epoch[x.list] == epoch &&
        scan_from[x.list] == n)
      scan_from[x.list] = x.next;  // every node before the successor is still pinned
    List& l = lists[x.list];
    if (x.prev >= 0) nodes[x.prev].next = x.next; else l.head = x.next;
    if (x.next >= 0) nodes[x.next].prev = x.prev; else l.tail = x.prev;
    x.prev = x.next = -1;
    l.size -= 1;
    x.list = ARCKV_LIST_NONE;
  }
  void push_mru(int32_t n, int32_t list) {
    Node& x = nodes[n];
    List& l = lists[list];
    x.list = list;
    x.prev = l.tail;
    x.next = -1;
    if (l.tail >= 0) nodes[l.tail].next = n; else l.head = n;
    l.tail = n;
    l.size += 1;
  }
  int32_t new_node(uint64_t key, int32_t phys) {
    int32_t n;
    if (!free_nodes.empty()) { n = free_nodes.back(); free_nodes.pop_back(); }
    else { n = static_cast<int32_t>(nodes.size()); nodes.emplace_back(); }
    Node& x = nodes[n];
    x = Node();
    x.key = key;
    x.phys = phys;
    index.insert(key, n);
    return n;
  }
  void erase_node(int32_t n) {
    index.erase(nodes[n].key);
    nodes[n].list = ARCKV_LIST_NONE;
    free_nodes.push_back(n);
  }
  bool pinned(int32_t n) const { return in_flight && nodes[n].pin_epoch == epoch; }
  // LRU-most unpinned page of T1 or T2.  Within a batch, pins are only added and every page
  // that enters T1 / T2 is pinned right away, so the pinned run at the LRU end only grows:
  // scan_from[list] (valid for the current epoch) is where the last scan stopped, and every
  // page before it is pinned.  Each batch therefore walks a pinned page at most once instead
  // of once per eviction.
  int32_t lru_unpinned(int32_t list) {
    const bool cached = in_flight && (list == ARCKV_LIST_T1 || list == ARCKV_LIST_T2) &&
                        scan_epoch[list] == epoch;
    int32_t n = cached ? scan_from[list] : lists[list].head;
    while (n >= 0 && pinned(n)) n = nodes[n].next;
    if (in_flight && (list == ARCKV_LIST_T1 || list == ARCKV_LIST_T2)) {
      scan_from[list] = n;
      scan_epoch[list] = epoch;
    }
    return n;
  }
  // The page a policy evicts from a resident list: the LRU-most unpinned page, or, with a
  // victim window W > 1, the deepest of the W least recently used unpinned pages (the first
  // such page on ties).  Only the first one moves the scan cursor.
  int32_t pick_victim(int32_t list) {
    const int32_t first = lru_unpinned(list);
    if (window <= 1 || first < 0) return first;
    int32_t best = first, seen = 1;
    for (int32_t m = nodes[first].next; m >= 0 && seen < window; m = nodes[m].next) {
      if (pinned(m)) continue;
      if (nodes[m].depth > nodes[best].depth) best = m;
      ++seen;
    }
    return best;
  }
  int32_t find(uint64_t key) const {
    return index.find(key);
  }
  bool resident(uint64_t key) const {
    const int32_t n = find(key);
    return n >= 0 && (nodes[n].list == ARCKV_LIST_T1 || nodes[n].list == ARCKV_LIST_T2);
  }
  // resident and, without intra-batch reuse, not born in the batch being planned
  bool reusable_node(int32_t n) const {
    return n >= 0 && (nodes[n].list == ARCKV_LIST_T1 || nodes[n].list == ARCKV_LIST_T2) &&
           (intra_batch_reuse || nodes[n].born_epoch != epoch);
  }
  void drop_lru(int32_t list, arckv_event& ev) {
    const int32_t n = lists[list].head;
    ev.dropped = nodes[n].key;
    ev.dropped_from = list;
    unlink(n);
    erase_node(n);
  }

  // ---- ARC --------------------------------------------------------------------------
  bool replace(bool x_in_b2, Victim& v) {
    const int64_t n1 = lists[ARCKV_LIST_T1].size;
    const bool prefer_t1 =
        n1 > 0 && (static_cast<double>(n1) > p || (x_in_b2 && static_cast<double>(n1) == p));
    int32_t first = prefer_t1 ? ARCKV_LIST_T1 : ARCKV_LIST_T2;
    int32_t second = prefer_t1 ? ARCKV_LIST_T2 : ARCKV_LIST_T1;
    int32_t src = first;
    int32_t n = pick_victim(first);
    if (n < 0) { src = second; n = pick_victim(second); }
    if (n < 0) return false;
    v.key = nodes[n].key;
    v.from = src;
    v.phys = nodes[n].phys;
    unlink(n);
    nodes[n].phys = -1;
    push_mru(n, src == ARCKV_LIST_T1 ? ARCKV_LIST_B1 : ARCKV_LIST_B2);
    return true;
  }

  int32_t take_free(int32_t& phys) {
    if (free_blocks.empty()) return arckv::fail(ARCKV_ENOSPC, "page free list exhausted");
    phys = free_blocks.front();
    free_blocks.pop_front();
    return ARCKV_OK;
  }

  // hint: x's node when the caller already looked it up (a pinned prefix page), else -1
  int32_t reference_arc(uint64_t x, int32_t hint, arckv_event& ev, int32_t& node_out) {
    const int64_t c_ = c;
    int32_t n = hint >= 0 ? hint : find(x);
    const int32_t where = n >= 0 ? nodes[n].list : ARCKV_LIST_NONE;
    Victim v;
    if (where == ARCKV_LIST_T1 || where == ARCKV_LIST_T2) {           // Case I
      unlink(n);
      push_mru(n, ARCKV_LIST_T2);
      ev.kase = ARCKV_CASE_I;
    } else if (where == ARCKV_LIST_B1 || where == ARCKV_LIST_B2) {    // Cases II / III
      const double b1 = static_cast<double>(lists[ARCKV_LIST_B1].size);
      const double b2 = static_cast<double>(lists[ARCKV_LIST_B2].size);
      const bool in_b2 = where == ARCKV_LIST_B2;
      if (policy != ARCKV_POLICY_ARC) {
        // DBL / FRC: the target stays where it was set
      } else if (!in_b2) {
        const double d1 = b1 >= b2 ? 1.0 : b2 / b1;
        p = std::min(p + d1, static_cast<double>(c_));
      } else {
        const double d2 = b2 >= b1 ? 1.0 : b1 / b2;
        p = std::max(p - d2, 0.0);
      }
      if (!replace(in_b2, v)) return arckv::fail(ARCKV_ENOSPC, "REPLACE: every page pinned");
      unlink(n);
      nodes[n].phys = v.phys;
      nodes[n].born_epoch = epoch;
      push_mru(n, ARCKV_LIST_T2);
      ev.kase = in_b2 ? ARCKV_CASE_III : ARCKV_CASE_II;
    } else {                                                          // Case IV
      const int64_t t1 = lists[ARCKV_LIST_T1].size, t2 = lists[ARCKV_LIST_T2].size;
      const int64_t b1 = lists[ARCKV_LIST_B1].size, b2 = lists[ARCKV_LIST_B2].size;
      int32_t phys = -1;
      if (t1 + b1 == c_) {
        if (t1 < c_) {                                                // IV-A
          drop_lru(ARCKV_LIST_B1, ev);
          if (!replace(false, v)) return arckv::fail(ARCKV_ENOSPC, "REPLACE: every page pinned");
          phys = v.phys;
          ev.kase = ARCKV_CASE_IVA;
        } else {                                                      // IV-A, |T1| = c
          const int32_t d = pick_victim(ARCKV_LIST_T1);
          if (d < 0) return arckv::fail(ARCKV_ENOSPC, "IV-A: every T1 page pinned");
          phys = nodes[d].phys;
          ev.dropped = nodes[d].key;
          ev.dropped_from = ARCKV_LIST_T1;
          unlink(d);
          erase_node(d);
          ev.kase = ARCKV_CASE_IVA_T1DEL;
        }
      } else {                                                        // IV-B
        const int64_t total = t1 + t2 + b1 + b2;
        if (total >= c_) {
          if (total == 2 * c_) drop_lru(ARCKV_LIST_B2, ev);
          if (!replace(false, v)) return arckv::fail(ARCKV_ENOSPC, "REPLACE: every page pinned");
          phys = v.phys;
        } else {
          const int32_t st = take_free(phys);
          if (st != ARCKV_OK) return st;
        }
        ev.kase = ARCKV_CASE_IVB;
      }
      n = new_node(x, phys);
      nodes[n].born_epoch = epoch;
      push_mru(n, ARCKV_LIST_T1);
    }
    ev.evicted = v.from != ARCKV_LIST_NONE ? v.key : 0;
    ev.evicted_from = v.from;
    ev.phys_block = nodes[n].phys;
    nodes[n].pin_epoch = epoch;
    node_out = n;
    return ARCKV_OK;
  }

  // ---- LRU --------------------------------------------------------------------------
  int32_t reference_lru(uint64_t x, int32_t hint, arckv_event& ev, int32_t& node_out) {
    int32_t n = hint >= 0 ? hint : find(x);
    if (n >= 0) {
      unlink(n);
      push_mru(n, ARCKV_LIST_T1);
      ev.kase = ARCKV_CASE_LRU_HIT;
    } else {
      int32_t phys = -1;
      if (lists[ARCKV_LIST_T1].size == c) {
        const int32_t vtm = pick_victim(ARCKV_LIST_T1);
        if (vtm < 0) return arckv::fail(ARCKV_ENOSPC, "LRU: every page pinned");
        phys = nodes[vtm].phys;
        ev.evicted = nodes[vtm].key;
        ev.evicted_from = ARCKV_LIST_T1;
        unlink(vtm);
        erase_node(vtm);
      } else {
        const int32_t st = take_free(phys);
        if (st != ARCKV_OK) return st;
      }
      n = new_node(x, phys);
      nodes[n].born_epoch = epoch;
      push_mru(n, ARCKV_LIST_T1);
      ev.kase = ARCKV_CASE_LRU_MISS;
    }
    ev.phys_block = nodes[n].phys;
    nodes[n].pin_epoch = epoch;
    node_out = n;
    return ARCKV_OK;
  }

  // digest: the block's digest in check mode, else 0 (unknown)
  int32_t reference(uint64_t x, int32_t hint, int32_t depth, uint64_t digest, int32_t& phys_out) {
    arckv_event ev{};
    ev.key = x;
    int32_t n = -1;
    const int32_t st = policy == ARCKV_POLICY_LRU ? reference_lru(x, hint, ev, n)
                                                  : reference_arc(x, hint, ev, n);
    if (st != ARCKV_OK) return st;
    nodes[n].depth = depth;
    // a hit keeps the KV (and the digest, unless this reference knows it); any other case
    // (re)writes the page's KV for this block
    const bool hit = ev.kase == ARCKV_CASE_I || ev.kase == ARCKV_CASE_LRU_HIT;
    if (!hit || digest != 0) nodes[n].digest = digest;
    ev.p_after = policy == ARCKV_POLICY_LRU ? 0.0 : p;
    phys_out = ev.phys_block;
    case_counts[ev.kase] += 1;
    references += 1;
    if (log_buf != nullptr && log_n < log_cap) log_buf[log_n] = ev;
    log_n += 1;
    return ARCKV_OK;
  }
};

// -------------------------------------------------------------------------------------------
// C ABI
// -------------------------------------------------------------------------------------------

extern "C" int32_t arckv_cache_create(const arckv_cache_cfg* cfg, arckv_cache** out) {
  if (cfg == nullptr || out == nullptr) return arckv::fail(ARCKV_EINVAL, "cache_create: NULL");
  *out = nullptr;
  if (cfg->policy != ARCKV_POLICY_ARC && cfg->policy != ARCKV_POLICY_LRU &&
      cfg->policy != ARCKV_POLICY_DBL && cfg->policy != ARCKV_POLICY_FRC)
    return arckv::fail(ARCKV_EINVAL, "cache_create: unknown policy %d", cfg->policy);
  if (cfg->policy == ARCKV_POLICY_FRC &&
      !(cfg->frc_p >= 0.0 && cfg->frc_p <= static_cast<double>(cfg->capacity_blocks)))
    return arckv::fail(ARCKV_EINVAL, "cache_create: frc_p %g not in [0, c]", cfg->frc_p);
  if (cfg->no_intra_batch_reuse != 0 && cfg->no_intra_batch_reuse != 1)
    return arckv::fail(ARCKV_EINVAL, "cache_create: no_intra_batch_reuse must be 0 or 1");
  if (cfg->ref_order != ARCKV_REF_TAIL_FIRST && cfg->ref_order != ARCKV_REF_HEAD_FIRST)
    return arckv::fail(ARCKV_EINVAL, "cache_create: unknown reference order");
  if (cfg->check_blocks != 0 && cfg->check_blocks != 1)
    return arckv::fail(ARCKV_EINVAL, "cache_create: check_blocks must be 0 or 1");
  if (cfg->victim_window < 0 || cfg->victim_window > 4096)
    return arckv::fail(ARCKV_EINVAL, "cache_create: victim window %d not in [0, 4096]", cfg->victim_window);
  if (cfg->capacity_blocks < 1 || cfg->scratch_blocks < 0 || cfg->num_phys_blocks > INT32_MAX / 16 ||
      cfg->num_phys_blocks - cfg->scratch_blocks < cfg->capacity_blocks)
    return arckv::fail(ARCKV_EINVAL,
                       "cache_create: need 1 <= capacity <= num_phys - scratch (c=%lld phys=%lld scratch=%lld)",
                       (long long)cfg->capacity_blocks, (long long)cfg->num_phys_blocks,
                       (long long)cfg->scratch_blocks);
  const int64_t np = cfg->num_phys_blocks;
  std::vector<int32_t> order(static_cast<size_t>(np));
  if (cfg->initial_free_order != nullptr) {
    std::vector<char> seen(static_cast<size_t>(np), 0);
    for (int64_t i = 0; i < np; ++i) {
      const int32_t b = cfg->initial_free_order[i];
      if (b < 0 || b >= np || seen[b]) return arckv::fail(ARCKV_EINVAL, "cache_create: initial order is not a permutation");
      seen[b] = 1;
      order[i] = b;
    }
  } else {
    for (int64_t i = 0; i < np; ++i) order[i] = static_cast<int32_t>(i);
  }
  auto* c = new (std::nothrow) arckv_cache();
  if (c == nullptr) return arckv::fail(ARCKV_ENOSPC, "cache_create: out of host memory");
  c->policy = cfg->policy;
  c->p = cfg->policy == ARCKV_POLICY_DBL   ? static_cast<double>(cfg->capacity_blocks) / 2.0
         : cfg->policy == ARCKV_POLICY_FRC ? cfg->frc_p
                                           : 0.0;
  c->intra_batch_reuse = cfg->no_intra_batch_reuse == 0;
  c->check_blocks = cfg->check_blocks == 1;
  c->ref_order = cfg->ref_order;
  c->window = cfg->victim_window < 1 ? 1 : cfg->victim_window;
  c->c = cfg->capacity_blocks;
  c->num_phys = np;
  c->n_scratch = cfg->scratch_blocks;
  const int64_t n_pages = np - cfg->scratch_blocks;
  c->free_blocks.assign(order.begin(), order.begin() + n_pages);
  c->scratch_fifo.assign(order.begin() + n_pages, order.end());
  c->nodes.reserve(static_cast<size_t>(2 * c->c + 8));
  c->index.init(2 * c->c + 8);
  *out = c;
  return ARCKV_OK;
}

extern "C" int32_t arckv_cache_destroy(arckv_cache* cache) {
  delete cache;
  return ARCKV_OK;
}

extern "C" int32_t arckv_next_batch(const int64_t* n_tokens, int32_t n_avail, int32_t max_batch,
                                    int64_t capacity, int64_t scratch, int32_t* n_take) {
  if (n_take == nullptr || n_avail < 0 || max_batch < 1 || (n_avail > 0 && n_tokens == nullptr))
    return arckv::fail(ARCKV_EINVAL, "next_batch: bad arguments");
  int64_t blocks = 0, tails = 0;
  int32_t j = 0;
  while (j < n_avail && j < max_batch) {
    const int64_t nf = n_tokens[j] / ARCKV_BLOCK_TOKENS;
    const int64_t tl = n_tokens[j] % ARCKV_BLOCK_TOKENS ? 1 : 0;
    if (blocks + nf > capacity || tails + tl > scratch) break;
    blocks += nf;
    tails += tl;
    ++j;
  }
  *n_take = j;
  if (j == 0 && n_avail > 0)
    return arckv::fail(ARCKV_ENOSPC, "next_batch: request alone exceeds capacity or scratch");
  return ARCKV_OK;
}

extern "C" int32_t arckv_plan_batch(arckv_cache* c, const arckv_req* reqs, int32_t n_reqs,
                                    arckv_plan* plan) {
  if (c == nullptr || plan == nullptr || n_reqs < 0 || (n_reqs > 0 && reqs == nullptr))
    return arckv::fail(ARCKV_EINVAL, "plan_batch: bad arguments");
  if (c->in_flight) return arckv::fail(ARCKV_ESTATE, "plan_batch: previous batch not released");
  if (plan->cu_q == nullptr || plan->seq_lens == nullptr || plan->prefix_lens == nullptr ||
      plan->hit_blocks == nullptr || plan->block_tables == nullptr || plan->slot_mapping == nullptr)
    return arckv::fail(ARCKV_EINVAL, "plan_batch: NULL output array");
  // validation before any state change
  int64_t total_blocks = 0, tails = 0, total_tokens = 0;
  for (int32_t r = 0; r < n_reqs; ++r) {
    const arckv_req& q = reqs[r];
    if (q.n_tokens < 1 || q.n_tokens > INT32_MAX / 2 || q.n_full != q.n_tokens / ARCKV_BLOCK_TOKENS ||
        (q.n_full > 0 && q.hashes == nullptr))
      return arckv::fail(ARCKV_EINVAL, "plan_batch: request %d: length/hash count mismatch", r);
    const int64_t nb = (q.n_tokens + ARCKV_BLOCK_TOKENS - 1) / ARCKV_BLOCK_TOKENS;
    if (nb > plan->bt_stride)
      return arckv::fail(ARCKV_ENOSPC, "plan_batch: request %d needs %lld table entries, stride %d",
                         r, (long long)nb, plan->bt_stride);
    total_blocks += q.n_full;
    tails += q.n_tokens % ARCKV_BLOCK_TOKENS ? 1 : 0;
    total_tokens += q.n_tokens;
  }
  if (total_blocks > c->c)
    return arckv::fail(ARCKV_ENOSPC, "plan_batch: %lld full blocks exceed capacity %lld",
                       (long long)total_blocks, (long long)c->c);
  if (tails > static_cast<int64_t>(c->scratch_fifo.size()))
    return arckv::fail(ARCKV_ENOSPC, "plan_batch: %lld partial blocks, %zu scratch blocks free",
                       (long long)tails, c->scratch_fifo.size());
  if (total_tokens > plan->slot_cap || total_tokens > INT32_MAX)
    return arckv::fail(ARCKV_ENOSPC, "plan_batch: slot capacity %lld < %lld prompt tokens",
                       (long long)plan->slot_cap, (long long)total_tokens);
  if (c->check_blocks) {
    // identity -> (digest, request, block) of its first occurrence in the batch
    struct First { uint64_t digest; int32_t req; int64_t block; };
    thread_local std::unordered_map<uint64_t, First> first;
    first.clear();
    for (int32_t r = 0; r < n_reqs; ++r) {
      const arckv_req& q = reqs[r];
      if (q.digests == nullptr) continue;
      for (int64_t i = 0; i < q.n_full; ++i) {
        const uint64_t key = q.hashes[i], dg = q.digests[i];
        const auto ins = first.emplace(key, First{dg, r, i});
        if (!ins.second) {
          const First& f = ins.first->second;
          if (f.digest != dg)
            return arckv::fail(ARCKV_ECOLLISION,
                               "plan_batch: identity %016llx: request %d block %lld and request %d "
                               "block %lld are different blocks",
                               (unsigned long long)key, f.req, (long long)f.block, r, (long long)i);
          continue;
        }
        const int32_t n = c->find(key);
        if (n >= 0 && (c->nodes[n].list == ARCKV_LIST_T1 || c->nodes[n].list == ARCKV_LIST_T2) &&
            c->nodes[n].digest != 0 && c->nodes[n].digest != dg)
          return arckv::fail(ARCKV_ECOLLISION,
                             "plan_batch: identity %016llx: request %d block %lld differs from the "
                             "resident page (physical block %d)",
                             (unsigned long long)key, r, (long long)i, c->nodes[n].phys);
      }
    }
  }

  c->in_flight = true;  // pins of this batch are live from here until release
  int64_t n_slots = 0;
  int32_t max_q = 0, max_l = 0;
  plan->cu_q[0] = 0;
  for (int32_t r = 0; r < n_reqs; ++r) {
    const arckv_req& q = reqs[r];
    const int64_t nf = q.n_full;
    int64_t k = 0;
    // the prefix's nodes, looked up once: pinned below and handed to their references
    thread_local std::vector<int32_t> prefix_node;
    prefix_node.resize(static_cast<size_t>(nf > 0 ? nf : 1));
    // Lookups run in chunks ahead of the reusability checks, with the index lines and then
    // the nodes fetched some blocks ahead (the table and the nodes are far larger than the
    // caches); the prefix is the run of leading reusable nodes.  Nothing changes state in
    // between, so lookups past the first miss (at most one chunk) are only wasted work.
    constexpr int64_t kAhead = 8, kChunk = 128;
    for (int64_t i = 0; i < std::min(nf, kAhead); ++i) c->index.prefetch(q.hashes[i]);
    int64_t looked = 0;
    while (looked < nf) {
      const int64_t end = std::min(nf, looked + kChunk);
      for (int64_t i = looked; i < end; ++i) {
        if (i + kAhead < nf) c->index.prefetch(q.hashes[i + kAhead]);
        const int32_t n = c->find(q.hashes[i]);
        prefix_node[i] = n;
        if (n >= 0) __builtin_prefetch(&c->nodes[n]);
      }
      looked = end;
      while (k < looked && c->reusable_node(prefix_node[k])) ++k;
      if (k < looked) break;
    }
    if (k * ARCKV_BLOCK_TOKENS == q.n_tokens) k -= 1;  // whole prompt cached: recompute last block
    for (int64_t i = 0; i < k; ++i) c->nodes[prefix_node[i]].pin_epoch = c->epoch;
    int32_t* row = plan->block_tables + static_cast<int64_t>(r) * plan->bt_stride;
    for (int64_t i = 0; i < nf; ++i) {
      const int64_t b = c->ref_order == ARCKV_REF_TAIL_FIRST ? nf - 1 - i : i;
      int32_t phys = -1;
      const uint64_t dg = c->check_blocks && q.digests != nullptr ? q.digests[b] : 0;
      const int32_t st = c->reference(q.hashes[b], b < k ? prefix_node[b] : -1, static_cast<int32_t>(b), dg, phys);
      if (st != ARCKV_OK) return st;  // unreachable with the capacity check above
      row[b] = phys;
    }
    int64_t nb = nf;
    if (q.n_tokens % ARCKV_BLOCK_TOKENS) {
      const int32_t blk = c->scratch_fifo.front();
      c->scratch_fifo.pop_front();
      c->batch_scratch.push_back(blk);
      row[nb++] = blk;
    }
    for (int64_t i = nb; i < plan->bt_stride; ++i) row[i] = -1;
    const int64_t P = k * ARCKV_BLOCK_TOKENS;
    const int64_t S = q.n_tokens - P;
    for (int64_t j = P; j < q.n_tokens; ++j)
      plan->slot_mapping[n_slots++] =
          row[j / ARCKV_BLOCK_TOKENS] * ARCKV_BLOCK_TOKENS + static_cast<int32_t>(j % ARCKV_BLOCK_TOKENS);
    plan->seq_lens[r] = static_cast<int32_t>(q.n_tokens);
    plan->prefix_lens[r] = static_cast<int32_t>(P);
    plan->hit_blocks[r] = static_cast<int32_t>(k);
    plan->cu_q[r + 1] = plan->cu_q[r] + static_cast<int32_t>(S);
    max_q = std::max<int32_t>(max_q, static_cast<int32_t>(S));
    max_l = std::max<int32_t>(max_l, static_cast<int32_t>(q.n_tokens));
    c->requests += 1;
    c->prompt_tokens += q.n_tokens;
    c->prefix_hit_tokens += P;
    c->computed_tokens += S;
  }
  plan->n_slots = n_slots;
  plan->max_q_len = max_q;
  plan->max_seq_len = max_l;
  return ARCKV_OK;
}

extern "C" int32_t arckv_release_batch(arckv_cache* c) {
  if (c == nullptr) return arckv::fail(ARCKV_EINVAL, "release_batch: NULL");
  if (!c->in_flight) return arckv::fail(ARCKV_ESTATE, "release_batch: no batch in flight");
  c->epoch += 1;
  c->in_flight = false;
  for (int32_t b : c->batch_scratch) c->scratch_fifo.push_back(b);
  c->batch_scratch.clear();
  return ARCKV_OK;
}

extern "C" int32_t arckv_cache_stats(const arckv_cache* c, arckv_stats* s) {
  if (c == nullptr || s == nullptr) return arckv::fail(ARCKV_EINVAL, "cache_stats: NULL");
  *s = arckv_stats{};
  s->t1 = c->lists[ARCKV_LIST_T1].size;
  s->t2 = c->lists[ARCKV_LIST_T2].size;
  s->b1 = c->lists[ARCKV_LIST_B1].size;
  s->b2 = c->lists[ARCKV_LIST_B2].size;
  s->p = c->p;
  s->capacity = c->c;
  s->references = c->references;
  s->requests = c->requests;
  s->prompt_tokens = c->prompt_tokens;
  s->prefix_hit_tokens = c->prefix_hit_tokens;
  s->computed_tokens = c->computed_tokens;
  for (int i = 0; i < 8; ++i) s->case_counts[i] = c->case_counts[i];
  s->free_blocks = static_cast<int64_t>(c->free_blocks.size());
  s->scratch_free = static_cast<int64_t>(c->scratch_fifo.size());
  s->in_flight = c->in_flight ? 1 : 0;
  s->policy = c->policy;
  return ARCKV_OK;
}

extern "C" int32_t arckv_cache_set_log(arckv_cache* c, arckv_event* buf, int64_t cap) {
  if (c == nullptr || cap < 0) return arckv::fail(ARCKV_EINVAL, "set_log: bad arguments");
  c->log_buf = buf;
  c->log_cap = buf == nullptr ? 0 : cap;
  c->log_n = 0;
  return ARCKV_OK;
}

extern "C" int32_t arckv_cache_log_count(const arckv_cache* c, int64_t* n) {
  if (c == nullptr || n == nullptr) return arckv::fail(ARCKV_EINVAL, "log_count: NULL");
  *n = c->log_n;
  return ARCKV_OK;
}

extern "C" int32_t arckv_cache_snapshot(const arckv_cache* c, int32_t list, uint64_t* keys,
                                        int32_t* phys, int64_t cap, int64_t* n) {
  if (c == nullptr || n == nullptr || list < ARCKV_LIST_T1 || list > ARCKV_LIST_B2)
    return arckv::fail(ARCKV_EINVAL, "snapshot: bad arguments");
  const int64_t size = c->lists[list].size;
  *n = size;
  if (size > cap) return arckv::fail(ARCKV_ENOSPC, "snapshot: list holds %lld", (long long)size);
  int64_t i = 0;
  for (int32_t x = c->lists[list].head; x >= 0; x = c->nodes[x].next, ++i) {
    if (keys != nullptr) keys[i] = c->nodes[x].key;
    if (phys != nullptr) phys[i] = c->nodes[x].phys;
  }
  return ARCKV_OK;
}

bool arckv::cache_checks_blocks(const arckv_cache* c) { return c != nullptr && c->check_blocks; }

// -------------------------------------------------------------------------------------------
// Checkpoint / resume: the whole state between batches as a flat little-endian image of
// 64-bit words (identities and digests as unsigned, the rest as signed, p as its IEEE bits).
// -------------------------------------------------------------------------------------------

namespace {

constexpr uint64_t kImageMagic = 0x31304356'4B435241ull;  // "ARCKVC01"
constexpr int64_t kImageVersion = 1;

struct Writer {
  uint64_t* out;
  int64_t cap, n = 0;
  void put(uint64_t v) {
    if (out != nullptr && n < cap) out[n] = v;
    ++n;
  }
  void put_i(int64_t v) { put(static_cast<uint64_t>(v)); }
};

struct Reader {
  const uint64_t* in;
  int64_t n, i = 0;
  bool ok = true;
  uint64_t get() {
    if (i >= n) { ok = false; return 0; }
    return in[i++];
  }
  int64_t get_i() { return static_cast<int64_t>(get()); }
};

}  // namespace

extern "C" int32_t arckv_cache_save(const arckv_cache* c, void* buf, int64_t cap, int64_t* n) {
  if (c == nullptr || n == nullptr || cap < 0) return arckv::fail(ARCKV_EINVAL, "cache_save: bad arguments");
  if (c->in_flight) return arckv::fail(ARCKV_ESTATE, "cache_save: a batch is in flight");
  Writer w{static_cast<uint64_t*>(buf), buf == nullptr ? 0 : cap / 8};
  w.put(kImageMagic);
  w.put_i(kImageVersion);
  for (int64_t v : {static_cast<int64_t>(c->policy), static_cast<int64_t>(c->ref_order),
                    static_cast<int64_t>(c->window), static_cast<int64_t>(c->intra_batch_reuse),
                    static_cast<int64_t>(c->check_blocks), c->c, c->num_phys, c->n_scratch})
    w.put_i(v);
  w.put(__builtin_bit_cast(uint64_t, c->p));
  for (int64_t v : {c->references, c->requests, c->prompt_tokens, c->prefix_hit_tokens, c->computed_tokens})
    w.put_i(v);
  for (int64_t v : c->case_counts) w.put_i(v);
  for (int list = ARCKV_LIST_T1; list <= ARCKV_LIST_B2; ++list) {
    w.put_i(c->lists[list].size);
    for (int32_t x = c->lists[list].head; x >= 0; x = c->nodes[x].next) {
      const Node& nd = c->nodes[x];
      w.put(nd.key);
      w.put_i(nd.phys);
      w.put_i(nd.depth);
      w.put(nd.digest);
    }
  }
  w.put_i(static_cast<int64_t>(c->free_blocks.size()));
  for (int32_t b : c->free_blocks) w.put_i(b);
  w.put_i(static_cast<int64_t>(c->scratch_fifo.size()));
  for (int32_t b : c->scratch_fifo) w.put_i(b);
  w.put(kImageMagic);
  *n = w.n * 8;
  if (buf != nullptr && cap < *n)
    return arckv::fail(ARCKV_ENOSPC, "cache_save: image takes %lld bytes, capacity %lld",
                       (long long)*n, (long long)cap);
  return ARCKV_OK;
}

extern "C" int32_t arckv_cache_restore(const void* buf, int64_t n, arckv_cache** out) {
  if (buf == nullptr || out == nullptr || n < 8 || n % 8 != 0)
    return arckv::fail(ARCKV_EINVAL, "cache_restore: bad arguments");
  *out = nullptr;
  Reader r{static_cast<const uint64_t*>(buf), n / 8};
  auto bad = [](const char* what) { return arckv::fail(ARCKV_EINVAL, "cache_restore: %s", what); };
  if (r.get() != kImageMagic || r.get_i() != kImageVersion) return bad("not a cache image of this version");
  arckv_cache_cfg cfg{};
  cfg.policy = static_cast<int32_t>(r.get_i());
  cfg.ref_order = static_cast<int32_t>(r.get_i());
  cfg.victim_window = static_cast<int32_t>(r.get_i());
  const int64_t reuse = r.get_i(), check = r.get_i();
  cfg.no_intra_batch_reuse = reuse ? 0 : 1;
  cfg.check_blocks = check ? 1 : 0;
  cfg.capacity_blocks = r.get_i();
  cfg.num_phys_blocks = r.get_i();
  cfg.scratch_blocks = r.get_i();
  const double p = __builtin_bit_cast(double, r.get());
  cfg.frc_p = cfg.policy == ARCKV_POLICY_FRC ? p : 0.0;
  if (!r.ok || (reuse != 0 && reuse != 1) || (check != 0 && check != 1)) return bad("truncated header");
  arckv_cache* c = nullptr;
  int32_t st = arckv_cache_create(&cfg, &c);
  if (st != ARCKV_OK) return st;
  auto fail = [&](const char* what) { arckv_cache_destroy(c); return bad(what); };
  if (!(p >= 0.0 && p <= static_cast<double>(c->c))) return fail("p outside [0, c]");
  c->p = p;
  c->references = r.get_i();
  c->requests = r.get_i();
  c->prompt_tokens = r.get_i();
  c->prefix_hit_tokens = r.get_i();
  c->computed_tokens = r.get_i();
  for (int64_t& v : c->case_counts) v = r.get_i();
  std::vector<char> used(static_cast<size_t>(c->num_phys), 0);
  auto take = [&](int64_t b) {            // a physical block named once, in range
    if (b < 0 || b >= c->num_phys || used[b]) return false;
    used[b] = 1;
    return true;
  };
  int64_t total = 0;
  for (int list = ARCKV_LIST_T1; list <= ARCKV_LIST_B2; ++list) {
    const int64_t size = r.get_i();
    total += size;
    if (!r.ok || size < 0 || total > 2 * c->c) return fail("list sizes");      // |T1|+|T2|+|B1|+|B2| <= 2c
    const bool resident = list == ARCKV_LIST_T1 || list == ARCKV_LIST_T2;
    for (int64_t i = 0; i < size; ++i) {
      const uint64_t key = r.get();
      const int64_t phys = r.get_i(), depth = r.get_i();
      const uint64_t digest = r.get();
      if (!r.ok || c->find(key) >= 0) return fail("duplicate or truncated list entry");
      if (resident ? !take(phys) : phys != -1) return fail("physical block of a list entry");
      if (depth < 0 || depth > INT32_MAX) return fail("depth of a list entry");
      const int32_t x = c->new_node(key, static_cast<int32_t>(phys));
      c->nodes[x].depth = static_cast<int32_t>(depth);
      c->nodes[x].digest = digest;
      c->push_mru(x, list);
    }
  }
  if (c->lists[ARCKV_LIST_T1].size + c->lists[ARCKV_LIST_T2].size > c->c) return fail("more pages than c");
  c->free_blocks.clear();
  c->scratch_fifo.clear();
  for (std::deque<int32_t>* q : {&c->free_blocks, &c->scratch_fifo}) {
    const int64_t size = r.get_i();
    if (!r.ok || size < 0 || size > c->num_phys) return fail("free list sizes");
    for (int64_t i = 0; i < size; ++i) {
      const int64_t b = r.get_i();
      if (!r.ok || !take(b)) return fail("free list entry");
      q->push_back(static_cast<int32_t>(b));
    }
  }
  if (static_cast<int64_t>(c->scratch_fifo.size()) != c->n_scratch) return fail("scratch FIFO size");
  for (char u : used)
    if (!u) return fail("a physical block is neither in a list nor free");
  if (r.get() != kImageMagic || r.i != r.n) return fail("trailing words or missing end marker");
  *out = c;
  return ARCKV_OK;
}
