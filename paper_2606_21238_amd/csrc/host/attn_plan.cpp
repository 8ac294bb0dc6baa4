// Work decomposition of prefix-cached prefill attention (host side).
//
// A work item covers one query tile of `cols` "columns" of one (request, KV head): column
// c = token * G + g (G query heads share a KV head, token-major), so the K/V tiles a work
// item streams serve all G heads of its group at once.  The key range of a tile ends at the
// last visible key of its last column (causal: suffix token i of a request with P cached
// tokens sees keys 0..P+i).  Tiles are 256 columns wide, 128 when no request of the batch has
// more than 128 columns (short suffixes, decode-like batches), so that work-groups compute on
// fewer empty columns.  When a batch has fewer tiles than compute units (short suffixes over long cached
// prefixes), tiles are split along the key range so that the whole batch runs as one round of
// at most one item per compute unit: the smallest cap on key tiles per item (at least 8, i.e.
// 512 keys) for which the pieces fit, each tile cut into equal pieces under the cap.  Split
// items write fp32 partials plus a base-2 log-sum-exp, merged afterwards by one combine item
// per tile.
//
// With at least as many tiles as compute units, a tile longer than one compute unit's share
// of all key tiles (e.g. one long history in a decode batch) is cut to that share, so that it
// does not set the length of the launch.
//
// Narrow batches run persistent work-groups instead: the plan is a set of lists, one per
// work-group (kListItems entries each: its items in order, then idle padding), at most one list
// per compute unit when the items fit.  The tiles are packed into the lists in order, cut where
// a list's budget runs out, so that every list carries about the same cost (key tiles, plus
// kItemCost per item for the item's Q tile, its first tile's latency and its epilogue); a cut
// never leaves a piece shorter than kMinPiece key tiles.  The budget is the smallest that
// needs no more lists than compute units.  The kernel streams a list's items back to back.
//
// No item covers more than kMaxItemKeys keys (65536): a longer range is cut the same way, so the
// attention kernel can hold an item's block-table entries in LDS.
//
// Items are ordered longest key range first so the longest ones start first, and the order
// is interleaved over the 8 XCDs (work-groups are dispatched round-robin over XCDs, each with
// its own L2): all tiles of one (request, KV head) group land on the same XCD, so the K/V
// they all stream is fetched into that XCD's L2 once.
#include <algorithm>
#include <cmath>
#include <vector>

#include "internal.hpp"

namespace {

constexpr int kKeyTile = 64;  // keys per K/V tile (split boundaries are multiples of this)
constexpr int kXcds = 8;      // MI355X: 8 XCDs; dispatch round-robins work-groups over them
constexpr int64_t kItemCost = 4;  // list plans: cost of one item beyond its key tiles (measured)
constexpr int64_t kMinPiece = 4;  // list plans: shortest piece a cut may leave, in key tiles
constexpr int64_t kXcdSkewPermille = 25;  // work shifted from odd to even XCDs, per mille (measured)

struct Item {
  int32_t v[ARCKV_WORK_INTS];
  int64_t cost;
  int64_t group;
};

}  // namespace

extern "C" int32_t arckv_attention_plan(const int32_t* cu_q, const int32_t* seq_lens,
                                        int32_t n_reqs, int32_t num_q_heads, int32_t num_kv_heads,
                                        int32_t head_dim, int32_t num_cus, int32_t* work,
                                        int64_t work_cap, int64_t* n_work, int64_t* n_combine,
                                        int64_t* ws_bytes, int32_t* tile_cols) {
  if (n_work == nullptr || n_combine == nullptr || ws_bytes == nullptr || tile_cols == nullptr ||
      n_reqs < 0 ||
      (n_reqs > 0 && (cu_q == nullptr || seq_lens == nullptr)) || num_cus < 1 ||
      num_kv_heads < 1 || num_q_heads < 1)
    return arckv::fail(ARCKV_EINVAL, "attention_plan: bad arguments");
  if (num_q_heads % num_kv_heads != 0)
    return arckv::fail(ARCKV_EINVAL, "attention_plan: num_q_heads %% num_kv_heads != 0");
  const int G = num_q_heads / num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 5 && G != 8)
    return arckv::fail(ARCKV_EUNSUPPORTED, "attention_plan: group size %d not in {1,2,4,5,8}", G);
  if (head_dim != 64 && head_dim != 128)
    return arckv::fail(ARCKV_EUNSUPPORTED, "attention_plan: head_dim %d not in {64,128}", head_dim);
  if (n_reqs > 0 && cu_q[0] != 0) return arckv::fail(ARCKV_EINVAL, "attention_plan: cu_q[0] != 0");

  int64_t max_cols = 0;
  for (int32_t r = 0; r < n_reqs; ++r)
    max_cols = std::max<int64_t>(max_cols, (static_cast<int64_t>(cu_q[r + 1]) - cu_q[r]) * G);
  const int kCols = max_cols <= arckv::kNarrowCols ? arckv::kNarrowCols : arckv::kWideCols;
  *tile_cols = kCols;

  struct Tile { int32_t req, kvh, col_start, kv_end; };
  std::vector<Tile> tiles;
  for (int32_t r = 0; r < n_reqs; ++r) {
    const int64_t S = static_cast<int64_t>(cu_q[r + 1]) - cu_q[r];
    const int64_t L = seq_lens[r];
    if (S < 0 || L < S) return arckv::fail(ARCKV_EINVAL, "attention_plan: request %d has S=%lld L=%lld", r, (long long)S, (long long)L);
    const int64_t P = L - S;
    const int64_t ncols = S * G;
    for (int64_t cs = 0; cs < ncols; cs += kCols) {
      const int64_t last = std::min<int64_t>(cs + kCols, ncols) - 1;
      const int32_t kv_end = static_cast<int32_t>(P + last / G + 1);
      for (int32_t h = 0; h < num_kv_heads; ++h) {
        tiles.push_back({r, h, static_cast<int32_t>(cs), kv_end});
      }
    }
  }
  const int64_t base = static_cast<int64_t>(tiles.size());
  const int64_t target = static_cast<int64_t>(num_cus);  // one work-group per CU at a time
  auto key_tiles = [](const Tile& t) { return (static_cast<int64_t>(t.kv_end) + kKeyTile - 1) / kKeyTile; };

  if (kCols == arckv::kNarrowCols) {
    // ---- list plan ----------------------------------------------------------------------
    constexpr int64_t kMaxPiece = arckv::kMaxItemKeys / kKeyTile;
    struct Piece { int32_t tile; int64_t a, n; int32_t list; };  // key tiles [a, a + n)
    int64_t cost = 0, min_pieces = 0;
    for (const Tile& t : tiles) {
      const int64_t kt = key_tiles(t);
      const int64_t np = std::max<int64_t>(1, (kt + kMaxPiece - 1) / kMaxPiece);
      min_pieces += np;
      cost += kt + kItemCost * np;
    }
    const int64_t n_lists_max = std::max<int64_t>(target, (min_pieces + arckv::kListItems - 1) / arckv::kListItems);
    std::vector<Piece> pieces;
    // Packs the tiles in order into lists of budget B; returns the number of lists.  List k
    // runs on XCD k % 8; the work-groups of odd XCDs measured about 5 % slower per key tile
    // than those of even ones on the boxes timed, so even lists get a budget of
    // B (1 + kXcdSkewPermille / 1000) and odd ones B (1 - kXcdSkewPermille / 1000).
    auto pack = [&](int64_t B, bool keep) -> int64_t {
      if (keep) pieces.clear();
      const int64_t skew = B * kXcdSkewPermille / 1000;
      int64_t lists = 0, used = B, n_in = arckv::kListItems, Bk = B;
      for (int32_t ti = 0; ti < static_cast<int32_t>(tiles.size()); ++ti) {
        int64_t rem = key_tiles(tiles[ti]), a = 0;
        while (rem > 0) {
          if (n_in == arckv::kListItems || Bk - used - kItemCost < 1) {
            ++lists; used = 0; n_in = 0;
            Bk = (lists - 1) % 2 == 0 ? B + skew : B - skew;
          }
          const int64_t avail = std::min(Bk - used - kItemCost, kMaxPiece);
          int64_t take = rem;
          if (rem > avail) {
            take = avail;
            if (rem - take < kMinPiece) take = rem - kMinPiece;  // leave the next list a piece
            if (take < kMinPiece) {
              if (used > 0) { n_in = arckv::kListItems; continue; }  // start a fresh list
              take = std::min(rem, kMaxPiece);                      // an empty list takes it
            }
          }
          if (keep) pieces.push_back({ti, a, take, static_cast<int32_t>(lists - 1)});
          used += take + kItemCost;
          ++n_in;
          a += take;
          rem -= take;
        }
      }
      return lists;
    };
    int64_t n_lists = 0;
    if (base > 0) {
      int64_t lo = std::max<int64_t>(kItemCost + kMinPiece, (cost + n_lists_max - 1) / n_lists_max);
      // a list closes with less than 2 kMinPiece + kItemCost unused, so a budget that much above
      // the even share usually fits; the whole range is searched only when it does not
      int64_t hi = lo + 2 * kMinPiece + kItemCost;
      if (pack(hi, false) > n_lists_max) hi = std::max<int64_t>(hi, cost + kItemCost);
      while (lo < hi) {  // smallest budget that needs at most n_lists_max lists
        const int64_t mid = lo + (hi - lo) / 2;
        if (pack(mid, false) <= n_lists_max) hi = mid; else lo = mid + 1;
      }
      n_lists = pack(lo, true);
    }
    // items: pieces in list order; a tile cut into several pieces takes consecutive slots
    std::vector<int32_t> n_pieces(tiles.size(), 0), first_slot(tiles.size(), -1);
    for (const Piece& pc : pieces) ++n_pieces[pc.tile];
    int64_t slot = 0;
    std::vector<Item> combines;
    for (size_t ti = 0; ti < tiles.size(); ++ti)
      if (n_pieces[ti] > 1) {
        const Tile& t = tiles[ti];
        first_slot[ti] = static_cast<int32_t>(slot);
        combines.push_back({{t.req, t.kvh, t.col_start, static_cast<int32_t>(slot), n_pieces[ti], 0, 0, 0}, 0, 0});
        slot += n_pieces[ti];
      }
    std::vector<int32_t> next_piece(tiles.size(), 0);
    const Item idle{{-1, 0, 0, 0, 0, -1, 0, 0}, 0, -1};
    std::vector<Item> lists(static_cast<size_t>(n_lists * arckv::kListItems), idle);
    std::vector<int32_t> fill(static_cast<size_t>(n_lists), 0);
    for (const Piece& pc : pieces) {
      const Tile& t = tiles[pc.tile];
      const int32_t a = static_cast<int32_t>(pc.a * kKeyTile);
      const int32_t b = static_cast<int32_t>(std::min<int64_t>((pc.a + pc.n) * kKeyTile, t.kv_end));
      const int32_t sl = n_pieces[pc.tile] > 1 ? first_slot[pc.tile] + next_piece[pc.tile]++ : -1;
      lists[static_cast<size_t>(pc.list) * arckv::kListItems + fill[pc.list]++] =
          {{t.req, t.kvh, t.col_start, a, b, sl, 0, 0}, b - a, 0};
    }
    *n_work = static_cast<int64_t>(lists.size());
    *n_combine = static_cast<int64_t>(combines.size());
    *ws_bytes = slot * kCols * (static_cast<int64_t>(head_dim) + 1) * 4;
    if (work == nullptr) return ARCKV_OK;
    if (*n_work + *n_combine > work_cap)
      return arckv::fail(ARCKV_ENOSPC, "attention_plan: %lld items, capacity %lld",
                         (long long)(*n_work + *n_combine), (long long)work_cap);
    int32_t* w = work;
    for (const Item& it : lists) { std::copy(it.v, it.v + ARCKV_WORK_INTS, w); w += ARCKV_WORK_INTS; }
    for (const Item& it : combines) { std::copy(it.v, it.v + ARCKV_WORK_INTS, w); w += ARCKV_WORK_INTS; }
    return ARCKV_OK;
  }

  int64_t cap = INT32_MAX;  // key tiles per item
  if (base > 0) {
    int64_t total_t = 0, max_t = 0;
    for (const Tile& t : tiles) {
      total_t += key_tiles(t);
      max_t = std::max(max_t, key_tiles(t));
    }
    const int64_t share = std::max<int64_t>(8, (total_t + target - 1) / target);
    if (base < target) {
      int64_t lo = share, hi = std::max(lo, max_t);
      while (lo < hi) {  // smallest cap whose pieces fit in one round
        const int64_t mid = (lo + hi) / 2;
        int64_t cnt = 0;
        for (const Tile& t : tiles) cnt += (key_tiles(t) + mid - 1) / mid;
        if (cnt <= target) hi = mid; else lo = mid + 1;
      }
      cap = lo;
    } else {
      cap = share;  // several rounds: no item longer than one compute unit's share
    }
    cap = std::min<int64_t>(cap, arckv::kMaxItemKeys / kKeyTile);
  }

  std::vector<Item> items, combines;
  int64_t slot = 0;
  for (const Tile& t : tiles) {
    const int64_t nt = key_tiles(t);
    const int64_t ns = (nt + cap - 1) / cap;
    const int64_t group = static_cast<int64_t>(t.req) * num_kv_heads + t.kvh;
    if (ns <= 1) {
      items.push_back({{t.req, t.kvh, t.col_start, 0, t.kv_end, -1, 0, 0}, t.kv_end, group});
      continue;
    }
    for (int64_t s = 0; s < ns; ++s) {  // equal pieces of whole key tiles
      const int32_t a = static_cast<int32_t>(s * nt / ns * kKeyTile);
      const int32_t b = static_cast<int32_t>(std::min<int64_t>((s + 1) * nt / ns * kKeyTile, t.kv_end));
      items.push_back({{t.req, t.kvh, t.col_start, a, b, static_cast<int32_t>(slot + s), 0, 0}, b - a, group});
    }
    combines.push_back({{t.req, t.kvh, t.col_start, static_cast<int32_t>(slot), static_cast<int32_t>(ns), 0, 0, 0}, 0, group});
    slot += ns;
  }

  // XCD-aware order: assign whole groups to XCDs (largest first, to the XCD that would finish
  // first: odd XCDs, measured about 5 % slower per key tile, count their work 2.5 % heavier and
  // even ones 2.5 % lighter), then emit position-major so work-group i runs on XCD i % 8; each
  // XCD's list is longest first.
  const int64_t n_groups = static_cast<int64_t>(n_reqs) * num_kv_heads;  // group = req * hkv + kvh
  std::vector<int64_t> cost_of(static_cast<size_t>(n_groups), 0);
  std::vector<char> used(static_cast<size_t>(n_groups), 0);
  for (const Item& it : items) {
    cost_of[it.group] += it.cost;
    used[it.group] = 1;
  }
  std::vector<std::pair<int64_t, int64_t>> groups;  // (group, cost)
  for (int64_t g = 0; g < n_groups; ++g)
    if (used[g]) groups.push_back({g, cost_of[g]});
  std::sort(groups.begin(), groups.end(), [](const auto& a, const auto& b) {
    return a.second != b.second ? a.second > b.second : a.first < b.first;
  });
  std::vector<int32_t> xcd_of(static_cast<size_t>(n_groups), 0);
  int64_t load[kXcds] = {0};
  auto finish = [&](int x, int64_t c) {   // relative finishing time with c more work
    return (load[x] + c) * (x % 2 == 0 ? 1000 - kXcdSkewPermille : 1000 + kXcdSkewPermille);
  };
  for (const auto& g : groups) {
    int best = 0;
    for (int x = 1; x < kXcds; ++x) if (finish(x, g.second) < finish(best, g.second)) best = x;
    xcd_of[g.first] = best;
    load[best] += g.second;
  }
  std::vector<std::vector<Item>> per_xcd(kXcds);
  if (groups.size() >= static_cast<size_t>(kXcds)) {
    for (const Item& it : items) per_xcd[xcd_of[it.group]].push_back(it);
  } else {  // fewer groups than XCDs: spread tiles over all XCDs instead
    for (size_t i = 0; i < items.size(); ++i) per_xcd[i % kXcds].push_back(items[i]);
  }
  // Within an XCD: longest first (the tail of the launch is what load balance costs), but
  // items whose key ranges are within ~10 % of each other count as equally long and are kept
  // together by group, so that the work-groups running at the same time on the XCD are few
  // groups' query tiles streaming the same keys and values, which the XCD's L2 serves once.
  // The sort keys (length bucket, group rank, length) are computed once per item.
  std::vector<int64_t> rank_of(static_cast<size_t>(n_groups), 0);
  for (size_t g = 0; g < groups.size(); ++g) rank_of[groups[g].first] = static_cast<int64_t>(g);
  auto bucket = [](int64_t cost) {  // log_{1.1} of the key-range length
    return cost > 0 ? static_cast<int64_t>(std::log(static_cast<double>(cost)) / std::log(1.1)) : -1;
  };
  struct Key {
    int64_t bucket, rank, cost;
    int32_t idx;
  };
  std::vector<Key> keys;
  std::vector<Item> sorted;
  for (auto& v : per_xcd) {
    keys.clear();
    for (size_t i = 0; i < v.size(); ++i)
      keys.push_back({bucket(v[i].cost), rank_of[v[i].group], v[i].cost, static_cast<int32_t>(i)});
    std::stable_sort(keys.begin(), keys.end(), [](const Key& a, const Key& b) {
      if (a.bucket != b.bucket) return a.bucket > b.bucket;
      return a.rank != b.rank ? a.rank < b.rank : a.cost > b.cost;
    });
    sorted.clear();
    for (const Key& k : keys) sorted.push_back(v[k.idx]);
    v.swap(sorted);
  }
  size_t longest = 0;
  for (auto& v : per_xcd) longest = std::max(longest, v.size());
  std::vector<Item> ordered;
  ordered.reserve(longest * kXcds);
  for (size_t i = 0; i < longest; ++i)
    for (int x = 0; x < kXcds; ++x) {
      if (i < per_xcd[x].size()) ordered.push_back(per_xcd[x][i]);
      else ordered.push_back({{-1, 0, 0, 0, 0, -1, 0, 0}, 0, -1});  // idle slot keeps the XCD phase
    }
  // trailing idle slots carry no work; drop them
  while (!ordered.empty() && ordered.back().v[0] < 0) ordered.pop_back();

  *n_work = static_cast<int64_t>(ordered.size());
  *n_combine = static_cast<int64_t>(combines.size());
  *ws_bytes = slot * kCols * (static_cast<int64_t>(head_dim) + 1) * 4;
  if (work == nullptr) return ARCKV_OK;
  if (*n_work + *n_combine > work_cap)
    return arckv::fail(ARCKV_ENOSPC, "attention_plan: %lld items, capacity %lld",
                       (long long)(*n_work + *n_combine), (long long)work_cap);
  int32_t* w = work;
  for (const Item& it : ordered) { std::copy(it.v, it.v + ARCKV_WORK_INTS, w); w += ARCKV_WORK_INTS; }
  for (const Item& it : combines) { std::copy(it.v, it.v + ARCKV_WORK_INTS, w); w += ARCKV_WORK_INTS; }
  return ARCKV_OK;
}
