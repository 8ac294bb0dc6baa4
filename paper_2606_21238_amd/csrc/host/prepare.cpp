// One batch's host preparation in one call: chained block hashes of every prompt (or the
// caller's own, for requests whose hashes it keeps), the cache plan (hits, evictions,
// placement) and the attention work plan, written straight into one int32 buffer laid out the
// way the device steps read it, so that the caller's only remaining work is a single
// host-to-device copy.  Each stage is the library's own entry point (arckv_hash_blocks_batch,
// arckv_plan_batch, arckv_attention_plan); the results are identical to calling them one by one.
#include <algorithm>
#include <vector>

#include "internal.hpp"

namespace {

// Upper bound on work items + combine items of arckv_attention_plan for prompts of these
// lengths: a tile is at most 256 columns of one (request, KV head), or one per (request, KV
// head) when the batch uses narrower tiles (every request then fits one); key-range splits
// add at most num_cus pieces, or, where the cap on one item's keys (kMaxItemKeys) cuts finer,
// at most ceil(L / kMaxItemKeys) pieces per tile of a request of L tokens; the XCD-phase
// padding of the ordered list at most multiplies the pieces by the XCD count; there is at most
// one combine item per tile.
int64_t work_bound(const int64_t* n_tokens, int32_t n_reqs, int32_t G, int32_t hkv, int32_t num_cus) {
  int64_t tiles = 0, capped = 0;
  for (int32_t r = 0; r < n_reqs; ++r) {
    const int64_t t = hkv * std::max<int64_t>(1, (n_tokens[r] * G + arckv::kWideCols - 1) / arckv::kWideCols);
    tiles += t;
    capped += t * ((n_tokens[r] + arckv::kMaxItemKeys - 1) / arckv::kMaxItemKeys);
  }
  constexpr int64_t kXcds = 8;
  return kXcds * (tiles + num_cus + capped) + tiles;
}

// The common part: requests given as (hashes, n_tokens); `hashes[r]` holds n_tokens[r] / 16
// chained identities, `digests` (NULL: none) as many block digests per request.
int32_t prepare_planned(arckv_cache* cache, const uint64_t* const* hashes, const uint64_t* const* digests,
                        const int64_t* n_tokens,
                        int32_t n_reqs, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                        int32_t num_cus, int32_t* packed, int64_t packed_cap, int32_t* prefix_lens,
                        int32_t* hit_blocks, arckv_batch* out) {
  const int32_t G = num_q_heads / num_kv_heads;
  int64_t stride = 1, total_tokens = 0;
  for (int32_t r = 0; r < n_reqs; ++r) {
    stride = std::max<int64_t>(stride, (n_tokens[r] + ARCKV_BLOCK_TOKENS - 1) / ARCKV_BLOCK_TOKENS);
    total_tokens += n_tokens[r];
  }
  // layout: block tables | cu_q | seq_lens | slots (at most every token) | work items
  const int64_t fixed = static_cast<int64_t>(n_reqs) * stride + 2 * static_cast<int64_t>(n_reqs) + 1;
  const int64_t bound =
      fixed + total_tokens + ARCKV_WORK_INTS * work_bound(n_tokens, n_reqs, G, num_kv_heads, num_cus);
  out->n_packed = bound;
  if (packed == nullptr || packed_cap < bound)
    return arckv::fail(ARCKV_ENOSPC, "prepare_batch: packed buffer %lld ints, need up to %lld",
                       (long long)packed_cap, (long long)bound);
  thread_local std::vector<arckv_req> reqs;
  reqs.resize(static_cast<size_t>(n_reqs));
  for (int32_t r = 0; r < n_reqs; ++r)
    reqs[r] = arckv_req{hashes[r], n_tokens[r] / ARCKV_BLOCK_TOKENS, n_tokens[r],
                        digests != nullptr ? digests[r] : nullptr};

  out->n_reqs = n_reqs;
  out->bt_stride = static_cast<int32_t>(stride);
  out->off_block_tables = 0;
  out->off_cu_q = static_cast<int64_t>(n_reqs) * stride;
  out->off_seq_lens = out->off_cu_q + n_reqs + 1;
  out->off_slots = out->off_seq_lens + n_reqs;
  arckv_plan plan{};
  plan.block_tables = packed + out->off_block_tables;
  plan.bt_stride = out->bt_stride;
  plan.cu_q = packed + out->off_cu_q;
  plan.seq_lens = packed + out->off_seq_lens;
  plan.prefix_lens = prefix_lens;
  plan.hit_blocks = hit_blocks;
  plan.slot_mapping = packed + out->off_slots;
  plan.slot_cap = total_tokens;
  int32_t st = arckv_plan_batch(cache, reqs.data(), n_reqs, &plan);
  if (st != ARCKV_OK) return st;  // the cache is unchanged on every failure of the plan
  out->n_slots = plan.n_slots;
  out->max_q_len = plan.max_q_len;
  out->max_seq_len = plan.max_seq_len;

  out->off_work = out->off_slots + plan.n_slots;
  int64_t n_work = 0, n_combine = 0, ws = 0;
  int32_t tile_cols = 0;
  st = arckv_attention_plan(plan.cu_q, plan.seq_lens, n_reqs, num_q_heads, num_kv_heads, head_dim,
                            num_cus, packed + out->off_work, (packed_cap - out->off_work) / ARCKV_WORK_INTS,
                            &n_work, &n_combine, &ws, &tile_cols);
  if (st != ARCKV_OK) {
    // within the bound this cannot happen; leave no half-prepared batch behind
    const std::string msg = arckv_last_error();
    arckv_release_batch(cache);
    return arckv::fail(st, "prepare_batch: %s (batch released)", msg.c_str());
  }
  out->n_work = n_work;
  out->n_combine = n_combine;
  out->ws_bytes = ws;
  out->tile_cols = tile_cols;
  out->n_packed = out->off_work + (n_work + n_combine) * ARCKV_WORK_INTS;
  return ARCKV_OK;
}

int32_t check_args(arckv_cache* cache, const void* seqs, const int64_t* n_tokens, int32_t n_reqs,
                   int32_t num_q_heads, int32_t num_kv_heads, int32_t num_cus, const int32_t* prefix_lens,
                   const int32_t* hit_blocks, arckv_batch* out) {
  if (cache == nullptr || out == nullptr || n_reqs < 1 || seqs == nullptr || n_tokens == nullptr ||
      prefix_lens == nullptr || hit_blocks == nullptr || num_cus < 1 || num_kv_heads < 1 ||
      num_q_heads < 1 || num_q_heads % num_kv_heads != 0)
    return arckv::fail(ARCKV_EINVAL, "prepare_batch: bad arguments");
  for (int32_t r = 0; r < n_reqs; ++r)
    if (n_tokens[r] < 1 || n_tokens[r] > INT32_MAX / 2)
      return arckv::fail(ARCKV_EINVAL, "prepare_batch: request %d has %lld tokens", r, (long long)n_tokens[r]);
  *out = arckv_batch{};
  return ARCKV_OK;
}

}  // namespace

extern "C" int32_t arckv_prepare_batch(arckv_cache* cache, const int32_t* const* tokens,
                                       const int64_t* n_tokens, int32_t n_reqs, uint64_t root,
                                       int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                       int32_t num_cus, int32_t* packed, int64_t packed_cap,
                                       int32_t* prefix_lens, int32_t* hit_blocks,
                                       arckv_batch* out) {
  int32_t st = check_args(cache, tokens, n_tokens, n_reqs, num_q_heads, num_kv_heads, num_cus,
                          prefix_lens, hit_blocks, out);
  if (st != ARCKV_OK) return st;
  int64_t total_blocks = 0;
  for (int32_t r = 0; r < n_reqs; ++r) {
    if (tokens[r] == nullptr) return arckv::fail(ARCKV_EINVAL, "prepare_batch: request %d", r);
    total_blocks += n_tokens[r] / ARCKV_BLOCK_TOKENS;
  }
  thread_local std::vector<uint64_t> hashes;
  thread_local std::vector<int64_t> offsets;
  thread_local std::vector<const uint64_t*> rows;
  hashes.resize(static_cast<size_t>(std::max<int64_t>(total_blocks, 1)));
  offsets.resize(static_cast<size_t>(n_reqs) + 1);
  st = arckv_hash_blocks_batch(tokens, n_tokens, n_reqs, root, hashes.data(),
                               static_cast<int64_t>(hashes.size()), offsets.data());
  if (st != ARCKV_OK) return st;
  rows.resize(static_cast<size_t>(n_reqs));
  for (int32_t r = 0; r < n_reqs; ++r) rows[r] = hashes.data() + offsets[r];
  thread_local std::vector<uint64_t> digests;
  thread_local std::vector<const uint64_t*> drows;
  if (arckv::cache_checks_blocks(cache)) {   // check mode: the blocks' digests as well
    digests.resize(hashes.size());
    drows.resize(static_cast<size_t>(n_reqs));
    for (int32_t r = 0; r < n_reqs; ++r) {
      int64_t nf = 0;
      st = arckv_digest_blocks(tokens[r], n_tokens[r], root, digests.data() + offsets[r],
                               offsets[r + 1] - offsets[r], &nf);
      if (st != ARCKV_OK) return st;
      drows[r] = digests.data() + offsets[r];
    }
  }
  return prepare_planned(cache, rows.data(), arckv::cache_checks_blocks(cache) ? drows.data() : nullptr,
                         n_tokens, n_reqs, num_q_heads, num_kv_heads, head_dim, num_cus, packed,
                         packed_cap, prefix_lens, hit_blocks, out);
}

extern "C" int32_t arckv_prepare_batch_hashed(arckv_cache* cache, const uint64_t* const* hashes,
                                              const int64_t* n_tokens, int32_t n_reqs,
                                              int32_t num_q_heads, int32_t num_kv_heads,
                                              int32_t head_dim, int32_t num_cus, int32_t* packed,
                                              int64_t packed_cap, int32_t* prefix_lens,
                                              int32_t* hit_blocks, arckv_batch* out) {
  int32_t st = check_args(cache, hashes, n_tokens, n_reqs, num_q_heads, num_kv_heads, num_cus,
                          prefix_lens, hit_blocks, out);
  if (st != ARCKV_OK) return st;
  for (int32_t r = 0; r < n_reqs; ++r)
    if (n_tokens[r] >= ARCKV_BLOCK_TOKENS && hashes[r] == nullptr)
      return arckv::fail(ARCKV_EINVAL, "prepare_batch_hashed: request %d has no hashes", r);
  return prepare_planned(cache, hashes, nullptr, n_tokens, n_reqs, num_q_heads, num_kv_heads, head_dim,
                         num_cus, packed, packed_cap, prefix_lens, hit_blocks, out);
}
