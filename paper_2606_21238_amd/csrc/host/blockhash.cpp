// Chained block identities: the key the block cache decides on.
//
// Cached KV is identified and evicted per 16-token block (paper, Sec. 3, last paragraph);
// a block's KV can only be reused when every earlier token is the same (prefix caching,
// Sec. 2), so its identity chains in the parent's identity:
//   h_i = FNV-1a-64(le64(h_{i-1}) || le32(tok[16 i]) .. le32(tok[16 i + 15])),  h_{-1} = root.
// FNV-1a-64: offset basis 0xcbf29ce484222325, prime 0x100000001b3, per byte h ^= b, h *= prime.
//
// Block digests (collision checks) chain the same way through a different function: per token
// d <- M(d + golden + token) with M the splitmix64 finaliser (Steele, Lea and Flood, "Fast
// splittable pseudorandom number generators", 2014); d_{-1} = M(root ^ seed).
#include <atomic>
#include <cstring>

#include "internal.hpp"

namespace {

constexpr uint64_t kFnvOffset = 0xcbf29ce484222325ull;
constexpr uint64_t kFnvPrime = 0x100000001b3ull;

inline uint64_t mix_byte(uint64_t h, uint8_t b) { return (h ^ b) * kFnvPrime; }

// identities are ANDed with this (test-only override; all ones otherwise)
std::atomic<uint64_t> g_identity_mask{~0ull};

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kDigestSeed = 0xD1B54A32D192ED03ull;

inline uint64_t splitmix_final(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

inline uint64_t digest_block(uint64_t parent, const int32_t* tok) {
  uint64_t d = parent;
  for (int t = 0; t < ARCKV_BLOCK_TOKENS; ++t)
    d = splitmix_final(d + kGolden + static_cast<uint32_t>(tok[t]));
  return d;
}

inline uint64_t hash_block(uint64_t parent, const int32_t* tok) {
  uint64_t h = kFnvOffset;
  for (int i = 0; i < 8; ++i) h = mix_byte(h, static_cast<uint8_t>(parent >> (8 * i)));
  for (int t = 0; t < ARCKV_BLOCK_TOKENS; ++t) {
    const uint32_t v = static_cast<uint32_t>(tok[t]);
    for (int i = 0; i < 4; ++i) h = mix_byte(h, static_cast<uint8_t>(v >> (8 * i)));
  }
  return h;
}

}  // namespace

extern "C" int32_t arckv_hash_blocks(const int32_t* tokens, int64_t n_tokens, uint64_t root,
                                     uint64_t* out, int64_t out_cap, int64_t* n_full) {
  if (n_tokens < 0 || n_full == nullptr || (n_tokens > 0 && tokens == nullptr))
    return arckv::fail(ARCKV_EINVAL, "hash_blocks: bad arguments");
  const int64_t nf = n_tokens / ARCKV_BLOCK_TOKENS;
  *n_full = nf;
  if (nf > out_cap || (nf > 0 && out == nullptr))
    return arckv::fail(ARCKV_ENOSPC, "hash_blocks: %lld blocks, capacity %lld",
                       (long long)nf, (long long)out_cap);
  const uint64_t mask = g_identity_mask.load(std::memory_order_relaxed);
  uint64_t h = root;
  for (int64_t i = 0; i < nf; ++i) {
    h = hash_block(h, tokens + i * ARCKV_BLOCK_TOKENS);
    out[i] = h & mask;
  }
  return ARCKV_OK;
}

extern "C" int32_t arckv_digest_blocks(const int32_t* tokens, int64_t n_tokens, uint64_t root,
                                       uint64_t* out, int64_t out_cap, int64_t* n_full) {
  if (n_tokens < 0 || n_full == nullptr || (n_tokens > 0 && tokens == nullptr))
    return arckv::fail(ARCKV_EINVAL, "digest_blocks: bad arguments");
  const int64_t nf = n_tokens / ARCKV_BLOCK_TOKENS;
  *n_full = nf;
  if (nf > out_cap || (nf > 0 && out == nullptr))
    return arckv::fail(ARCKV_ENOSPC, "digest_blocks: %lld blocks, capacity %lld",
                       (long long)nf, (long long)out_cap);
  uint64_t d = splitmix_final(root ^ kDigestSeed);
  for (int64_t i = 0; i < nf; ++i) {
    d = digest_block(d, tokens + i * ARCKV_BLOCK_TOKENS);
    out[i] = d;
  }
  return ARCKV_OK;
}

extern "C" int32_t arckv_test_set_hash_mask(uint64_t mask, uint64_t* previous) {
  const uint64_t old = g_identity_mask.exchange(mask);
  if (previous != nullptr) *previous = old;
  return ARCKV_OK;
}

// Many sequences at once: kLanes independent chains advance in lock-step, so the serial
// xor-multiply latency of one chain overlaps with the others.  A lane whose sequence ends takes
// the next unstarted sequence, so ragged lengths keep every lane busy.  Same definition, same
// result.
extern "C" int32_t arckv_hash_blocks_batch(const int32_t* const* tokens, const int64_t* n_tokens,
                                           int32_t n_seqs, uint64_t root, uint64_t* out,
                                           int64_t out_cap, int64_t* offsets) {
  constexpr int kLanes = 8;
  if (n_seqs < 0 || offsets == nullptr || (n_seqs > 0 && (tokens == nullptr || n_tokens == nullptr)))
    return arckv::fail(ARCKV_EINVAL, "hash_blocks_batch: bad arguments");
  offsets[0] = 0;
  for (int32_t r = 0; r < n_seqs; ++r) {
    if (n_tokens[r] < 0 || (n_tokens[r] > 0 && tokens[r] == nullptr))
      return arckv::fail(ARCKV_EINVAL, "hash_blocks_batch: sequence %d", r);
    offsets[r + 1] = offsets[r] + n_tokens[r] / ARCKV_BLOCK_TOKENS;
  }
  if (offsets[n_seqs] > out_cap || (offsets[n_seqs] > 0 && out == nullptr))
    return arckv::fail(ARCKV_ENOSPC, "hash_blocks_batch: %lld blocks, capacity %lld",
                       (long long)offsets[n_seqs], (long long)out_cap);
  // lane state: its sequence (-1: idle), the next block, the chain value, token and output cursors
  int32_t seq[kLanes];
  int64_t left[kLanes];
  uint64_t h[kLanes];
  const int32_t* tok[kLanes];
  uint64_t* dst[kLanes];
  int32_t next = 0;
  auto refill = [&](int l) {
    seq[l] = -1;
    while (next < n_seqs && n_tokens[next] < ARCKV_BLOCK_TOKENS) ++next;  // no full block
    if (next == n_seqs) return;
    seq[l] = next;
    left[l] = n_tokens[next] / ARCKV_BLOCK_TOKENS;
    h[l] = root;
    tok[l] = tokens[next];
    dst[l] = out + offsets[next];
    ++next;
  };
  int busy = 0;
  for (int l = 0; l < kLanes; ++l) {
    refill(l);
    busy += seq[l] >= 0;
  }
  static const int32_t kZeros[ARCKV_BLOCK_TOKENS] = {};
  const uint64_t mask = g_identity_mask.load(std::memory_order_relaxed);
  while (busy > 0) {
    uint64_t x[kLanes];
    const int32_t* t16[kLanes];
    for (int l = 0; l < kLanes; ++l) {
      x[l] = kFnvOffset;
      t16[l] = seq[l] >= 0 ? tok[l] : kZeros;  // idle lanes hash zeros, never stored
    }
    for (int byte = 0; byte < 8; ++byte)
      for (int l = 0; l < kLanes; ++l) x[l] = mix_byte(x[l], static_cast<uint8_t>(h[l] >> (8 * byte)));
    for (int t = 0; t < ARCKV_BLOCK_TOKENS; ++t) {
      uint32_t v[kLanes];
      for (int l = 0; l < kLanes; ++l) v[l] = static_cast<uint32_t>(t16[l][t]);
      for (int byte = 0; byte < 4; ++byte)
        for (int l = 0; l < kLanes; ++l) x[l] = mix_byte(x[l], static_cast<uint8_t>(v[l] >> (8 * byte)));
    }
    for (int l = 0; l < kLanes; ++l) {
      if (seq[l] < 0) continue;
      h[l] = x[l];
      *dst[l]++ = x[l] & mask;
      tok[l] += ARCKV_BLOCK_TOKENS;
      if (--left[l] == 0) {
        refill(l);
        busy -= seq[l] < 0;
      }
    }
  }
  return ARCKV_OK;
}
