// Chained block identities: the key the block cache decides on.
//
// Cached KV is identified and evicted per 16-token block (paper, Sec. 3, last paragraph);
// a block's KV can only be reused when every earlier token is the same (prefix caching,
// Sec. 2), so its identity chains in the parent's identity:
//   h_i = FNV-1a-64(le64(h_{i-1}) || le32(tok[16 i]) .. le32(tok[16 i + 15])),  h_{-1} = root.
// FNV-1a-64: offset basis 0xcbf29ce484222325, prime 0x100000001b3, per byte h ^= b, h *= prime.
#include <cstring>

#include "internal.hpp"

namespace {

constexpr uint64_t kFnvOffset = 0xcbf29ce484222325ull;
constexpr uint64_t kFnvPrime = 0x100000001b3ull;

inline uint64_t mix_byte(uint64_t h, uint8_t b) { return (h ^ b) * kFnvPrime; }

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
  uint64_t h = root;
  for (int64_t i = 0; i < nf; ++i) {
    h = hash_block(h, tokens + i * ARCKV_BLOCK_TOKENS);
    out[i] = h;
  }
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
      *dst[l]++ = x[l];
      tok[l] += ARCKV_BLOCK_TOKENS;
      if (--left[l] == 0) {
        refill(l);
        busy -= seq[l] < 0;
      }
    }
  }
  return ARCKV_OK;
}
