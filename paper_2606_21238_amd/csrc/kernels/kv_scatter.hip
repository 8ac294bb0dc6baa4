// KV scatter: write the K/V rows of the computed (uncached) tokens into their pool slots.
//
// The serving engine processes a miss by regenerating the block's KV (paper, Sec. 3); the
// tokens of a batch that prefill computes are written into the physical blocks the planner
// chose.  Pool layout version 1: K [blocks][kv_heads][16][D] (token-major), V
// [blocks][kv_heads][D][16] (dim-major, so that the attention kernel's P.V contraction reads
// 8 consecutive tokens of one dimension as one 16-byte operand).
//
// One work-group handles 64 tokens of one KV head.  K rows are copied as 16-byte chunks
// (consecutive lanes, consecutive chunks of one row).  V rows are staged through LDS and
// written transposed: the 64 lanes of a wave take 64 consecutive tokens of one dimension, so
// tokens of one block land on consecutive 2-byte addresses.  Bytes are copied, never
// converted: the result is bit-exact.  Slots outside the pool are skipped.
#include <hip/hip_runtime.h>

#include "../host/internal.hpp"

namespace {

constexpr int kTok = 64;
constexpr int kThreads = 256;

template <int D>
__global__ __launch_bounds__(kThreads) void kv_scatter_kernel(
    uint16_t* __restrict__ k_pool, uint16_t* __restrict__ v_pool,
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    const int32_t* __restrict__ slots, int64_t n_tokens, int64_t n_slots, int hkv) {
  constexpr int CH = D / 8;            // 16-byte chunks per row
  constexpr int VROW = D + 2;          // padded LDS row (in u16) so column reads spread over banks
  __shared__ uint32_t sv32[kTok * VROW / 2];
  __shared__ int32_t sslot[kTok];
  uint16_t* sv = reinterpret_cast<uint16_t*>(sv32);

  const int h = blockIdx.y;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kTok;
  const int tid = threadIdx.x;
  if (tid < kTok) {
    const int64_t t = t0 + tid;
    int32_t s = t < n_tokens ? slots[t] : -1;
    sslot[tid] = (s >= 0 && s < n_slots) ? s : -1;
  }
  __syncthreads();

  // K: direct 16-byte copies; V: into LDS (row = token, padded)
  for (int c = tid; c < kTok * CH; c += kThreads) {
    const int tl = c / CH, ch = c % CH;
    const int64_t t = t0 + tl;
    if (t >= n_tokens) continue;
    const int64_t src = (t * hkv + h) * D + ch * 8;
    const int32_t s = sslot[tl];
    if (s >= 0) {
      const uint4 kv = *reinterpret_cast<const uint4*>(k_new + src);
      const int64_t blk = s >> 4;
      *reinterpret_cast<uint4*>(k_pool + ((blk * hkv + h) * 16 + (s & 15)) * D + ch * 8) = kv;
    }
    const uint4 vv = *reinterpret_cast<const uint4*>(v_new + src);
    uint32_t* dst = sv32 + (tl * VROW + ch * 8) / 2;  // VROW and ch*8 are even: 4-byte aligned
    dst[0] = vv.x; dst[1] = vv.y; dst[2] = vv.z; dst[3] = vv.w;
  }
  __syncthreads();

  // V: lane = token, loop over dimensions
  const int tl = tid & (kTok - 1);
  const int s = sslot[tl];
  if (s < 0 || t0 + tl >= n_tokens) return;
  const int64_t base = ((static_cast<int64_t>(s >> 4) * hkv + h) * D) * 16 + (s & 15);
  for (int d = tid >> 6; d < D; d += kThreads / kTok)
    v_pool[base + static_cast<int64_t>(d) * 16] = sv[tl * VROW + d];
}

}  // namespace

extern "C" int32_t arckv_kv_scatter(void* k_pool, void* v_pool, const void* k_new,
                                    const void* v_new, const int32_t* slot_mapping,
                                    int64_t n_tokens, int64_t num_blocks, int32_t num_kv_heads,
                                    int32_t head_dim, void* stream) {
  if (n_tokens < 0 || num_blocks < 0 || num_kv_heads < 1)
    return arckv::fail(ARCKV_EINVAL, "kv_scatter: bad sizes");
  if (head_dim != 64 && head_dim != 128)
    return arckv::fail(ARCKV_EUNSUPPORTED, "kv_scatter: head_dim %d not in {64,128}", head_dim);
  if (n_tokens == 0) return ARCKV_OK;
  if (k_pool == nullptr || v_pool == nullptr || k_new == nullptr || v_new == nullptr ||
      slot_mapping == nullptr)
    return arckv::fail(ARCKV_EINVAL, "kv_scatter: NULL pointer");
  const dim3 grid(static_cast<unsigned>((n_tokens + kTok - 1) / kTok), num_kv_heads);
  auto* st = static_cast<hipStream_t>(stream);
  auto* kp = static_cast<uint16_t*>(k_pool);
  auto* vp = static_cast<uint16_t*>(v_pool);
  auto* kn = static_cast<const uint16_t*>(k_new);
  auto* vn = static_cast<const uint16_t*>(v_new);
  const int64_t n_slots = num_blocks * 16;
  if (head_dim == 64)
    hipLaunchKernelGGL(kv_scatter_kernel<64>, grid, dim3(kThreads), 0, st, kp, vp, kn, vn,
                       slot_mapping, n_tokens, n_slots, num_kv_heads);
  else
    hipLaunchKernelGGL(kv_scatter_kernel<128>, grid, dim3(kThreads), 0, st, kp, vp, kn, vn,
                       slot_mapping, n_tokens, n_slots, num_kv_heads);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return arckv::fail(ARCKV_EDEVICE, "kv_scatter: %s", hipGetErrorString(e));
  return ARCKV_OK;
}
