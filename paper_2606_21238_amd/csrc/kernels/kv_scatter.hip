// KV scatter: write the K/V rows of the computed (uncached) tokens into their pool slots.
//
// A cache miss costs a recomputation: prefill produces the block's K/V again (paper, Sec. 3),
// and the rows of the tokens it computed go into the physical blocks the planner chose.
// Pool layout version 1: K [blocks][kv_heads][16][D] (token-major), V [blocks][kv_heads][D][16]
// (dim-major, so that the attention kernel's P.V contraction reads 8 consecutive tokens of one
// dimension as one 16-byte operand).
//
// A work-group handles 64 tokens of one KV head and DPW of its head dimensions: 16 for small
// batches, so that a decode step still spreads over many work-groups; the whole head
// otherwise.  K rows are copied as 16-byte chunks.  V rows are staged through LDS and written
// dim-major.  A run is 8 tokens of the work-group whose slots are 8 consecutive slots of one
// block starting at a multiple of 8 (most of a prefill, wherever its request starts in the
// batch); a run's 8 values of one dimension go out as one 16-byte store, with consecutive
// lanes on consecutive dimensions so that a wave's stores are contiguous.  Every other token
// is written the coalesced 2-byte way: lane = token, 64 consecutive tokens of one dimension
// per store instruction.  Bytes are copied, never converted: the result is bit-exact.  Slots
// outside the pool are skipped.
#include <hip/hip_runtime.h>

#include "../host/internal.hpp"
#include "device_checks.hpp"

namespace {

constexpr int kTok = 64;              // tokens per work-group: one wave's lanes
constexpr int kThreads = 256;
constexpr int kMaxRuns = kTok / 8;

template <int D, int DPW>
__global__ __launch_bounds__(kThreads) void kv_scatter_kernel(
    uint16_t* __restrict__ k_pool, uint16_t* __restrict__ v_pool,
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    const int32_t* __restrict__ slots, int64_t n_tokens, int64_t n_slots, int hkv) {
  constexpr int CH = DPW / 8;          // 16-byte chunks of a row slice
  constexpr int VROW = DPW + 2;        // padded LDS row (u16): column reads spread over banks
  __shared__ uint32_t sv32[kTok * VROW / 2];
  __shared__ int32_t sslot[kTok];
  __shared__ int32_t run_tok[kMaxRuns], run_slot[kMaxRuns];
  __shared__ int32_t n_runs;
  __shared__ uint64_t covered;         // bit t: token t belongs to a run
  uint16_t* sv = reinterpret_cast<uint16_t*>(sv32);
  const int h = blockIdx.y;
  const int d0 = blockIdx.z * DPW;     // first dimension of the slice
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kTok;
  const int tid = threadIdx.x;
  if (tid < kTok) {
    const int64_t t = t0 + tid;
    const int32_t s = t < n_tokens ? slots[t] : -1;
    ARCKV_CHECK_LANE(t < n_tokens && !(s >= 0 && s < n_slots), ARCKV_CHECK_SLOT);
    sslot[tid] = (s >= 0 && s < n_slots) ? s : -1;
  }
  __syncthreads();
  if (tid < kTok) {                    // wave 0: find the runs
    const int32_t s = sslot[tid];
    bool start = s >= 0 && (s & 7) == 0 && tid + 7 < kTok;
    for (int j = 1; j < 8 && start; ++j) start = sslot[tid + j] == s + j;
    const uint64_t m = __builtin_amdgcn_ballot_w64(start);
    if (start) {
      const int r = __builtin_popcountll(m & ((1ull << tid) - 1));  // runs never overlap
      run_tok[r] = tid;
      run_slot[r] = s;
    }
    if (tid == 0) {
      uint64_t c = 0;
      for (int j = 0; j < 8; ++j) c |= m << j;
      covered = c;
      n_runs = __builtin_popcountll(m);
    }
  }
  // K: direct 16-byte copies; V: into LDS (row = token, padded)
  for (int c = tid; c < kTok * CH; c += kThreads) {
    const int tl = c / CH, ch = c % CH;
    const int64_t t = t0 + tl;
    if (t >= n_tokens) continue;
    const int64_t src = (t * hkv + h) * D + d0 + ch * 8;
    const int32_t s = sslot[tl];
    if (s >= 0) {
      const uint4 kv = *reinterpret_cast<const uint4*>(k_new + src);
      const int64_t blk = s >> 4;
      *reinterpret_cast<uint4*>(k_pool + ((blk * hkv + h) * 16 + (s & 15)) * D + d0 + ch * 8) = kv;
    }
    const uint4 vv = *reinterpret_cast<const uint4*>(v_new + src);
    uint32_t* dst = sv32 + (tl * VROW + ch * 8) / 2;  // VROW and ch*8 are even: 4-byte aligned
    dst[0] = vv.x; dst[1] = vv.y; dst[2] = vv.z; dst[3] = vv.w;
  }
  __syncthreads();
  // V of the runs: (run, dimension) per thread, dimensions fastest across lanes
  const int nr = n_runs;
  for (int e = tid; e < nr * DPW; e += kThreads) {
    const int r = e / DPW, dl = e % DPW, d = d0 + dl;
    const int tl = run_tok[r];
    const int32_t sb = run_slot[r];
    uint16_t v8[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v8[j] = sv[(tl + j) * VROW + dl];
    uint4 w;
    w.x = v8[0] | (static_cast<uint32_t>(v8[1]) << 16);
    w.y = v8[2] | (static_cast<uint32_t>(v8[3]) << 16);
    w.z = v8[4] | (static_cast<uint32_t>(v8[5]) << 16);
    w.w = v8[6] | (static_cast<uint32_t>(v8[7]) << 16);
    *reinterpret_cast<uint4*>(v_pool + ((static_cast<int64_t>(sb >> 4) * hkv + h) * D + d) * 16 + (sb & 15)) = w;
  }
  // V of the other tokens: lane = token, dimensions over the waves
  const int tl = tid & (kTok - 1);
  const int32_t s = sslot[tl];
  if (s < 0 || t0 + tl >= n_tokens || ((covered >> tl) & 1ull)) return;
  const int64_t base = ((static_cast<int64_t>(s >> 4) * hkv + h) * D + d0) * 16 + (s & 15);
  for (int d = tid >> 6; d < DPW; d += kThreads / kTok)
    v_pool[base + static_cast<int64_t>(d) * 16] = sv[tl * VROW + d];
}

}  // namespace

ARCKV_DEFINE_CHECK_READER(read_scatter_checks)

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
  for (const void* p : {static_cast<const void*>(k_pool), static_cast<const void*>(v_pool), k_new, v_new})
    if (reinterpret_cast<uintptr_t>(p) % 16 != 0)
      return arckv::fail(ARCKV_EINVAL, "kv_scatter: pools and new rows must be 16-byte aligned");
  // small batches (decode) split the head dimension finely to spread over more work-groups
  const bool small = n_tokens <= 1024;
  const int dpw = small ? 16 : head_dim;
  const dim3 grid(static_cast<unsigned>((n_tokens + kTok - 1) / kTok), num_kv_heads,
                  static_cast<unsigned>(head_dim / dpw));
  auto* st = static_cast<hipStream_t>(stream);
  auto* kp = static_cast<uint16_t*>(k_pool);
  auto* vp = static_cast<uint16_t*>(v_pool);
  auto* kn = static_cast<const uint16_t*>(k_new);
  auto* vn = static_cast<const uint16_t*>(v_new);
  const int64_t n_slots = num_blocks * 16;
#define ARCKV_SCATTER(DD, PW)                                                               \
  hipLaunchKernelGGL((kv_scatter_kernel<DD, PW>), grid, dim3(kThreads), 0, st, kp, vp, kn, vn, \
                     slot_mapping, n_tokens, n_slots, num_kv_heads)
  if (head_dim == 64) {
    if (small) ARCKV_SCATTER(64, 16); else ARCKV_SCATTER(64, 64);
  } else {
    if (small) ARCKV_SCATTER(128, 16); else ARCKV_SCATTER(128, 128);
  }
#undef ARCKV_SCATTER
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return arckv::fail(ARCKV_EDEVICE, "kv_scatter: %s", hipGetErrorString(e));
  return ARCKV_OK;
}
