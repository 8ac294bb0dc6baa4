// Producer of the computed tokens' Q/K/V: projection of their hidden states and rotary
// position embedding (the attention inputs of a prefill; the paper serves Qwen3-14B, Sec. 4,
// and the layer details follow its public configuration).
//
//   y = x W^T            x [T][H] bf16, W [(Hq + 2 Hkv) D][H] bf16, y rounded to bf16
//   q, k = rotary(y_q, y_k) at each token's absolute position; v = y_v
//
// One kernel does the projection and the rotation, so y never goes to memory:
//  * a work-group computes a 256-token x 256-output tile of y with v_mfma_f32_32x32x16_bf16;
//    its 8 waves form two groups of 4 (waves w and w + 4 share a SIMD), group g owning tokens
//    128 g .. +127 and each wave 64 tokens x 128 outputs (2 x 4 accumulator blocks of 32 x 32);
//  * x and W tiles of 32 columns of H stream global -> LDS with 16-byte direct loads (SGPR
//    base + 32-bit lane offsets) into a 4-stage ring, three stages ahead; a row's 16-byte
//    chunk c is stored at c ^ ((row / 4) % 4), so 16 lanes of an operand read hit 16
//    different 16-byte slots of the banks;
//  * the two groups run half a step apart (ping-pong): while one group's waves issue their
//    16 MFMAs of a step, the other group's waves, on the same SIMDs, read their operands of
//    the step from LDS and issue their share of the loads; every half step ends at a
//    work-group barrier, so the SIMDs' matrix units are fed by one wave or the other;
//  * the epilogue rounds y to bf16 into LDS as a [token][output] tile, then every thread
//    takes 16-byte chunks of a token's head: it rotates the (i, i + D/2) pairs in fp32 with the
//    token's (cos, sin) (its own chunk and the partner chunk D/2 away), rounds again and
//    stores the chunk whole into Q, K or V.  Values pass through.
// The (cos, sin) table of every token (D/2 angles p * theta^(-2i/D), in fp64 reduced mod 2 pi,
// then fp32 sine and cosine) comes from a small pre-pass into the caller's workspace; it finds
// each token's position from cu_q / seq_lens (suffix token i of request r sits at
// L_r - S_r + i).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "../host/internal.hpp"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kTM = 256;        // tokens per work-group tile
constexpr int kTN = 256;        // outputs per work-group tile
constexpr int kKB = 32;         // columns of H per ring stage
constexpr int kStages = 4;
constexpr int kThreads = 512;
constexpr int kGroupM = 4;       // token tiles per group of the tile order
constexpr int kStageBytes = (kTM + kTN) * kKB * 2;       // x tile then W tile: 32 KiB
constexpr int kLoadsX = kTM * kKB * 2 / (kThreads * 16);  // 16-byte loads per thread per x tile
constexpr int kLoadsW = kTN * kKB * 2 / (kThreads * 16);
static_assert(kLoadsX == 2 && kLoadsW == 2, "two loads of each tile per thread");

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {  // nearest even; inputs finite
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

// 16 bytes per lane from global memory straight into LDS: lane l reads base + ofs_l and
// writes LDS bytes [M0 + 16 l, M0 + 16 l + 16); the kernel counts these loads itself with
// vmcnt.  The SGPR base + 32-bit offset form halves the address traffic of 64-bit lane
// addresses.
__device__ __forceinline__ void load_lds16(const void* base, uint32_t ofs, lds_void* l) {
  const uint32_t m = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(l));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(ofs), "s"(base), "s"(m)
               : "memory", "m0");
}

// (cos, sin) of every token's D/2 rotary angles: tab[t][i], i < D/2.  A work-group computes
// the D/2 frequencies once (fp64 pow) and then walks tokens grid-stride, 256 / (D/2) at a
// time; the angle p f is reduced mod 2 pi in fp64 (k = floor(a / 2 pi), a - 2 pi k in one
// fma), then fp32 sine and cosine.
constexpr int kTableBlocks = 1024;
template <int D>
__global__ __launch_bounds__(256) void rope_table_kernel(int64_t n_tokens, const int32_t* __restrict__ cu_q,
                                                          const int32_t* __restrict__ seq_lens, int n_reqs,
                                                          double theta, float2* __restrict__ tab) {
  constexpr int HALF = D / 2;
  constexpr int kTokPer = 256 / HALF;     // tokens per pass of the work-group
  constexpr double kTwoPi = 6.283185307179586476925;
  __shared__ double freq[HALF];
  if (threadIdx.x < HALF) freq[threadIdx.x] = std::pow(theta, -2.0 * static_cast<int>(threadIdx.x) / D);
  __syncthreads();
  const int i = threadIdx.x % HALF;
  const double f = freq[i];
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * kTokPer + threadIdx.x / HALF; t < n_tokens;
       t += static_cast<int64_t>(gridDim.x) * kTokPer) {
    int lo = 0, hi = n_reqs - 1;          // request of token t: the last r with cu_q[r] <= t
    while (lo < hi) {
      const int mid = (lo + hi + 1) / 2;
      if (cu_q[mid] <= t) lo = mid; else hi = mid - 1;
    }
    const int64_t p = static_cast<int64_t>(seq_lens[lo]) - (cu_q[lo + 1] - cu_q[lo]) + (t - cu_q[lo]);
    const double a = static_cast<double>(p) * f;
    const double r = std::fma(-std::floor(a / kTwoPi), kTwoPi, a);
    float sn, cs;
    sincosf(static_cast<float>(r), &sn, &cs);
    tab[t * HALF + i] = make_float2(cs, sn);
  }
}

// POOL: K and V go straight into the paged pools (layout V1; k_out and v_out are then the
// pools) at slots[t] instead of into [token][head][dim] rows: K rows as 16-byte chunks, V (dim-major blocks) as 8 consecutive tokens of one dim per
// 16-byte store where the 8 tokens hold 8 aligned consecutive slots, else one 2-byte store per
// token.  Slots outside [0, n_slots) are skipped, as the scatter does.
template <int D, bool POOL>
__global__ __launch_bounds__(kThreads, 1) void qkv_gemm_rope_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w, int n_tokens, int hidden,
    int n_out, int hq, int hkv, const float2* __restrict__ tab, uint16_t* __restrict__ q_out,
    uint16_t* __restrict__ k_out, uint16_t* __restrict__ v_out, const int32_t* __restrict__ slots,
    int64_t n_slots) {
  __shared__ __attribute__((aligned(1024))) char smem[kTM * (kTN * 2 + 16)];   // ring, then the y tile
  __shared__ int32_t tslot[POOL ? kTM : 1];                                      // the tile's slots
  // Tile order.  Work-groups are dealt to the 8 XCDs in turn (b -> XCD b % 8) and each XCD has
  // its own L2, so logical tile L = (b % 8) * (G / 8) + b / 8 gives every XCD a contiguous run
  // of tiles; runs go over groups of kGroupM token tiles output-tile by output-tile, so the
  // ~32 tiles one XCD holds at a time share 4 x tiles and 8 W tiles in its L2.
  const int n_tiles_n = n_out / kTN + (n_out % kTN ? 1 : 0);
  const int n_tiles_m = n_tokens / kTM + (n_tokens % kTM ? 1 : 0);
  const int b = blockIdx.x, full = gridDim.x & ~7;
  const int L = b < full ? (b % 8) * (full / 8) + b / 8 : b;
  const int group = L / (kGroupM * n_tiles_n), in_group = L % (kGroupM * n_tiles_n);
  const int first_m = group * kGroupM, gm = min(n_tiles_m - first_m, kGroupM);
  const int tile_m = first_m + in_group % gm, tile_n = in_group / gm;
  const int t0 = tile_m * kTM, n0 = tile_n * kTN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2, wi = wave & 3;
  const int l32 = lane & 31, hg = lane >> 5;
  const int row0 = grp * 128 + (wi & 1) * 64;      // wave's 64 tokens of the tile
  const int col0 = (wi >> 1) * 128;                // wave's 128 outputs of the tile

  uint32_t xofs[kLoadsX], wofs[kLoadsW];          // byte offsets from the tile's first row
#pragma unroll
  for (int i = 0; i < kLoadsX; ++i) {
    const int row = 128 * i + 16 * wave + lane / 4;
    const int c = (lane % 4) ^ ((row >> 2) & 3);
    const int t = min(t0 + row, n_tokens - 1) - t0;
    xofs[i] = static_cast<uint32_t>(t * hidden + c * 8) * 2u;
    const int n = min(n0 + row, n_out - 1) - n0;
    wofs[i] = static_cast<uint32_t>(n * hidden + c * 8) * 2u;
  }
  const uint16_t* xbase = x + static_cast<int64_t>(t0) * hidden;
  const uint16_t* wbase = w + static_cast<int64_t>(n0) * hidden;
  const int n_k = hidden / kKB;
  auto issue = [&](int s) {       // stages past the end reload the last one into a free buffer
    char* st = smem + (s % kStages) * kStageBytes;
    const int k0 = min(s, n_k - 1) * kKB;
#pragma unroll
    for (int i = 0; i < kLoadsX; ++i)
      load_lds16(xbase + k0, xofs[i], (lds_void*)(st + i * 8192 + wave * 1024));
#pragma unroll
    for (int i = 0; i < kLoadsW; ++i)
      load_lds16(wbase + k0, wofs[i], (lds_void*)(st + kTM * kKB * 2 + i * 8192 + wave * 1024));
  };

  f32x16_t acc[2][4];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x16_t{};

  const int xr0 = row0 + l32, wr0 = col0 + l32;
  bf16x8_t a[2][2], bq[2][4];
  auto read_frags = [&](int s) {
    const char* xb = smem + (s % kStages) * kStageBytes;
    const char* wb = xb + kTM * kKB * 2;
#pragma unroll
    for (int ks = 0; ks < kKB / 16; ++ks) {
      const int c = ks * 2 + hg;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const int r = xr0 + mb * 32;
        a[ks][mb] = *reinterpret_cast<const bf16x8_t*>(xb + r * 64 + ((c ^ ((r >> 2) & 3)) * 16));
      }
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int r = wr0 + nb * 32;
        bq[ks][nb] = *reinterpret_cast<const bf16x8_t*>(wb + r * 64 + ((c ^ ((r >> 2) & 3)) * 16));
      }
    }
  };
  auto mfmas = [&]() {
#pragma unroll
    for (int ks = 0; ks < kKB / 16; ++ks)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks][mb], bq[ks][nb], acc[mb][nb], 0, 0, 0);
  };

  // ---- main loop, in half steps that all end at a work-group barrier.  Group 0 reads step s
  // in half step 2s and multiplies in 2s + 1; group 1 reads in 2s + 1 and multiplies in 2s + 2.
  // A wave issues its share of stage s + 3 right after reading step s; that stage's buffer held
  // stage s - 1, which group 0 read in half step 2s - 2 and group 1 in 2s - 1, both done.  Each
  // wave has 4 loads per stage; vmcnt(8) at the end of a half step leaves at most its two
  // newest stages in flight, so stage s + 1 is in LDS (barrier) before group 0 reads it in
  // half step 2s + 2.  Stages past the end are issued as well (a copy of the last one into a
  // buffer nobody reads any more), which keeps the counts constant.
  for (int s = 0; s < kStages - 1; ++s) issue(s);
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(2 * (kLoadsX + kLoadsW)) : "memory");
  if (grp == 1) asm volatile("s_barrier" ::: "memory");       // group 1 runs one half step behind
  for (int s = 0; s < n_k; ++s) {
    __builtin_amdgcn_sched_barrier(0);
    read_frags(s);
    issue(s + kStages - 1);
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(2 * (kLoadsX + kLoadsW)) : "memory");
    __builtin_amdgcn_sched_barrier(0);
    mfmas();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(2 * (kLoadsX + kLoadsW)) : "memory");
  }
  __builtin_amdgcn_sched_barrier(0);
  if (grp == 0) asm volatile("s_barrier" ::: "memory");       // same barrier count in both groups
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");             // no LDS write may still be in flight

  // ---- epilogue: y tile (bf16) -> LDS [token][output] (row pitch kPitch bytes), then each
  // thread rotates 16-byte chunks with their partner chunk D/2 away and stores them whole
  asm volatile("s_barrier" ::: "memory");
  constexpr int kPitch = kTN * 2 + 16;
  char* ep = smem;
  if constexpr (POOL)   // read once here (published by the barrier below), not per chunk
    if (tid < kTM) tslot[tid] = t0 + tid < n_tokens ? slots[t0 + tid] : -1;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row0 + mb * 32 + (r / 4) * 8 + hg * 4 + (r % 4);
        *reinterpret_cast<uint16_t*>(ep + row * kPitch + (col0 + nb * 32 + l32) * 2) = f32_to_bf16(acc[mb][nb][r]);
      }
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  const int nrot = (hq + hkv) * D;
  typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
#pragma unroll 4
  for (int it = 0; it < kTM * kTN / 8 / kThreads; ++it) {
    const int qc = it * kThreads + tid;
    const int row = qc / (kTN / 8), o = (qc % (kTN / 8)) * 8;
    const int t = t0 + row, n = n0 + o;
    if (t >= n_tokens || n >= n_out) continue;
    if (POOL && n >= nrot) continue;               // V: the pass below
    const int head = n / D, i0 = n % D;
    const u32x4_t own = *reinterpret_cast<const u32x4_t*>(ep + row * kPitch + o * 2);
    u32x4_t res = own;
    if (n < nrot) {
      const bool lo = i0 < D / 2;
      const u32x4_t par = *reinterpret_cast<const u32x4_t*>(ep + row * kPitch + (lo ? o + D / 2 : o - D / 2) * 2);
      const float4* cs = reinterpret_cast<const float4*>(tab + static_cast<int64_t>(t) * (D / 2) + (lo ? i0 : i0 - D / 2));
      const float sg = lo ? -1.f : 1.f;      // lo: a c - b s; hi: a c + b s (a own, b partner)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 c2 = cs[j];             // (cos, sin) of elements 2j and 2j + 1
        const float a0 = bf16_to_f32(own[j] & 0xFFFF), a1 = bf16_to_f32(own[j] >> 16);
        const float b0 = bf16_to_f32(par[j] & 0xFFFF), b1 = bf16_to_f32(par[j] >> 16);
        const uint32_t o0 = f32_to_bf16(a0 * c2.x + sg * (b0 * c2.y));
        const uint32_t o1 = f32_to_bf16(a1 * c2.z + sg * (b1 * c2.w));
        res[j] = o0 | (o1 << 16);
      }
    }
    uint16_t* dst;
    if (head < hq) {
      dst = q_out + (static_cast<int64_t>(t) * hq + head) * D + i0;
    } else if (head < hq + hkv) {
      if constexpr (POOL) {
        const int32_t sl = tslot[row];
        if (sl < 0 || sl >= n_slots) continue;
        dst = k_out + ((static_cast<int64_t>(sl >> 4) * hkv + head - hq) * 16 + (sl & 15)) * D + i0;
      } else {
        dst = k_out + (static_cast<int64_t>(t) * hkv + head - hq) * D + i0;
      }
    } else {
      dst = v_out + (static_cast<int64_t>(t) * hkv + head - hq - hkv) * D + i0;
    }
    *reinterpret_cast<u32x4_t*>(dst) = res;
  }
  if constexpr (POOL) {
    // V columns of the tile into the dim-major pool: item p is 8 tokens (rows 8 g .. 8 g + 7)
    // of one output column; consecutive threads take consecutive columns of the same tokens.
    if (n0 + kTN > nrot) {                                        // uniform
#pragma unroll 2
      for (int it = 0; it < (kTM / 8) * kTN / kThreads; ++it) {
        const int p = it * kThreads + tid;
        const int g = p / kTN, oc = p % kTN;
        const int n = n0 + oc, tf = t0 + 8 * g;
        if (n < nrot || n >= n_out || tf >= n_tokens) continue;
        const int vh = (n - nrot) / D, dim = (n - nrot) % D;
        int32_t sl[8];
        uint16_t val[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          sl[j] = tslot[8 * g + j];                               // -1 past the last token
          val[j] = *reinterpret_cast<const uint16_t*>(ep + (8 * g + j) * kPitch + oc * 2);
        }
        bool run = (sl[0] & 7) == 0 && sl[0] >= 0 && sl[0] + 7 < n_slots;
#pragma unroll
        for (int j = 1; j < 8; ++j) run = run && sl[j] == sl[0] + j;
        if (run) {     // 8 aligned consecutive slots: one block, one 16-byte row segment
          u32x4_t v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = static_cast<uint32_t>(val[2 * j]) | (static_cast<uint32_t>(val[2 * j + 1]) << 16);
          *reinterpret_cast<u32x4_t*>(v_out + ((static_cast<int64_t>(sl[0] >> 4) * hkv + vh) * D + dim) * 16 +
                                      (sl[0] & 15)) = v;
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (sl[j] >= 0 && sl[j] < n_slots)
              v_out[((static_cast<int64_t>(sl[j] >> 4) * hkv + vh) * D + dim) * 16 + (sl[j] & 15)] = val[j];
        }
      }
    }
  }
}

}  // namespace

namespace {

// Shared by arckv_qkv_rope and arckv_qkv_rope_to_pool: pool == true writes K and V into the
// pools k_dst / v_dst (num_blocks blocks) at slots.
int32_t qkv_rope_launch(const char* fn, const void* x, const void* w_qkv, int64_t n_tokens, int32_t hidden,
                        int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, const int32_t* cu_q,
                        const int32_t* seq_lens, int32_t n_reqs, double rope_theta, void* workspace,
                        int64_t ws_bytes, void* q_out, void* k_dst, void* v_dst, bool pool, int64_t num_blocks,
                        const int32_t* slots, void* stream) {
  if (n_tokens < 0 || hidden < 1 || num_q_heads < 1 || num_kv_heads < 1 || n_reqs < 0 ||
      num_q_heads % num_kv_heads != 0 || !(rope_theta > 1.0) || !std::isfinite(rope_theta))
    return arckv::fail(ARCKV_EINVAL, "%s: bad sizes or theta", fn);
  if (head_dim != 64 && head_dim != 128)
    return arckv::fail(ARCKV_EUNSUPPORTED, "%s: head_dim %d not in {64,128}", fn, head_dim);
  const int64_t n_out = static_cast<int64_t>(num_q_heads + 2 * num_kv_heads) * head_dim;
  if (hidden % kKB != 0 || hidden > (1 << 22) || n_out % 128 != 0)   // (32-bit load offsets in a tile)
    return arckv::fail(ARCKV_EUNSUPPORTED,
                       "%s: hidden %d must be a multiple of %d (at most 2^22) and the %lld outputs of 128",
                       fn, hidden, kKB, (long long)n_out);
  if (pool && (num_blocks < 1 || num_blocks > (int64_t{1} << 27)))
    return arckv::fail(ARCKV_EINVAL, "%s: num_blocks %lld", fn, (long long)num_blocks);
  if (n_tokens == 0) return ARCKV_OK;
  if (n_tokens > INT32_MAX - kTM || n_out > INT32_MAX || n_reqs < 1 ||
      static_cast<int64_t>(hidden) * n_tokens > (int64_t{1} << 40))
    return arckv::fail(ARCKV_EINVAL, "%s: %lld tokens, %lld outputs, %d requests", fn,
                       (long long)n_tokens, (long long)n_out, n_reqs);
  if (x == nullptr || w_qkv == nullptr || cu_q == nullptr || seq_lens == nullptr ||
      workspace == nullptr || q_out == nullptr || k_dst == nullptr || v_dst == nullptr ||
      (pool && slots == nullptr))
    return arckv::fail(ARCKV_EINVAL, "%s: NULL pointer", fn);
  for (const void* p : {x, w_qkv, static_cast<const void*>(workspace), static_cast<const void*>(q_out),
                        static_cast<const void*>(k_dst), static_cast<const void*>(v_dst)})
    if (reinterpret_cast<uintptr_t>(p) % 16 != 0)
      return arckv::fail(ARCKV_EINVAL, "%s: x, w_qkv, workspace and outputs must be 16-byte aligned", fn);
  const int64_t tab_bytes = n_tokens * (head_dim / 2) * static_cast<int64_t>(sizeof(float2));
  if (ws_bytes < tab_bytes)
    return arckv::fail(ARCKV_ENOSPC, "%s: workspace %lld bytes < %lld", fn, (long long)ws_bytes,
                       (long long)tab_bytes);
  auto* s = static_cast<hipStream_t>(stream);
  auto* tab = static_cast<float2*>(workspace);
  const dim3 tgrid(static_cast<unsigned>(std::min<int64_t>(kTableBlocks, (n_tokens * (head_dim / 2) + 255) / 256)));
  const int64_t n_tiles_n = (n_out + kTN - 1) / kTN;
  const dim3 grid(static_cast<unsigned>(n_tiles_n * ((n_tokens + kTM - 1) / kTM)));
  auto* xp = static_cast<const uint16_t*>(x);
  auto* wp = static_cast<const uint16_t*>(w_qkv);
  auto* q = static_cast<uint16_t*>(q_out);
  auto* k = static_cast<uint16_t*>(k_dst);
  auto* v = static_cast<uint16_t*>(v_dst);
  const int T = static_cast<int>(n_tokens), N = static_cast<int>(n_out);
  const int64_t n_slots = pool ? num_blocks * 16 : 0;
  auto go = [&](auto d_tag, auto pool_tag) {
    constexpr int D = decltype(d_tag)::value;
    constexpr bool P = decltype(pool_tag)::value;
    hipLaunchKernelGGL(rope_table_kernel<D>, tgrid, dim3(256), 0, s, n_tokens, cu_q, seq_lens, n_reqs, rope_theta, tab);
    hipLaunchKernelGGL((qkv_gemm_rope_kernel<D, P>), grid, dim3(kThreads), 0, s, xp, wp, T, hidden, N,
                       num_q_heads, num_kv_heads, tab, q, k, v, slots, n_slots);
  };
  using D64 = std::integral_constant<int, 64>;
  using D128 = std::integral_constant<int, 128>;
  if (head_dim == 64) {
    if (pool) go(D64{}, std::true_type{}); else go(D64{}, std::false_type{});
  } else {
    if (pool) go(D128{}, std::true_type{}); else go(D128{}, std::false_type{});
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return arckv::fail(ARCKV_EDEVICE, "%s: %s", fn, hipGetErrorString(e));
  return ARCKV_OK;
}

}  // namespace

extern "C" int32_t arckv_qkv_rope(const void* x, const void* w_qkv, int64_t n_tokens, int32_t hidden,
                                  int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                  const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs,
                                  double rope_theta, void* workspace, int64_t ws_bytes, void* q_out,
                                  void* k_out, void* v_out, void* stream) {
  return qkv_rope_launch("qkv_rope", x, w_qkv, n_tokens, hidden, num_q_heads, num_kv_heads, head_dim, cu_q,
                         seq_lens, n_reqs, rope_theta, workspace, ws_bytes, q_out, k_out, v_out, false, 0,
                         nullptr, stream);
}

extern "C" int32_t arckv_qkv_rope_to_pool(const void* x, const void* w_qkv, int64_t n_tokens, int32_t hidden,
                                          int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                          const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs,
                                          double rope_theta, void* workspace, int64_t ws_bytes, void* q_out,
                                          void* k_pool, void* v_pool, int64_t num_blocks,
                                          const int32_t* slot_mapping, void* stream) {
  return qkv_rope_launch("qkv_rope_to_pool", x, w_qkv, n_tokens, hidden, num_q_heads, num_kv_heads, head_dim,
                         cu_q, seq_lens, n_reqs, rope_theta, workspace, ws_bytes, q_out, k_pool, v_pool, true,
                         num_blocks, slot_mapping, stream);
}
