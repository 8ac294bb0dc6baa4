// Prefix-cached paged prefill attention for CDNA4 (gfx950).
//
// What it computes (paper, Sec. 2): prefill runs the uncached part of each prompt; with
// prefix caching the computed queries attend to the reused KV of the cached prefix and,
// causally, to each other.  For request r (L tokens, P cached, S = L - P computed), query head
// h and position j in [P, L):  o = softmax(scale * q . K[0..j]^T) . V[0..j], KV head h / G.
// K and V are read through the request's block table from the paged pool (16-token blocks,
// Sec. 4; layout V1: K [blk][kvh][16][D], V [blk][kvh][D][16]).
//
// Design (MI355X-first):
//  * One work-group = 4 wave64s = one 256-column query tile of one (request, KV head); a
//    column is (token, head-of-group), token-major, so every K/V tile a work-group loads
//    serves all G query heads of its KV head (GQA packed into the MFMA N dimension).
//  * Transposed formulation: S^T = K . Q^T and O^T = V^T . P^T with v_mfma_f32_32x32x16_bf16.
//    Query columns sit on lanes, keys / head dims on the M (register) dimension, so a lane
//    owns whole columns: row max and row sum are in-lane plus one exchange with lane +- 32.
//    Each wave owns 64 columns (two 32-column N blocks), so every K/V operand read from LDS
//    feeds two MFMAs.
//  * K rows are fed to the MFMA in an order that swaps bits 2 and 3 of the row index; the
//    accumulator layout of S^T then puts 8 consecutive keys per lane half, which is exactly
//    the B-operand layout of the P.V step, so P^T goes from registers to the next MFMA with
//    no shuffle, and V^T (dim-major blocks) is read as one 16-byte operand per lane.
//  * K/V tiles of 64 keys (4 blocks) are gathered from the scattered physical blocks with
//    16-byte loads into registers, then into double-buffered, XOR-swizzled LDS; the next
//    tile's loads are in flight while the current tile is multiplied.
//  * fp32 online softmax in base 2 (scale * log2 e folded into one FMA per score), causal
//    masking only on tiles that cross the diagonal, bf16 P with fp32 accumulation.
//  * Long key ranges with too few query tiles are split by the host plan; split items write
//    fp32 partials plus a base-2 log-sum-exp that attn_combine merges.
#include <hip/hip_runtime.h>

#include <cmath>

#include "../host/internal.hpp"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // 4 wave64
constexpr int kCols = 256;     // query columns per work-group (64 per wave)
constexpr int kBK = 64;        // keys per K/V tile

struct Work {
  int32_t req, kvh, col_start, kv_start, kv_end, slot, pad0, pad1;
};

// LDS swizzles (16-byte chunk index XOR a function of the row) so that the 8 lanes served
// together by ds_read_b128 hit 8 different bank groups.
__device__ __forceinline__ int swz_k(int row) { return (row & 3) | ((row >> 1) & 4); }
__device__ __forceinline__ int swz_v(int row) { return row & 7; }
// MFMA row i of S^T is fed by K row pi(i): bits 2 and 3 swapped.
__device__ __forceinline__ int pi_row(int i) { return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int D, int G>
__global__ __launch_bounds__(kThreads, 1) void prefill_attn_kernel(
    const uint16_t* __restrict__ k_pool, const uint16_t* __restrict__ v_pool,
    const uint16_t* __restrict__ q, uint16_t* __restrict__ out,
    const int32_t* __restrict__ block_tables, int bt_stride,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ seq_lens, int n_reqs,
    const Work* __restrict__ work, int64_t n_q, int64_t num_blocks, int hq, int hkv,
    float scale_log2, float* __restrict__ ws_o, float* __restrict__ ws_lse, int64_t ws_slots) {
  constexpr int KCH = D / 8;                        // 16-byte chunks per K row
  constexpr int KSTEPS = D / 16;                    // k-steps of Q.K^T
  constexpr int DM = D / 32;                        // 32-row blocks of O^T
  constexpr int KLOADS = kBK * KCH / kThreads;      // K chunks per thread per tile
  constexpr int VLOADS = D * (kBK / 8) / kThreads;  // V chunks per thread per tile
  __shared__ __attribute__((aligned(16))) uint16_t sk[2][kBK * D];
  __shared__ __attribute__((aligned(16))) uint16_t sv[2][D * kBK];

  const Work w = work[blockIdx.x];
  if (w.req < 0 || w.req >= n_reqs || w.kvh < 0 || w.kvh >= hkv || w.col_start < 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hg = lane >> 5;
  const int q0 = cu_q[w.req];
  const int S = cu_q[w.req + 1] - q0;
  const int L = seq_lens[w.req];
  const int P = L - S;
  const int ncols = S * G;
  const int32_t* bt = block_tables + static_cast<int64_t>(w.req) * bt_stride;
  const int nblk = min((L + 15) >> 4, bt_stride);
  const int64_t kvh_off = w.kvh;

  // ---- this lane's two query columns and their Q^T operands --------------------------
  int pos[2];
  bool cval[2];
  int64_t qrow[2];
  bf16x8_t qf[2][KSTEPS];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int col = w.col_start + wave * 64 + nb * 32 + l32;
    const int tok = col / G, g = col % G;
    cval[nb] = col < ncols && (q0 + tok) < n_q;
    pos[nb] = cval[nb] ? P + tok : -1;
    qrow[nb] = static_cast<int64_t>(q0 + tok) * hq + w.kvh * G + g;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (cval[nb])
        qf[nb][ks] = *reinterpret_cast<const bf16x8_t*>(q + qrow[nb] * D + ks * 16 + hg * 8);
      else
        qf[nb][ks] = bf16x8_t{};
    }
  }

  const int last_col = min(w.col_start + kCols, ncols) - 1;
  const int wg_max_pos = P + last_col / G;
  const int wg_min_pos = P + w.col_start / G;
  const int kv_lo = max(w.kv_start, 0);
  const int kv_hi = min(w.kv_end, wg_max_pos + 1);

  // ---- K/V tile gather: pool -> registers -> LDS ---------------------------------------
  uint4 kreg[KLOADS], vreg[VLOADS];
  auto load_tile = [&](int t0) {
#pragma unroll
    for (int i = 0; i < KLOADS; ++i) {
      const int c = tid + i * kThreads;
      const int row = c / KCH, ch = c % KCH;
      const int tok = t0 + row, b = tok >> 4;
      const int32_t phys = b < nblk ? bt[b] : -1;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (tok < L && phys >= 0 && phys < num_blocks)
        v = *reinterpret_cast<const uint4*>(
            k_pool + ((static_cast<int64_t>(phys) * hkv + kvh_off) * 16 + (tok & 15)) * D + ch * 8);
      kreg[i] = v;
    }
#pragma unroll
    for (int i = 0; i < VLOADS; ++i) {
      const int c = tid + i * kThreads;
      const int d = c >> 3, ch = c & 7;  // 8 chunks of 8 keys per 64-key row
      const int tok = t0 + ch * 8, b = tok >> 4;
      const int32_t phys = b < nblk ? bt[b] : -1;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (tok < L && phys >= 0 && phys < num_blocks) {
        v = *reinterpret_cast<const uint4*>(
            v_pool + ((static_cast<int64_t>(phys) * hkv + kvh_off) * D + d) * 16 + (ch & 1) * 8);
        const int valid = L - tok;  // keys past the prompt end hold stale bytes: zero them
        if (valid < 8) {
          uint32_t* u = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (2 * j >= valid) u[j] = 0;
            else if (2 * j + 1 >= valid) u[j] &= 0xFFFFu;
          }
        }
      }
      vreg[i] = v;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KLOADS; ++i) {
      const int c = tid + i * kThreads;
      const int row = c / KCH, ch = c % KCH;
      *reinterpret_cast<uint4*>(&sk[buf][row * D + ((ch ^ swz_k(row)) * 8)]) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < VLOADS; ++i) {
      const int c = tid + i * kThreads;
      const int d = c >> 3, ch = c & 7;
      *reinterpret_cast<uint4*>(&sv[buf][d * kBK + ((ch ^ swz_v(d)) * 8)]) = vreg[i];
    }
  };

  f32x16_t o[DM][2];
#pragma unroll
  for (int md = 0; md < DM; ++md) o[md][0] = o[md][1] = f32x16_t{};
  float m_run[2] = {-INFINITY, -INFINITY};
  float l_run[2] = {0.f, 0.f};

  if (kv_lo < kv_hi) {
    load_tile(kv_lo);
    store_tile(0);
  }
  __syncthreads();

  int buf = 0;
  for (int t0 = kv_lo; t0 < kv_hi; t0 += kBK, buf ^= 1) {
    const bool has_next = t0 + kBK < kv_hi;
    if (has_next) load_tile(t0 + kBK);

    // S^T (64 keys x 64 columns per wave) = K . Q^T
    f32x16_t s[2][2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      s[mb][0] = s[mb][1] = f32x16_t{};
      const int row = mb * 32 + pi_row(l32);
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        const int ch = 2 * ks + hg;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(&sk[buf][row * D + ((ch ^ swz_k(row)) * 8)]);
        s[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[0][ks], s[mb][0], 0, 0, 0);
        s[mb][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[1][ks], s[mb][1], 0, 0, 0);
      }
    }

    // online softmax; accumulator register r of S^T block mb holds key
    // t0 + 32 mb + 16 (r / 8) + 8 hg + r % 8 for this lane's column
    const bool need_mask = (t0 + kBK - 1 > wg_min_pos) || (t0 + kBK > L);
    bf16x8_t pb[2][4];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      float mx = -INFINITY;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float x = s[mb][nb][r];
          if (need_mask) {
            const int key = t0 + mb * 32 + 16 * (r >> 3) + 8 * hg + (r & 7);
            if (key > pos[nb]) x = -INFINITY;
          }
          s[mb][nb][r] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[nb], mx * scale_log2);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(m_run[nb] - m_use);
      m_run[nb] = m_new;
#pragma unroll
      for (int md = 0; md < DM; ++md) o[md][nb] *= alpha;
      float lsum = 0.f;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          f32x8_t pv;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float p = fast_exp2(fmaf(s[mb][nb][8 * half + j], scale_log2, -m_use));
            pv[j] = p;
            lsum += p;
          }
          pb[nb][2 * mb + half] = __builtin_convertvector(pv, bf16x8_t);
        }
      l_run[nb] = l_run[nb] * alpha + lsum;
    }

    // O^T (D x 64 columns per wave) += V^T . P^T
#pragma unroll
    for (int md = 0; md < DM; ++md) {
      const int d = md * 32 + l32;
#pragma unroll
      for (int sp = 0; sp < 4; ++sp) {
        const int ch = 2 * sp + hg;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(&sv[buf][d * kBK + ((ch ^ swz_v(d)) * 8)]);
        o[md][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[0][sp], o[md][0], 0, 0, 0);
        o[md][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[1][sp], o[md][1], 0, 0, 0);
      }
    }

    if (has_next) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: O^T register r of block md holds dim 32 md + 8 (r / 4) + 4 hg + r % 4 ----
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const float lt = l_run[nb] + __shfl_xor(l_run[nb], 32);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    const int local = wave * 64 + nb * 32 + l32;
    if (w.slot < 0) {
      if (!cval[nb]) continue;
      uint16_t* dst = out + qrow[nb] * D;
#pragma unroll
      for (int md = 0; md < DM; ++md)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          f32x4_t v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = o[md][nb][4 * r4 + j] * inv;
          const bf16x4_t b = __builtin_convertvector(v, bf16x4_t);
          *reinterpret_cast<bf16x4_t*>(dst + md * 32 + 8 * r4 + 4 * hg) = b;
        }
    } else if (w.slot < ws_slots) {
      float* po = ws_o + (static_cast<int64_t>(w.slot) * kCols + local) * D;
#pragma unroll
      for (int md = 0; md < DM; ++md)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          f32x4_t v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = o[md][nb][4 * r4 + j] * inv;
          *reinterpret_cast<f32x4_t*>(po + md * 32 + 8 * r4 + 4 * hg) = v;
        }
      if (hg == 0)
        ws_lse[static_cast<int64_t>(w.slot) * kCols + local] =
            lt > 0.f ? m_run[nb] + __log2f(lt) : -INFINITY;
    }
  }
}

// Merges the key-range splits of one query tile: o = sum_s 2^lse_s O_s / sum_s 2^lse_s.
template <int D>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(
    uint16_t* __restrict__ out, const Work* __restrict__ items, const int32_t* __restrict__ cu_q,
    int n_reqs, int64_t n_q, int hq, int G, const float* __restrict__ ws_o,
    const float* __restrict__ ws_lse, int64_t ws_slots) {
  const Work w = items[blockIdx.x];  // {req, kvh, col_start, slot0, n_splits}
  const int slot0 = w.kv_start, ns = w.kv_end;
  if (w.req < 0 || w.req >= n_reqs || w.kvh < 0 || (w.kvh + 1) * G > hq || w.col_start < 0 ||
      slot0 < 0 || ns < 1 || slot0 + ns > ws_slots)
    return;
  const int q0 = cu_q[w.req];
  const int ncols = (cu_q[w.req + 1] - q0) * G;
  constexpr int D4 = D / 4;
  for (int e = threadIdx.x; e < kCols * D4; e += kThreads) {
    const int local = e / D4, d4 = e % D4;
    const int col = w.col_start + local;
    if (col >= ncols) continue;
    const int tok = col / G, g = col % G;
    if (q0 + tok >= n_q) continue;
    float m = -INFINITY;
    for (int s = 0; s < ns; ++s) m = fmaxf(m, ws_lse[static_cast<int64_t>(slot0 + s) * kCols + local]);
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    for (int s = 0; s < ns; ++s) {
      const float lse = ws_lse[static_cast<int64_t>(slot0 + s) * kCols + local];
      const float wt = lse == -INFINITY ? 0.f : fast_exp2(lse - m);
      wsum += wt;
      const f32x4_t v = *reinterpret_cast<const f32x4_t*>(
          ws_o + (static_cast<int64_t>(slot0 + s) * kCols + local) * D + 4 * d4);
      acc += wt * v;
    }
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    const bf16x4_t b = __builtin_convertvector(acc * inv, bf16x4_t);
    *reinterpret_cast<bf16x4_t*>(out + (static_cast<int64_t>(q0 + tok) * hq + w.kvh * G + g) * D + 4 * d4) = b;
  }
}

template <int D, int G>
void launch_attn(dim3 grid, hipStream_t st, const uint16_t* kp, const uint16_t* vp,
                 const uint16_t* q, uint16_t* out, const int32_t* bt, int bt_stride,
                 const int32_t* cu_q, const int32_t* seq_lens, int n_reqs, const Work* work,
                 int64_t n_q, int64_t num_blocks, int hq, int hkv, float scale_log2, float* ws_o,
                 float* ws_lse, int64_t ws_slots) {
  hipLaunchKernelGGL((prefill_attn_kernel<D, G>), grid, dim3(kThreads), 0, st, kp, vp, q, out,
                     bt, bt_stride, cu_q, seq_lens, n_reqs, work, n_q, num_blocks, hq, hkv,
                     scale_log2, ws_o, ws_lse, ws_slots);
}

}  // namespace

extern "C" int32_t arckv_prefill_attention(const void* k_pool, const void* v_pool, const void* q,
                                           void* out, const int32_t* block_tables,
                                           int32_t bt_stride, const int32_t* cu_q,
                                           const int32_t* seq_lens, int32_t n_reqs, int64_t n_q,
                                           int64_t num_blocks, const int32_t* work,
                                           int64_t n_work, int64_t n_combine,
                                           int32_t num_q_heads, int32_t num_kv_heads,
                                           int32_t head_dim, float scale, void* workspace,
                                           int64_t ws_bytes, void* stream) {
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads != 0 || n_reqs < 0 ||
      n_q < 0 || num_blocks < 0 || n_work < 0 || n_combine < 0 || ws_bytes < 0 || bt_stride < 0 ||
      !std::isfinite(scale) || scale <= 0.f)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: bad sizes or scale");
  const int G = num_q_heads / num_kv_heads;
  if (head_dim != 64 && head_dim != 128)
    return arckv::fail(ARCKV_EUNSUPPORTED, "prefill_attention: head_dim %d not in {64,128}", head_dim);
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return arckv::fail(ARCKV_EUNSUPPORTED, "prefill_attention: group size %d not in {1,2,4,8}", G);
  if (n_work == 0 && n_combine == 0) return ARCKV_OK;
  if (k_pool == nullptr || v_pool == nullptr || q == nullptr || out == nullptr ||
      block_tables == nullptr || cu_q == nullptr || seq_lens == nullptr || work == nullptr)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: NULL pointer");
  if (n_work > INT32_MAX || n_combine > INT32_MAX)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: too many work items");
  const int64_t slot_bytes = static_cast<int64_t>(kCols) * (head_dim + 1) * 4;
  const int64_t ws_slots = workspace != nullptr ? ws_bytes / slot_bytes : 0;
  if (n_combine > 0 && ws_slots == 0)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: split plan needs a workspace");
  float* ws_o = static_cast<float*>(workspace);
  float* ws_lse = ws_o == nullptr ? nullptr : ws_o + ws_slots * kCols * head_dim;
  auto* st = static_cast<hipStream_t>(stream);
  auto* kp = static_cast<const uint16_t*>(k_pool);
  auto* vp = static_cast<const uint16_t*>(v_pool);
  auto* qp = static_cast<const uint16_t*>(q);
  auto* op = static_cast<uint16_t*>(out);
  auto* wk = reinterpret_cast<const Work*>(work);
  const float scale_log2 = scale * 1.4426950408889634f;

  if (n_work > 0) {
    const dim3 grid(static_cast<unsigned>(n_work));
#define ARCKV_LAUNCH(DD, GG)                                                                   \
  launch_attn<DD, GG>(grid, st, kp, vp, qp, op, block_tables, bt_stride, cu_q, seq_lens,       \
                      n_reqs, wk, n_q, num_blocks, num_q_heads, num_kv_heads, scale_log2,      \
                      ws_o, ws_lse, ws_slots)
    if (head_dim == 64) {
      switch (G) {
        case 1: ARCKV_LAUNCH(64, 1); break;
        case 2: ARCKV_LAUNCH(64, 2); break;
        case 4: ARCKV_LAUNCH(64, 4); break;
        default: ARCKV_LAUNCH(64, 8); break;
      }
    } else {
      switch (G) {
        case 1: ARCKV_LAUNCH(128, 1); break;
        case 2: ARCKV_LAUNCH(128, 2); break;
        case 4: ARCKV_LAUNCH(128, 4); break;
        default: ARCKV_LAUNCH(128, 8); break;
      }
    }
#undef ARCKV_LAUNCH
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
      return arckv::fail(ARCKV_EDEVICE, "prefill_attention: %s", hipGetErrorString(e));
  }
  if (n_combine > 0) {
    const dim3 grid(static_cast<unsigned>(n_combine));
    const Work* items = wk + n_work;
    if (head_dim == 64)
      hipLaunchKernelGGL(attn_combine_kernel<64>, grid, dim3(kThreads), 0, st, op, items, cu_q,
                         n_reqs, n_q, num_q_heads, G, ws_o, ws_lse, ws_slots);
    else
      hipLaunchKernelGGL(attn_combine_kernel<128>, grid, dim3(kThreads), 0, st, op, items, cu_q,
                         n_reqs, n_q, num_q_heads, G, ws_o, ws_lse, ws_slots);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
      return arckv::fail(ARCKV_EDEVICE, "attn_combine: %s", hipGetErrorString(e));
  }
  return ARCKV_OK;
}
