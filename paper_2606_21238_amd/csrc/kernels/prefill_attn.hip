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
//  * A work item is one query tile of one (request, KV head) over a key range; a column is
//    (token, head-of-group), token-major, so every K/V tile loaded serves all G query heads
//    of its KV head (GQA packed into the MFMA N dimension).  Wide tiles (256 columns): one
//    work-group per item, 8 waves x 32 columns.  Narrow tiles (128 columns: short suffixes and
//    decode-like batches): persistent work-groups that each stream a host-balanced list of
//    items through one continuous load pipeline, 4 x 32 columns with the two groups of 4 waves
//    taking the two 32-key halves of every K/V tile (separate online softmax states, merged
//    through LDS at the end of each item).
//  * Transposed formulation: S^T = K . Q^T and O^T = V^T . P^T with v_mfma_f32_32x32x16_bf16.
//    Query columns sit on lanes, keys / head dims on the M (register) dimension, so a lane
//    owns whole columns: row max and row sum are in-lane plus one exchange with lane +- 32.
//    Each wave owns 32 columns (one MFMA N block); with 32 columns a wave fits in 256
//    registers, so a SIMD holds two waves of the work-group and interleaves one wave's MFMAs
//    with the other's softmax.
//  * K rows are fed to the MFMA in an order that swaps bits 2 and 3 of the row index; the
//    accumulator layout of S^T then puts 8 consecutive keys per lane half, which is exactly
//    the B-operand layout of the P.V step, so P^T goes from registers to the next MFMA with
//    no shuffle, and V^T (dim-major blocks) is read as one 16-byte operand per lane.
//  * K/V tiles of 64 keys (4 blocks) are gathered from the scattered physical blocks with
//    16-byte direct global-to-LDS loads (the block's base in SGPRs, a 32-bit offset per lane)
//    into a ring of XOR-swizzled LDS tiles; two or three
//    tiles are in flight while the current one is multiplied.  The query tile comes through
//    the same direct loads (narrow tiles: as an element of the ring), so the first wait covers
//    the queries and tile 0 only.
//  * fp32 online softmax in base 2 (scale * log2 e folded into one FMA per score), causal
//    masking only on tiles that cross the diagonal, bf16 P with fp32 accumulation.  The
//    running maximum is lazy: O and l are rescaled only when a score exceeds it by more than
//    2^kLazy.  The wide kernel finds that from the exponentials' lane sums (non-negative
//    terms: a sum within the bound keeps every term within it) and takes column maxima only
//    on an item's first tile or when a sum exceeds the bound.
//  * Long key ranges with too few query tiles are split by the host plan (wide tiles: into
//    one round of work-groups; narrow tiles: where a list's budget ends); split items write
//    fp32 partials plus a base-2 log-sum-exp that attn_combine merges.
#include <hip/hip_runtime.h>

#include <cmath>
#include <mutex>
#include <type_traits>

#include "../host/internal.hpp"
#include "device_checks.hpp"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kStages = 4;                         // K/V tiles resident in LDS (ring)
constexpr int kBK = 64;        // keys per K/V tile (4 blocks of 16)
constexpr float kLazy = 8.0f;  // rescale O only when a column max grows by > 2^8
constexpr float kLazySum = 256.0f;  // 2^kLazy

struct Work {
  int32_t req, kvh, col_start, kv_start, kv_end, slot, pad0, pad1;
};
static_assert(sizeof(Work) == ARCKV_WORK_INTS * sizeof(int32_t), "a work item is ARCKV_WORK_INTS ints");
// read-only kernel inputs seen through the constant address space (scalar loads)
typedef __attribute__((address_space(4))) const int32_t cint32;

// MFMA row i of S^T is fed by K row pi(i) (bits 2 and 3 swapped): then accumulator register r
// of a lane in half hg holds key 16 (r / 8) + 8 hg + r % 8 of its 32-key block, which is the
// B-operand order of the P.V step.
__device__ __forceinline__ int pi_row(int i) { return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1); }

// LDS layouts (ds_read_b128 is conflict-free when each 16-lane group reads 16 different
// 16-byte slots of a 256-byte bank window):
//  K tile: 64 key rows of D bf16; 16-byte chunk c of row r stored at chunk c ^ fk(r).
//  V tile: block-major [4][D][16 keys]; 16-byte half h of dim row d stored at h ^ sv(d).
template <int D>
__device__ __forceinline__ int fk(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
__device__ __forceinline__ int sv(int d) { return (d >> 3) & 1; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// v_permlane32_swap(a, b) exchanges the upper half of a with the lower half of b.  With b = a,
// one result holds lanes 0..31 of x in both halves and the other lanes 32..63, so the max / sum
// of the pair combines lanes l and l ^ 32 in every lane with no LDS round trip.  (The results
// are copied to scalars before the bit casts: a bit cast of a vector element subscript was
// compiled as a cast of element 0.)
__device__ __forceinline__ void halves(float x, float& lo, float& hi) {
  const uint32_t a = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(a, a, false, false);
  const uint32_t r0 = r[0], r1 = r[1];
  lo = __builtin_bit_cast(float, r0);
  hi = __builtin_bit_cast(float, r1);
}
__device__ __forceinline__ float max_halves(float x) {
  float lo, hi;
  halves(x, lo, hi);
  return fmaxf(lo, hi);
}
__device__ __forceinline__ float sum_halves(float x) {
  float lo, hi;
  halves(x, lo, hi);
  return lo + hi;
}

// 16 bytes per lane from global memory straight into LDS (lane l writes LDS bytes
// [M0 + 16 l, M0 + 16 l + 16)).  Written as inline assembly on purpose: the compiler's wait
// insertion treats its own LDS-DMA loads as pending LDS traffic and then waits for every LDS
// read to return before each MFMA; the kernel does its own vmcnt accounting for these loads
// (every compiler-visible vector load has completed before the first one is issued).
__device__ __forceinline__ void load_lds16(const void* g, lds_void* l) {
  const uint32_t m = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(l));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(m)
               : "memory", "m0");
}
// The same from a wave-uniform 64-bit base held in SGPRs plus a 32-bit byte offset per lane.
// The K/V tiles load this way (one block of one head per instruction and wave): the lanes then
// carry 4 address bytes instead of 8, which measured 1-2.5 % faster on long suffixes.
__device__ __forceinline__ void load_lds16_s(const void* base, uint32_t ofs, lds_void* l) {
  const uint32_t m = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(l));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(ofs), "s"(base), "s"(m)
               : "memory", "m0");
}

// Narrow tiles (128 query columns: short suffixes and decode-like batches) run as persistent
// work-groups.  The host plan hands every work-group a list of up to kListItems items (its live
// items first, then idle padding), balanced so that the lists of a launch carry about equal
// work; a work-group streams its list back to back through one LDS ring.  The ring's elements
// are, per item, the item's Q tile and then its K/V tiles (a 128-column Q tile is exactly the
// size of one K/V tile pair), and the loads run three elements ahead across item boundaries,
// so the pipeline does not drain between items.
//
// Eight waves: four column waves of 32 columns times two key halves; half h takes keys
// [32 h, 32 h + 32) of every 64-key tile with its own online softmax, and at the end of an item
// half 1 hands (m, l, O) to half 0 through the two ring stages that are free at that point.
// Two waves share each SIMD, so one wave's exponentials overlap the other's MFMAs.
template <int D, int G>
__global__ __launch_bounds__(512, 1) void prefill_attn_list_kernel(
    const uint16_t* __restrict__ k_pool, const uint16_t* __restrict__ v_pool,
    const uint16_t* __restrict__ q, uint16_t* __restrict__ out,
    const int32_t* __restrict__ block_tables, int bt_stride,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ seq_lens, int n_reqs,
    const Work* __restrict__ work, int64_t n_q, int64_t num_blocks, int hq, int hkv,
    float scale_log2, float* __restrict__ ws_o, float* __restrict__ ws_lse, int64_t ws_slots) {
  constexpr int kThreads = 512;
  constexpr int kCW = 4;                         // column waves of 32 columns
  constexpr int kCols = kCW * 32;                // query columns of a narrow tile
  constexpr int KSTEPS = D / 16;                 // k-steps of Q.K^T
  constexpr int DM = D / 32;                     // 32-row blocks of O^T
  constexpr int TILE = kBK * D * 2;              // bytes of one K (or V) tile
  constexpr int STAGE = 2 * TILE;                // one ring element: K then V, or a Q tile
  static_assert(kCols * D * 2 == STAGE, "a Q tile fills one ring stage");
  constexpr int kRing = 5;                       // three elements in flight + two free stages
  constexpr int LDB = kThreads * 16;             // bytes one load instruction moves per WG
  constexpr int NLD = TILE / LDB;                // 16-byte direct loads per thread per K tile
  constexpr int NEL = STAGE / LDB;               // ... per ring element
  constexpr int BLK_BYTES = 16 * D * 2;          // one block of one head, K or V
  static_assert(NLD >= 1 && TILE % LDB == 0, "tile must be a multiple of one WG-wide load");
  constexpr int MDR = DM / 2;                    // O blocks a half hands over per merge pass
  static_assert(kCW * MDR * 4 * 64 * 16 == STAGE, "one merge pass fills one stage");
  __shared__ __attribute__((aligned(1024))) char smem[kRing * STAGE];
  if (n_q <= 0) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cw = wave % kCW, kh = wave / kCW;    // column wave, key half
  const int l32 = lane & 31, hg = lane >> 5;
  auto stage = [&](int e) { return smem + (e % kRing) * STAGE; };

  // ---- the items of the list ------------------------------------------------------------
  // Entries up to the first idle one (request < 0) are the list; an entry naming no request,
  // KV head or column is skipped (and recorded in a device-checked build).  Everything the
  // cursors need of an entry is computed once, before the first load of the ring, into a table
  // of two registers (lane 8 f + j holds field f of entry j), so that moving to the next item
  // costs register reads only: a memory load there would wait for the loads of the ring.
  enum { F_OK, F_REQ, F_KVH, F_COL, F_SLOT, F_Q0, F_NCOLS, F_P,
         F_L, F_KVLO, F_NT, F_MINPOS, F_NBLK };  // F_OK: 1 item, 0 skipped entry, -1 past the end
  int32_t tbl[2];
  {
    const int j = lane & 7, f = lane >> 3;
    const Work w = work[static_cast<int64_t>(blockIdx.x) * arckv::kListItems + j];
    const uint64_t idle = __builtin_amdgcn_ballot_w64(lane < arckv::kListItems && w.req < 0);
    const bool live = (idle & ((2ull << j) - 1)) == 0;
    const bool bad = w.req >= n_reqs || w.kvh < 0 || w.kvh >= hkv || w.col_start < 0;
    ARCKV_CHECK_LANE(lane < arckv::kListItems && live && bad, ARCKV_CHECK_WORK);
    const bool ok = live && !bad;
    const int q0 = ok ? cu_q[w.req] : 0;
    const int S = ok ? cu_q[w.req + 1] - q0 : 0;
    const int L = ok ? seq_lens[w.req] : 0;
    const int P = L - S, ncols = S * G;
    const int last_col = min(w.col_start + kCols, ncols) - 1;
    const int kv_lo = max(w.kv_start, 0);
    const int kv_hi = min(w.kv_end, P + last_col / G + 1);
    const int nt = ok && kv_hi > kv_lo ? (kv_hi - kv_lo + kBK - 1) / kBK : 0;
    const int v0[8] = {ok ? 1 : (live ? 0 : -1), w.req, w.kvh, w.col_start, w.slot, q0, ncols, P};
    const int v1[8] = {L, kv_lo, nt, P + w.col_start / G, min((L + 15) >> 4, bt_stride), 0, 0, 0};
    int t0 = 0, t1 = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      t0 = f == k ? v0[k] : t0;
      t1 = f == k ? v1[k] : t1;
    }
    tbl[0] = t0;
    tbl[1] = t1;
  }
  auto field = [&](int fld, int j) {
    return fld < 8 ? __builtin_amdgcn_readlane(tbl[0], fld * 8 + j) : __builtin_amdgcn_readlane(tbl[1], (fld - 8) * 8 + j);
  };
  // The block tables are read through the constant address space: the kernel never writes
  // them, and this keeps their (uniform) loads scalar after the epilogue stores of an earlier
  // item, where a vector load would make the compiler wait for every load of the ring.
  const cint32* const cbt = (const cint32*)(block_tables);
  struct Item {
    int j, req, kvh, col_start, slot, q0, L, P, ncols, kv_lo, nt, min_pos, nblk;
    const cint32* bt;
  };
  auto find_item = [&](int j, Item& it) -> bool {
    for (; j < arckv::kListItems; ++j) {
      const int st = field(F_OK, j);
      if (st < 0) return false;
      if (st == 0) continue;
      it.j = j;
      it.req = field(F_REQ, j);
      it.kvh = field(F_KVH, j);
      it.col_start = field(F_COL, j);
      it.slot = field(F_SLOT, j);
      it.q0 = field(F_Q0, j);
      it.ncols = field(F_NCOLS, j);
      it.P = field(F_P, j);
      it.L = field(F_L, j);
      it.kv_lo = field(F_KVLO, j);
      it.nt = field(F_NT, j);
      it.min_pos = field(F_MINPOS, j);
      it.nblk = field(F_NBLK, j);
      it.bt = cbt + static_cast<int64_t>(it.req) * bt_stride;
      return true;
    }
    return false;
  };

  // ---- loads: direct global -> LDS, one ring element per call ------------------------------
  // load i of a thread covers LDS bytes [i*LDB + wave*1024 + lane*16, +16) of a K or V tile;
  // each wave's 1 KiB lies inside one block, so the block's physical address is wave-uniform.
  int k_off[NLD], v_off[NLD], blk_of[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int posb = i * LDB + wave * 1024 + lane * 16;
    const int r = posb / (2 * D), p = (posb % (2 * D)) / 16;      // K: row r, stored chunk p
    blk_of[i] = (i * LDB + wave * 1024) / BLK_BYTES;               // the same for every lane
    k_off[i] = (r & 15) * D + ((p ^ fk<D>(r)) * 8);               // elements inside the block
    const int qv = posb % BLK_BYTES, d = qv / 32, h = ((qv / 16) & 1) ^ sv(d);
    v_off[i] = d * 16 + h * 8;
  }
  const int64_t blk_stride = static_cast<int64_t>(hkv) * 16 * D;  // elements per physical block
  // block entries outside [0, num_blocks) (negative ones too, as unsigned) read block 0
  const uint32_t nb32 = static_cast<uint32_t>(num_blocks < INT32_MAX ? num_blocks : INT32_MAX);
  // The load cursor: item `ld`, next element `lt` (-1: its Q tile, else K/V tile lt), and the
  // physical blocks of its next K/V tile.  Those are read at the end of the element before
  // (prefetch_ph, right before its wait), so the scalar loads' latency hides under that wait.
  Item ld;
  bool ld_live = find_item(0, ld);
  int lt = -1, n_issued = 0;
  int32_t next_ph[NLD];
  auto fetch_ph = [&](int tile) {
    const int b0 = (ld.kv_lo + tile * kBK) >> 4;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int b = b0 + blk_of[i];
      next_ph[i] = b < ld.nblk ? ld.bt[b] : 0;
    }
  };
  // Q tile: column c (a row of q) holds its 16-byte chunks j at slot j ^ fk(c); columns past
  // the request load row 0 of q, never read back.
  auto load_q = [&](char* st) {
#pragma unroll
    for (int j = 0; j < NEL; ++j) {
      const int b = j * LDB + wave * 1024 + lane * 16;
      const int c = b / (2 * D), p = (b % (2 * D)) / 16;
      const int gc = ld.col_start + c;
      const int tok = gc / G, g = gc % G;
      const bool ok = gc < ld.ncols && (ld.q0 + tok) < n_q;
      const int64_t row = ok ? static_cast<int64_t>(ld.q0 + tok) * hq + ld.kvh * G + g : 0;
      load_lds16(q + row * D + ((p ^ fk<D>(c)) * 8), (lds_void*)(st + j * LDB + wave * 1024));
    }
  };
  auto prefetch_ph = [&]() {
    if (ld_live && lt >= 0) fetch_ph(lt);
  };
  auto load_kv = [&](char* st) {
    int32_t ph[NLD];
#pragma unroll
    for (int i = 0; i < NLD; ++i) ph[i] = next_ph[i];
    const int64_t head_k = static_cast<int64_t>(ld.kvh) * 16 * D;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      ARCKV_CHECK_WAVE(ph[i] < 0 || ph[i] >= num_blocks, ARCKV_CHECK_BLOCK);
      // wave-uniform (the wave's 1 KiB lies in one block); an entry out of range reads block 0
      const int32_t pb = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(ph[i]) >= nb32 ? 0 : ph[i]);
      const int64_t base = static_cast<int64_t>(pb) * blk_stride + head_k;
      load_lds16_s(k_pool + base, static_cast<uint32_t>(k_off[i]) * 2u, (lds_void*)(st + i * LDB + wave * 1024));
      load_lds16_s(v_pool + base, static_cast<uint32_t>(v_off[i]) * 2u, (lds_void*)(st + TILE + i * LDB + wave * 1024));
    }
  };
  // Issues the next element of the list (NEL loads per thread) into its ring stage; false
  // once the list is exhausted (nothing issued).
  auto issue = [&]() -> bool {
    if (!ld_live) return false;
    char* st = stage(n_issued);
    if (lt < 0) load_q(st);
    else load_kv(st);
    ++lt;
    if (lt >= ld.nt) {
      ld_live = find_item(ld.j + 1, ld);
      lt = -1;
    }
    ++n_issued;
    return true;
  };
  // End of an element: every element up to the one after next is in LDS (only the newest,
  // issued at the start of this element, may be pending: loads complete in order), and every
  // wave's LDS reads have returned.  The wait and the barrier are written out: a fenced
  // __syncthreads() would also wait for the newest loads.
  auto end_element = [&](bool issued) {
    prefetch_ph();
    if (issued) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(NEL) : "memory");
    else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };
  auto lds_barrier = [&]() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

  // ---- MFMA pieces ------------------------------------------------------------------------
  bf16x8_t qf[KSTEPS];
  // S^T (this wave's 32 keys of the tile x its 32 columns) = K . Q^T
  auto mma_s = [&](f32x16_t& s, const char* kb) {
    s = f32x16_t{};
    const int r = kh * 32 + pi_row(l32);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const int c = 2 * ks + hg;
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(kb + r * 2 * D + ((c ^ fk<D>(r)) * 16));
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s, 0, 0, 0);
    }
  };
  f32x16_t o[DM];
  float m_run, l_run, alpha;
  bool pending = false;  // wave-uniform
  int pos = -1;          // this lane's query position (-1: no column)
  // causal / prompt-end mask: accumulator register r holds key t0 + 32 kh + 16 (r / 8) +
  // 8 hg + r % 8 of this lane's column
  auto apply_mask = [&](f32x16_t& s, int t0) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = t0 + kh * 32 + 16 * (r >> 3) + 8 * hg + (r & 7);
      s[r] = key > pos ? -INFINITY : s[r];
    }
  };
  // Column maximum of a tile (base-2 scaled) and the lazy-rescale decision, without branches:
  // the running maximum moves only when some column of the wave grew by more than 2^kLazy;
  // then O and l are scaled by alpha before the next P.V product (apply_rescale).
  auto update_max = [&](const f32x16_t& s) {
    float m = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) m = fmaxf(m, s[r]);
    const float mx = max_halves(m) * scale_log2;
    pending = __builtin_amdgcn_ballot_w64(mx > m_run + kLazy) != 0;
    const float m_new = pending ? fmaxf(m_run, mx) : m_run;
    alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_run - m_new);
    m_run = m_new;
  };
  auto apply_rescale = [&]() {
    if (pending) {
      l_run *= alpha;
#pragma unroll
      for (int md = 0; md < DM; ++md) o[md] *= alpha;
    }
  };
  // p = 2^(s * scale * log2 e - m) rounded to bf16: the P^T operands of the P.V product.  The
  // row sums accumulate the fp32 p (before the rounding the P.V operand gets).
  uint32_t pw[2][4];
  auto exp_phase = [&](const f32x16_t& s) {
    const float mu = m_run == -INFINITY ? 0.f : m_run;
    float lsum = -0.f;                   // -0 + x == x for every x: the first add folds away
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x2_t two = {fast_exp2(fmaf(s[8 * half + 2 * j], scale_log2, -mu)),
                             fast_exp2(fmaf(s[8 * half + 2 * j + 1], scale_log2, -mu))};
        lsum += two[0];
        lsum += two[1];
        pw[half][j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(two, bf16x2_t));
      }
    l_run += lsum;
  };
  // O^T (D x this wave's columns) += V^T . P^T over this half's two 16-key blocks of the tile
  auto mma_pv = [&](const char* vb) {
#pragma unroll
    for (int sp = 0; sp < 2; ++sp)
#pragma unroll
      for (int md = 0; md < DM; ++md) {
        const int d = md * 32 + l32;
        const int blk = kh * 2 + sp;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(vb + blk * BLK_BYTES + d * 32 + ((hg ^ sv(d)) * 16));
        const u32x4_t w4 = {pw[sp][0], pw[sp][1], pw[sp][2], pw[sp][3]};
        o[md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8_t, w4), o[md], 0, 0, 0);
      }
  };
  // keys >= L of the prompt's last tile may hold stale bytes (even NaN patterns): zero their V
  auto zero_v_tail = [&](char* vbytes, int t0, int L) {
    uint16_t* vb = reinterpret_cast<uint16_t*>(vbytes);
    for (int x = tid; x < kBK * D; x += kThreads) {
      const int key = x & (kBK - 1), d = x / kBK;
      if (t0 + key >= L) {
        const int blk = key >> 4, kk = key & 15;
        const int h = ((kk >> 3) ^ sv(d));
        vb[(blk * BLK_BYTES + d * 32 + h * 16) / 2 + (kk & 7)] = 0;
      }
    }
  };

  // ---- the pipeline -------------------------------------------------------------------------
  // Element e is consumed after elements <= e + 1 are in LDS (a K/V tile's step multiplies the
  // next tile's K as well); element e + 3 is issued at its start into the stage element e - 2
  // used, free since the barrier ending element e - 1.
  {
    issue();
    prefetch_ph();
    issue();
    prefetch_ph();
    end_element(issue());
  }
  int e = 0;  // element being consumed
  Item it;
  f32x16_t sa, sb;
  for (bool live = find_item(0, it); live; live = find_item(it.j + 1, it)) {
    // ---- element e: the item's Q tile -> registers; S(0) --------------------------------
    const bool iq = issue();
    const int col = it.col_start + cw * 32 + l32;
    const bool cval = col < it.ncols && (it.q0 + col / G) < n_q;
    pos = cval ? it.P + col / G : -1;
    {
      const char* qs = stage(e);
      const int c = cw * 32 + l32;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks)
        qf[ks] = cval ? *reinterpret_cast<const bf16x8_t*>(qs + c * 2 * D + (((ks * 2 + hg) ^ fk<D>(c)) * 16))
                      : bf16x8_t{};
    }
#pragma unroll
    for (int md = 0; md < DM; ++md) o[md] = f32x16_t{};
    m_run = -INFINITY;
    l_run = 0.f;
    pending = false;
    const int nt = it.nt;
    auto tile_masked = [&](int t) {
      const int t0 = it.kv_lo + t * kBK;
      return (t0 + kBK - 1 > it.min_pos) || (t0 + kBK > it.L);
    };
    if (nt > 0) {
      mma_s(sa, stage(e + 1));
      if (tile_masked(0)) apply_mask(sa, it.kv_lo);
      update_max(sa);
    }
    end_element(iq);
    ++e;

    // ---- elements e .. e + nt - 1: the K/V tiles -------------------------------------------
    // step i: S(i+1) = K(i+1) Q^T (beside the exponentials of tile i), O += V(i) P(i), then the
    // mask and maximum of tile i+1.  A rescale decided at step i is applied at step i+1.  Steps
    // whose next tile needs masking run in a second, peeled loop.
    auto step = [&](auto mask_next, f32x16_t& sc, f32x16_t& sn, int i) {
      constexpr bool MASK_NEXT = decltype(mask_next)::value;
      const int t0 = it.kv_lo + i * kBK;
      const bool iss = issue();
      char* cur = stage(e);
      if (t0 + kBK > it.L) {  // uniform: only the tile holding the prompt end
        zero_v_tail(cur + TILE, t0, it.L);
        lds_barrier();
      }
      apply_rescale();
      mma_s(sn, stage(e + 1));  // past the item's last tile this reads another element: unused
      exp_phase(sc);
      mma_pv(cur + TILE);
      if constexpr (MASK_NEXT) {
        if (i + 1 < nt) {       // never feed an element that is not this item's tile to the max
          apply_mask(sn, t0 + kBK);
          update_max(sn);
        }
      } else {
        update_max(sn);         // main-loop steps always have a next tile
      }
      end_element(iss);
      ++e;
    };
    int n_main = nt > 0 ? nt - 1 : 0;
    {
      int lo = 0, hi = n_main;  // first step whose next tile is masked (monotone), else n_main
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (tile_masked(mid + 1)) hi = mid; else lo = mid + 1;
      }
      n_main = lo;
    }
    int i = 0;
    for (; i + 1 < n_main; i += 2) {
      step(std::false_type{}, sa, sb, i);
      step(std::false_type{}, sb, sa, i + 1);
    }
    if (i < n_main) {
      step(std::false_type{}, sa, sb, i);
      sa = sb;
      ++i;
    }
    for (; i < nt; ++i) {
      step(std::true_type{}, sa, sb, i);
      sa = sb;
    }

    // ---- key halves: half 1 hands (m, l, O) to half 0 ---------------------------------------
    // Consumed elements e - 1 and e - 2 leave their stages free until element e + 3 and e + 4
    // are issued (at the starts of elements e and e + 1).  Pass 0: O blocks [0, MDR) through
    // stage e - 1, m and l through stage e - 2; pass 1: O blocks [MDR, DM) through stage e - 1.
    // Layout: O as [column wave][block][r / 4][lane] float4; m, l as [column wave][lane].
    {
      f32x4_t* xo = reinterpret_cast<f32x4_t*>(stage(e + kRing - 1)) + cw * (MDR * 4 * 64);
      float* xm = reinterpret_cast<float*>(stage(e + kRing - 2)) + cw * 128;
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int pass = 0; pass < 2; ++pass) {
        if (kh == 1) {
#pragma unroll
          for (int mdr = 0; mdr < MDR; ++mdr)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              f32x4_t v;
#pragma unroll
              for (int j = 0; j < 4; ++j) v[j] = o[pass * MDR + mdr][4 * r4 + j];
              xo[(mdr * 4 + r4) * 64 + lane] = v;
            }
          if (pass == 0) {
            xm[lane] = m_run;
            xm[64 + lane] = l_run;
          }
        }
        lds_barrier();
        if (kh == 0) {
          if (pass == 0) {
            const float mb = xm[lane], lb = xm[64 + lane];
            const float m = fmaxf(m_run, mb);
            a = m_run == -INFINITY ? 0.f : fast_exp2(m_run - m);
            b = mb == -INFINITY ? 0.f : fast_exp2(mb - m);
            l_run = a * l_run + b * lb;
            m_run = m;
          }
#pragma unroll
          for (int mdr = 0; mdr < MDR; ++mdr)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              const f32x4_t v = xo[(mdr * 4 + r4) * 64 + lane];
#pragma unroll
              for (int j = 0; j < 4; ++j)
                o[pass * MDR + mdr][4 * r4 + j] = a * o[pass * MDR + mdr][4 * r4 + j] + b * v[j];
            }
        }
        if (pass == 0) lds_barrier();
      }
    }
    // Half 1 may run ahead into the next item: its first issue writes stage e + 3 (= e - 2),
    // whose last reads (m, l) came before the barrier that ended pass 0.

    // ---- epilogue (half 0): O^T register r of block md holds dim 32 md + 8 (r / 4) + 4 hg + r % 4
    // (the row sum pairs lanes l and l ^ 32, so every lane of the wave takes part)
    const float lt_sum = sum_halves(l_run);
    const float inv = lt_sum > 0.f ? 1.f / lt_sum : 0.f;
    const float lse = lt_sum > 0.f ? m_run + __log2f(lt_sum) : -INFINITY;
    if (kh == 0 && cval) {
      if (it.slot < 0) {
        uint16_t* dst = out + (static_cast<int64_t>(it.q0 + col / G) * hq + it.kvh * G + col % G) * D;
#pragma unroll
        for (int md = 0; md < DM; ++md)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            f32x4_t v;
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = o[md][4 * r4 + j] * inv;
            *reinterpret_cast<bf16x4_t*>(dst + md * 32 + 8 * r4 + 4 * hg) = __builtin_convertvector(v, bf16x4_t);
          }
      } else if (it.slot < ws_slots) {
        const int local = cw * 32 + l32;
        float* po = ws_o + (static_cast<int64_t>(it.slot) * kCols + local) * D;
#pragma unroll
        for (int md = 0; md < DM; ++md)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            f32x4_t v;
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = o[md][4 * r4 + j] * inv;
            *reinterpret_cast<f32x4_t*>(po + md * 32 + 8 * r4 + 4 * hg) = v;
          }
        if (hg == 0) ws_lse[static_cast<int64_t>(it.slot) * kCols + local] = lse;
      }
    }
  }
}

// Wide tiles (256 columns, 8 waves of 32 columns), scheduled as a ping-pong.  Every wave runs
// the same step on tile j as two halves:
//   V(j): mask (diagonal tiles), column max, lazy rescale of O, exponentials -> P(j), row sums
//   M(j): O += V(j) P(j)  (16 MFMAs), then S(j+1) = K(j+1) Q^T  (16 MFMAs)
// Waves 0-3 run half a step ahead of waves 4-7 (a workgroup barrier ends every half step), and
// waves w and w + 4 share a SIMD, so on every SIMD one wave's exponentials run while the other
// wave's MFMAs do.  S is single-buffered (V(j) consumes S(j) before M(j) writes S(j+1)); the
// registers this frees hold the LDS operands of the MFMA phase four MFMAs ahead of their use.
//
// Half steps are numbered globally: group 0 (waves 0-3) runs M(-1) = S(0) in half step 0, then
// V(j) in 2j+1 and M(j) in 2j+2; group 1 runs the same one half step later.  Each wave issues
// its pieces of tile t during its M(t-3) (tiles 0-2 before the loop), one load every few MFMAs
// (half step 2t-4 for group 0, 2t-3 for group 1), and they must be complete by the end of half
// step 2t-1, the barrier before tile t's first reader (group 0's M(t-1)).  They overwrite the
// ring stage of tile t-4, whose last reader (group 1's M(t-4)) ran in half step 2t-5.  The block
// numbers come from a copy of the item's block-table slice in LDS, read one tile ahead.
template <int D, int G>
__global__ __launch_bounds__(512, 1) void prefill_attn_pp_kernel(
    const uint16_t* __restrict__ k_pool, const uint16_t* __restrict__ v_pool,
    const uint16_t* __restrict__ q, uint16_t* __restrict__ out,
    const int32_t* __restrict__ block_tables, int bt_stride,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ seq_lens, int n_reqs,
    const Work* __restrict__ work, int64_t n_q, int64_t num_blocks, int hq, int hkv,
    float scale_log2, float* __restrict__ ws_o, float* __restrict__ ws_lse, int64_t ws_slots) {
  constexpr int kThreads = 512;
  constexpr int kCols = arckv::kWideCols;
  static_assert(kCols == 8 * 32, "8 waves of 32 columns");
  constexpr int KSTEPS = D / 16;                 // k-steps of Q.K^T
  constexpr int DM = D / 32;                     // 32-row blocks of O^T
  constexpr int TILE = kBK * D * 2;              // bytes of one K (or V) tile
  constexpr int NLD = TILE / (kThreads * 16);    // 16-byte direct loads per thread per tile
  constexpr int LDB = kThreads * 16;             // bytes one load instruction moves per WG
  constexpr int BLK_BYTES = 16 * D * 2;          // one block of one head, K or V
  constexpr int NOP = 4 * DM + 2 * KSTEPS;       // MFMAs of a full M phase
  constexpr int PD = 3;                          // LDS operands in flight ahead of their MFMA (3 measured 1-2 % faster than 2, 4, 5 or 6)
  static_assert(NLD >= 1 && TILE % LDB == 0, "tile must be a multiple of one WG-wide load");
  constexpr int kTbl = arckv::kMaxItemKeys / 16;  // block-table entries of one work item
  __shared__ __attribute__((aligned(1024))) char smem[kStages * 2 * TILE];  // stage s: K, then V
  __shared__ int32_t tbl[kTbl];

  const Work w = work[blockIdx.x];
  // an idle item (request -1) pads the XCD phase; anything else out of range is malformed
  ARCKV_CHECK_WAVE(w.req >= n_reqs || (w.req >= 0 && (w.kvh < 0 || w.kvh >= hkv || w.col_start < 0)),
                   ARCKV_CHECK_WORK);
  if (w.req < 0 || w.req >= n_reqs || w.kvh < 0 || w.kvh >= hkv || w.col_start < 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;
  const int l32 = lane & 31, hg = lane >> 5;
  const int q0 = cu_q[w.req];
  const int S = cu_q[w.req + 1] - q0;
  const int L = seq_lens[w.req];
  const int P = L - S;
  const int ncols = S * G;
  const int32_t* bt = block_tables + static_cast<int64_t>(w.req) * bt_stride;
  const int nblk = min((L + 15) >> 4, bt_stride);

  // ---- this lane's query column and its Q^T operands ------------------------------------
  const int col = w.col_start + wave * 32 + l32;
  const int tok = col / G, g = col % G;
  const bool cval = col < ncols && (q0 + tok) < n_q;
  const int pos = cval ? P + tok : -1;
  bf16x8_t qf[KSTEPS];
  {
    const int64_t qrow = static_cast<int64_t>(q0 + tok) * hq + w.kvh * G + g;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks)
      qf[ks] = cval ? *reinterpret_cast<const bf16x8_t*>(q + qrow * D + ks * 16 + hg * 8) : bf16x8_t{};
  }

  const int last_col = min(w.col_start + kCols, ncols) - 1;
  const int wg_max_pos = P + last_col / G;
  const int wg_min_pos = P + w.col_start / G;
  const int kv_lo = max(w.kv_start, 0);
  const int kv_hi = min(w.kv_end, wg_max_pos + 1);
  const int ntiles = kv_hi > kv_lo ? (kv_hi - kv_lo + kBK - 1) / kBK : 0;

  // ---- direct global -> LDS tile loads (as in prefill_attn_list_kernel) ------------------
  int k_off[NLD], v_off[NLD], blk_of[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int posb = i * LDB + wave * 1024 + lane * 16;
    const int r = posb / (2 * D), p = (posb % (2 * D)) / 16;
    blk_of[i] = posb / BLK_BYTES;
    k_off[i] = (r & 15) * D + ((p ^ fk<D>(r)) * 8);
    const int qv = posb % BLK_BYTES, d = qv / 32, h = ((qv / 16) & 1) ^ sv(d);
    v_off[i] = d * 16 + h * 8;
  }
  const int64_t head_k = static_cast<int64_t>(w.kvh) * 16 * D;
  const int64_t blk_stride = static_cast<int64_t>(hkv) * 16 * D;
  const uint32_t nb32 = static_cast<uint32_t>(num_blocks < INT32_MAX ? num_blocks : INT32_MAX);
  // The item's block-table entries (blocks b_lo .. b_lo + n_tbl - 1) are copied to LDS once:
  // the loop then looks them up there.  Scalar loads of the table inside the loop would force
  // a wait for the scalar memory round trip at every tile (and, while one is in flight, full
  // waits on every LDS operand read, since scalar loads may return out of order).  The host
  // plan keeps every item within kMaxItemKeys keys, so n_tbl <= kTbl.
  const int b_lo = kv_lo >> 4;
  const int n_tbl = max(0, min(min(nblk - b_lo, ntiles * (kBK / 16)), kTbl));
  constexpr int kTblPer = kTbl / kThreads;
  int32_t tbl_v[kTblPer];
#pragma unroll
  for (int k = 0; k < kTblPer; ++k) {
    const int e = tid + k * kThreads;
    tbl_v[k] = e < n_tbl ? bt[b_lo + e] : 0;
  }
  // Lane i < NLD of next_v holds the physical block of the next tile's piece i, looked up one
  // tile ahead with a lane-dependent address (so it stays in a vector register and its LDS
  // read has long returned when readlane takes it).
  const int blk_lane = blk_of[lane % NLD];
  int32_t next_v = 0;
  auto fetch_next = [&](int tile) {
    const int b = ((tile * kBK) >> 4) + blk_lane;   // relative to b_lo
    next_v = b < n_tbl ? tbl[b] : 0;
  };
  auto issue = [&](int tile, const int32_t (&ph)[NLD]) {
    char* st = smem + (tile % kStages) * 2 * TILE;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      ARCKV_CHECK_WAVE(ph[i] < 0 || ph[i] >= num_blocks, ARCKV_CHECK_BLOCK);
      // wave-uniform (the wave's 1 KiB lies in one block); an entry out of range reads block 0
      const int32_t pb = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(ph[i]) >= nb32 ? 0 : ph[i]);
      const int64_t base = static_cast<int64_t>(pb) * blk_stride + head_k;
      load_lds16_s(k_pool + base, static_cast<uint32_t>(k_off[i]) * 2u, (lds_void*)(st + i * LDB + wave * 1024));
      load_lds16_s(v_pool + base, static_cast<uint32_t>(v_off[i]) * 2u, (lds_void*)(st + TILE + i * LDB + wave * 1024));
    }
  };
  // tiles issued before the table is in LDS read their entries from the global table
  auto load_tile_global = [&](int tile) {
    int32_t ph[NLD];
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int b = b_lo + ((tile * kBK) >> 4) + blk_of[i];
      ph[i] = b < nblk ? bt[b] : 0;
    }
    issue(tile, ph);
  };

  f32x16_t o[DM];
#pragma unroll
  for (int md = 0; md < DM; ++md) o[md] = f32x16_t{};
  f32x16_t sacc[2];                 // S^T of one tile: 2 blocks of 32 keys x this wave's columns
  uint32_t pw[4][4];                // P^T operands: 4 blocks of 16 keys, bf16 pairs
  float m_run = -INFINITY, l_run = 0.f;

  // ---- V phase ----------------------------------------------------------------------------
  // S^T register r of key block mb holds key t0 + 32 mb + 16 (r / 8) + 8 hg + r % 8
  auto v_phase = [&](int j, auto masked) {
    const int t0 = kv_lo + j * kBK;
    if constexpr (decltype(masked)::value) {   // diagonal or prompt-end tile
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = t0 + mb * 32 + 16 * (r >> 3) + 8 * hg + (r & 7);
          sacc[mb][r] = key > pos ? -INFINITY : sacc[mb][r];
        }
    }
    // Exponentials against the running maximum first.  Every term p = 2^(s c - m) is >= 0,
    // so a lane whose sum stays <= 2^kLazy has every term <= 2^kLazy, which is all the lazy
    // rescale has to guarantee.  Only when some lane's sum exceeds that (or on the item's
    // first tile, before any maximum is known) are the column maxima taken, O and l rescaled
    // and the exponentials computed again.
    auto exps = [&](float mu) {
      float sum = -0.f;                  // -0 + x == x for every x: the first add folds away
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int half = 0; half < 2; ++half)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const f32x2_t two = {fast_exp2(fmaf(sacc[mb][8 * half + 2 * jj], scale_log2, -mu)),
                                 fast_exp2(fmaf(sacc[mb][8 * half + 2 * jj + 1], scale_log2, -mu))};
            sum += two[0];
            sum += two[1];
            pw[2 * mb + half][jj] = __builtin_bit_cast(uint32_t, __builtin_convertvector(two, bf16x2_t));
          }
      return sum;
    };
    float lsum = 0.f;
    bool pending = true;
    if (j > 0) {                                                   // wave-uniform
      lsum = exps(m_run == -INFINITY ? 0.f : m_run);
      pending = __builtin_amdgcn_ballot_w64(!(lsum <= kLazySum)) != 0;   // also catches inf / NaN sums
    }
    if (pending) {
      float m = -INFINITY;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) m = fmaxf(m, sacc[mb][r]);
      const float mx = max_halves(m) * scale_log2;
      const float m_new = fmaxf(m_run, mx);
      const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int md = 0; md < DM; ++md) o[md] *= alpha;
      lsum = exps(m_run == -INFINITY ? 0.f : m_run);
    }
    l_run += lsum;
  };
  // keys >= L of the last tile may hold stale bytes (even NaN patterns): zero their V in LDS
  // (group 0 only, 256 threads; published by the barrier that ends the half step)
  auto zero_v_tail = [&](int tile, int t0) {
    uint16_t* vb = reinterpret_cast<uint16_t*>(smem + (tile % kStages) * 2 * TILE + TILE);
    for (int e = tid; e < kBK * D; e += kThreads / 2) {
      const int key = e & (kBK - 1), d = e / kBK;
      if (t0 + key >= L) {
        const int blk = key >> 4, kk = key & 15;
        const int h = ((kk >> 3) ^ sv(d));
        vb[(blk * BLK_BYTES + d * 32 + h * 16) / 2 + (kk & 7)] = 0;
      }
    }
  };

  // ---- M phase: operand n < 4 DM is V^T of (key block n / DM, dim block n % DM) for P.V;
  // the rest are K rows of (k-step (n - 4 DM) / 2, key block n % 2) for S = K Q^T -----------
  // with_load: this wave's 2 NLD direct loads of tile load_t are issued one every
  // N / (2 NLD) MFMAs instead of back to back: all waves issuing theirs right after a barrier
  // queue behind each other at the load unit (about 16 cycles per 1 KiB instruction).
  auto m_phase = [&](int j, auto with_s, auto with_load, int load_t) {
    constexpr bool WITH_S = decltype(with_s)::value;
    constexpr bool WITH_LOAD = decltype(with_load)::value;
    constexpr int N = WITH_S ? NOP : 4 * DM;
    const char* vb = smem + (j % kStages) * 2 * TILE + TILE;
    const char* kb = smem + ((j + 1) % kStages) * 2 * TILE;
    const int vlane = l32 * 32 + ((hg ^ sv(l32)) * 16);          // sv(md * 32 + l32) == sv(l32)
    auto op_at = [&](int n) -> bf16x8_t {
      if (n < 4 * DM) {
        const int sp = n / DM, md = n % DM;
        return *reinterpret_cast<const bf16x8_t*>(vb + sp * BLK_BYTES + md * 1024 + vlane);
      }
      const int ks = (n - 4 * DM) / 2, mb = (n - 4 * DM) % 2;
      const int r = mb * 32 + pi_row(l32);
      const int c = 2 * ks + hg;
      return *reinterpret_cast<const bf16x8_t*>(kb + r * 2 * D + ((c ^ fk<D>(r)) * 16));
    };
    const uint16_t* ld_src[2 * NLD];
    uint32_t ld_ofs[2 * NLD];
    lds_void* ld_dst[2 * NLD];
    if constexpr (WITH_LOAD) {
      char* st = smem + (load_t % kStages) * 2 * TILE;
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        const int32_t ph = __builtin_amdgcn_readlane(next_v, i);
        ARCKV_CHECK_WAVE(ph < 0 || ph >= num_blocks, ARCKV_CHECK_BLOCK);
        const int32_t pb = static_cast<uint32_t>(ph) >= nb32 ? 0 : ph;  // never used unmasked
        const int64_t base = static_cast<int64_t>(pb) * blk_stride + head_k;
        ld_src[2 * i] = k_pool + base;
        ld_ofs[2 * i] = static_cast<uint32_t>(k_off[i]) * 2u;
        ld_dst[2 * i] = (lds_void*)(st + i * LDB + wave * 1024);
        ld_src[2 * i + 1] = v_pool + base;
        ld_ofs[2 * i + 1] = static_cast<uint32_t>(v_off[i]) * 2u;
        ld_dst[2 * i + 1] = (lds_void*)(st + TILE + i * LDB + wave * 1024);
      }
      fetch_next(load_t + 1);
    }
    constexpr int LD_EVERY = N / (2 * NLD);
    bf16x8_t opv[N];
#pragma unroll
    for (int n = 0; n < PD; ++n) opv[n] = op_at(n);
#pragma unroll
    for (int n = 0; n < N; ++n) {
      if constexpr (WITH_LOAD)
        if (n % LD_EVERY == LD_EVERY / 2) load_lds16_s(ld_src[n / LD_EVERY], ld_ofs[n / LD_EVERY], ld_dst[n / LD_EVERY]);
      if (n + PD < N) opv[n + PD] = op_at(n + PD);
      if (n < 4 * DM) {
        const int sp = n / DM, md = n % DM;
        const u32x4_t w4 = {pw[sp][0], pw[sp][1], pw[sp][2], pw[sp][3]};
        o[md] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(opv[n], __builtin_bit_cast(bf16x8_t, w4), o[md], 0, 0, 0);
      } else {
        const int ks = (n - 4 * DM) / 2, mb = (n - 4 * DM) % 2;
        sacc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(opv[n], qf[ks], ks == 0 ? f32x16_t{} : sacc[mb], 0, 0, 0);
      }
    }
    // keep the operand reads PD ahead: DS reads, then one MFMA and one read at a time
    __builtin_amdgcn_sched_group_barrier(0x100, PD, 0);
#pragma unroll
    for (int n = 0; n < N - PD; ++n) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, PD, 0);
  };
  // S(0) of M(-1): K(0) Q^T only
  auto s_first = [&]() {
    const char* kb = smem;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const int r = mb * 32 + pi_row(l32);
        const int c = 2 * ks + hg;
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(kb + r * 2 * D + ((c ^ fk<D>(r)) * 16));
        sacc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], ks == 0 ? f32x16_t{} : sacc[mb], 0, 0, 0);
      }
  };

  // ---- the half-step pipeline -------------------------------------------------------------
  // wait_tile: this wave's loads of tile t are complete (the only loads that may still be in
  // flight are those of tile t + 1, if it was issued), its LDS reads have returned, then the
  // workgroup barrier publishes every wave's part of the tile.
  // A barrier orders memory operations only: pure register arithmetic could still be moved
  // across it (the exponentials of V(j) sunk next to their use in M(j), which would put both
  // phases into one half step).  These empty volatile statements consume each phase's
  // results, so the results are computed before the barrier that ends the phase.
  auto pin_v = [&]() {
#pragma unroll
    for (int sp = 0; sp < 4; ++sp)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) asm volatile("" ::"v"(pw[sp][jj]));
    asm volatile("" ::"v"(l_run), "v"(m_run));
  };
  auto pin_m = [&]() {
#pragma unroll
    for (int md = 0; md < DM; ++md) asm volatile("" ::"v"(o[md][0]));
    asm volatile("" ::"v"(sacc[0][0]), "v"(sacc[1][0]));
  };
  auto barrier_plain = [&]() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };
  auto barrier_wait = [&](int) {   // the one tile issued after the awaited one may be in flight
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(2 * NLD) : "memory");
  };
  // The table, the Q loads and tile 0 (read in half step 0): one vmcnt(0) covers them (an
  // instruction the compiler's wait insertion understands, so it adds none of its own before
  // Q is used).  Tiles 1 and 2 go out after it, to arrive while S(0) is computed: the waits
  // in the loop already leave one tile in flight beyond the one a phase reads.  The barrier
  // publishes the table without waiting for those loads.
  if (ntiles > 0) load_tile_global(0);
  __builtin_amdgcn_s_waitcnt(0x0F70);
  for (int t = 1; t < kStages - 1; ++t)
    if (t < ntiles) load_tile_global(t);
#pragma unroll
  for (int k = 0; k < kTblPer; ++k) {
    const int e = tid + k * kThreads;
    if (e < n_tbl) tbl[e] = tbl_v[k];
  }
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  fetch_next(kStages - 1);
  if (ntiles > 0) {
    const int e_tile = (L - kv_lo + kBK - 1) / kBK - 1;   // the tile holding key L - 1
    if (grp == 1) barrier_plain();                      // half step 0: group 1 waits
    s_first();                                           // M(-1)
    pin_m();
    if (grp == 1) barrier_wait(1); else barrier_plain(); // group 1's M(-1) ends half step 1
    auto step = [&](int j, auto masked) {
      // ---- V(j): half step 2j + 1 (group 0) / 2j + 2 (group 1)
      if constexpr (decltype(masked)::value)
        if (grp == 0 && j == e_tile) zero_v_tail(j, kv_lo + j * kBK);
      v_phase(j, masked);
      pin_v();
      if (grp == 0) barrier_wait(j + 1); else barrier_plain();
      // ---- M(j): half step 2j + 2 (group 0) / 2j + 3 (group 1)
      // Every M phase issues one tile's loads, so that the waits count the same loads in every
      // step: past the key range (j + 3 >= ntiles) the loads fetch block 0 into the stage of
      // tile j - 1, which no wave reads any more.  On the last tile S(j+1) multiplies stale LDS;
      // it is never used.
      m_phase(j, std::true_type{}, std::true_type{}, j + 3);
      pin_m();
      if (grp == 0) barrier_plain();
      else if (j + 1 < ntiles) barrier_wait(j + 2);
    };
    // tiles that need the causal / prompt-end mask form a suffix of the key range
    auto tile_masked = [&](int t) {
      const int t0 = kv_lo + t * kBK;
      return (t0 + kBK - 1 > wg_min_pos) || (t0 + kBK > L);
    };
    int n_plain = ntiles;
    {
      int lo = 0, hi = ntiles;  // first masked tile, else ntiles
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (tile_masked(mid)) hi = mid; else lo = mid + 1;
      }
      n_plain = lo;
    }
    int j = 0;
    for (; j < n_plain; ++j) step(j, std::false_type{});
    for (; j < ntiles; ++j) step(j, std::true_type{});
    // no load may still write this workgroup's LDS when it ends
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  // ---- epilogue: O^T register r of block md holds dim 32 md + 8 (r / 4) + 4 hg + r % 4 ------
  const float lt = sum_halves(l_run);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  const float lse = lt > 0.f ? m_run + __log2f(lt) : -INFINITY;
#pragma unroll
  for (int md = 0; md < DM; ++md) o[md] *= inv;
  if (!cval) return;
  if (w.slot < 0) {
    uint16_t* dst = out + (static_cast<int64_t>(q0 + tok) * hq + w.kvh * G + g) * D;
#pragma unroll
    for (int md = 0; md < DM; ++md)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        f32x4_t v;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) v[jj] = o[md][4 * r4 + jj];
        *reinterpret_cast<bf16x4_t*>(dst + md * 32 + 8 * r4 + 4 * hg) = __builtin_convertvector(v, bf16x4_t);
      }
    return;
  }
  if (w.slot >= ws_slots) return;
  const int local = wave * 32 + l32;
  float* po = ws_o + (static_cast<int64_t>(w.slot) * kCols + local) * D;
#pragma unroll
  for (int md = 0; md < DM; ++md)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      f32x4_t v;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) v[jj] = o[md][4 * r4 + jj];
      *reinterpret_cast<f32x4_t*>(po + md * 32 + 8 * r4 + 4 * hg) = v;
    }
  if (hg == 0) ws_lse[static_cast<int64_t>(w.slot) * kCols + local] = lse;
}

// Merges the key-range splits of one query tile: o = sum_s 2^(lse_s - M) O_s / sum_s 2^(lse_s - M)
// with M = max_s lse_s, per column.  Grid: (combine items, tile_cols / kCombineCols); a block
// takes kCombineCols columns.  The first pieces' partial O (kCombinePre of them) and the lse
// of up to kCombineMaxSplits pieces are all requested at once, since the partials do not
// depend on the weights: one memory round trip instead of one for the lse, one for the
// weights and one for the partials.  The lse then turn into per-column weights in LDS, the
// preloaded partials are summed, and any further pieces stream with several loads in flight.
// The sums run over the pieces in order, as a plain loop would.
constexpr int kCombineThreads = 256;
constexpr int kCombineCols = 32;
constexpr int kCombineMaxSplits = 64;  // pieces weighted in LDS at a time
constexpr int kCombinePre = 4;         // pieces loaded before their weights are known

template <int D>
__global__ __launch_bounds__(kCombineThreads) void attn_combine_kernel(
    uint16_t* __restrict__ out, const Work* __restrict__ items, const int32_t* __restrict__ cu_q,
    int n_reqs, int64_t n_q, int hq, int G, int tile_cols, const float* __restrict__ ws_o,
    const float* __restrict__ ws_lse, int64_t ws_slots) {
  __shared__ float wt[kCombineMaxSplits][kCombineCols];  // lse of a batch of pieces, then weights
  __shared__ float mx[kCombineCols], inv[kCombineCols];
  const Work w = items[blockIdx.x];  // {req, kvh, col_start, slot0, n_splits}
  const int slot0 = w.kv_start, ns = w.kv_end;
  const bool bad = w.req < 0 || w.req >= n_reqs || w.kvh < 0 || (w.kvh + 1) * G > hq || w.col_start < 0 ||
                  slot0 < 0 || ns < 1 || slot0 + ns > ws_slots;
  ARCKV_CHECK_WAVE(bad, ARCKV_CHECK_WORK);
  if (bad) return;
  const int q0 = cu_q[w.req];
  const int ncols = (cu_q[w.req + 1] - q0) * G;
  const int c0 = blockIdx.y * kCombineCols;  // first local column of this block
  if (w.col_start + c0 >= ncols) return;     // (uniform) no column of the request here: decode
                                             // tiles fill 4 to 8 of their 128 columns
  constexpr int D4 = D / 4;
  constexpr int PER = kCombineCols * D4 / kCombineThreads;  // float4 slices per thread
  static_assert(PER * kCombineThreads == kCombineCols * D4, "combine split");
  const int tid = threadIdx.x;
  // slice k of this thread: block column (tid + k * threads) / D4, dims 4 * ((tid + k * threads) % D4)
  auto slice = [&](int s, int k) -> f32x4_t {
    const int e = tid + k * kCombineThreads;
    const float* po = ws_o + (static_cast<int64_t>(slot0 + s) * tile_cols + c0) * D;
    return *reinterpret_cast<const f32x4_t*>(po + static_cast<int64_t>(e / D4) * D + 4 * (e % D4));
  };
  f32x4_t pre[kCombinePre][PER];
#pragma unroll
  for (int s = 0; s < kCombinePre; ++s)
#pragma unroll
    for (int k = 0; k < PER; ++k) pre[s][k] = s < ns ? slice(s, k) : f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int nb0 = min(kCombineMaxSplits, ns);
  for (int e = tid; e < nb0 * kCombineCols; e += kCombineThreads) {
    const int s = e / kCombineCols, c = e % kCombineCols;
    wt[s][c] = ws_lse[static_cast<int64_t>(slot0 + s) * tile_cols + c0 + c];
  }
  __syncthreads();
  // per column: the maximum over all pieces, then the first batch's weights and their sum
  float wsum_part = 0.f;
  if (tid < kCombineCols) {
    float m = -INFINITY;
    for (int s = 0; s < nb0; ++s) m = fmaxf(m, wt[s][tid]);
    for (int s = nb0; s < ns; ++s)
      m = fmaxf(m, ws_lse[static_cast<int64_t>(slot0 + s) * tile_cols + c0 + tid]);
    mx[tid] = m;
    for (int s = 0; s < nb0; ++s) {
      const float l = wt[s][tid];
      const float x = l == -INFINITY ? 0.f : fast_exp2(l - m);
      wt[s][tid] = x;
      wsum_part += x;
    }
  }
  __syncthreads();
  f32x4_t acc[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    acc[k] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < kCombinePre; ++s)
      if (s < ns) acc[k] += wt[s][(tid + k * kCombineThreads) / D4] * pre[s][k];
  }
#pragma unroll 4
  for (int s = kCombinePre; s < nb0; ++s) {
    f32x4_t v[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) v[k] = slice(s, k);
#pragma unroll
    for (int k = 0; k < PER; ++k) acc[k] += wt[s][(tid + k * kCombineThreads) / D4] * v[k];
  }
  // more than kCombineMaxSplits pieces: further batches, weighted with the same maximum
  for (int sb = nb0; sb < ns; sb += kCombineMaxSplits) {
    const int nb = min(kCombineMaxSplits, ns - sb);
    __syncthreads();  // every thread is done with the previous batch's weights
    for (int e = tid; e < nb * kCombineCols; e += kCombineThreads) {
      const int s = e / kCombineCols, c = e % kCombineCols;
      const float l = ws_lse[static_cast<int64_t>(slot0 + sb + s) * tile_cols + c0 + c];
      wt[s][c] = l == -INFINITY ? 0.f : fast_exp2(l - mx[c]);
    }
    __syncthreads();
    if (tid < kCombineCols)
      for (int s = 0; s < nb; ++s) wsum_part += wt[s][tid];
#pragma unroll 4
    for (int s = 0; s < nb; ++s) {
      f32x4_t v[PER];
#pragma unroll
      for (int k = 0; k < PER; ++k) v[k] = slice(sb + s, k);
#pragma unroll
      for (int k = 0; k < PER; ++k) acc[k] += wt[s][(tid + k * kCombineThreads) / D4] * v[k];
    }
  }
  if (tid < kCombineCols) inv[tid] = wsum_part > 0.f ? 1.f / wsum_part : 0.f;
  __syncthreads();
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = tid + k * kCombineThreads;
    const int local = c0 + e / D4, d4 = e % D4;
    const int col = w.col_start + local;
    if (local >= tile_cols || col >= ncols) continue;
    const int tok = col / G, g = col % G;
    if (q0 + tok >= n_q) continue;
    const bf16x4_t b = __builtin_convertvector(acc[k] * inv[e / D4], bf16x4_t);
    *reinterpret_cast<bf16x4_t*>(out + (static_cast<int64_t>(q0 + tok) * hq + w.kvh * G + g) * D + 4 * d4) = b;
  }
}

constexpr int kWideNB = 1;  // 32-column MFMA blocks per wave on wide tiles
constexpr int kWideWaves = arckv::kWideCols / (32 * kWideNB);
static_assert(kWideWaves * 32 * kWideNB == arckv::kWideCols, "wide tile width");


}  // namespace

namespace {

int32_t prefill_attention(const void* k_pool, const void* v_pool, const void* q, void* out,
                          const int32_t* block_tables, int32_t bt_stride, const int32_t* cu_q,
                          const int32_t* seq_lens, int32_t n_reqs, int64_t n_q, int64_t num_blocks,
                          const int32_t* work, int64_t n_work, int64_t n_combine, int32_t tile_cols,
                          int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float scale,
                          void* workspace, int64_t ws_bytes, void* stream, hipEvent_t ev_begin,
                          hipEvent_t ev_mid, hipEvent_t ev_end) {
  if (num_q_heads < 1 || num_kv_heads < 1 || num_q_heads % num_kv_heads != 0 || n_reqs < 0 ||
      n_q < 0 || num_blocks < 0 || n_work < 0 || n_combine < 0 || ws_bytes < 0 || bt_stride < 0 ||
      !std::isfinite(scale) || scale <= 0.f)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: bad sizes or scale");
  const int G = num_q_heads / num_kv_heads;
  if (head_dim != 64 && head_dim != 128)
    return arckv::fail(ARCKV_EUNSUPPORTED, "prefill_attention: head_dim %d not in {64,128}", head_dim);
  if (G != 1 && G != 2 && G != 4 && G != 5 && G != 8)
    return arckv::fail(ARCKV_EUNSUPPORTED, "prefill_attention: group size %d not in {1,2,4,5,8}", G);
  if (tile_cols != arckv::kWideCols && tile_cols != arckv::kNarrowCols)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: tile_cols %d is not a planned width", tile_cols);
  if (tile_cols == arckv::kNarrowCols && n_work % arckv::kListItems != 0)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: a narrow plan has lists of %d items; n_work %lld",
                       arckv::kListItems, (long long)n_work);
  if (n_work == 0 && n_combine == 0) {  // nothing to run; the events still mark the stream
    for (hipEvent_t ev : {ev_begin, ev_mid, ev_end})
      if (ev != nullptr && hipEventRecord(ev, static_cast<hipStream_t>(stream)) != hipSuccess)
        return arckv::fail(ARCKV_EDEVICE, "prefill_attention: event record failed");
    return ARCKV_OK;
  }
  if (k_pool == nullptr || v_pool == nullptr || q == nullptr || out == nullptr ||
      block_tables == nullptr || cu_q == nullptr || seq_lens == nullptr || work == nullptr)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: NULL pointer");
  if (n_work > INT32_MAX || n_combine > INT32_MAX)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: too many work items");
  const int64_t slot_bytes = static_cast<int64_t>(tile_cols) * (head_dim + 1) * 4;
  const int64_t ws_slots = workspace != nullptr ? ws_bytes / slot_bytes : 0;
  if (n_combine > 0 && ws_slots == 0)
    return arckv::fail(ARCKV_EINVAL, "prefill_attention: split plan needs a workspace");
  float* ws_o = static_cast<float*>(workspace);
  float* ws_lse = ws_o == nullptr ? nullptr : ws_o + ws_slots * tile_cols * head_dim;
  auto* st = static_cast<hipStream_t>(stream);
  auto* kp = static_cast<const uint16_t*>(k_pool);
  auto* vp = static_cast<const uint16_t*>(v_pool);
  auto* qp = static_cast<const uint16_t*>(q);
  auto* op = static_cast<uint16_t*>(out);
  auto* wk = reinterpret_cast<const Work*>(work);
  const float scale_log2 = scale * 1.4426950408889634f;

  auto record = [&](hipEvent_t ev) -> bool {
    return ev == nullptr || hipEventRecord(ev, st) == hipSuccess;
  };
  if (!record(ev_begin)) return arckv::fail(ARCKV_EDEVICE, "prefill_attention: event record failed");
  if (n_work > 0) {
    const dim3 grid(static_cast<unsigned>(n_work));
    const dim3 list_grid(static_cast<unsigned>(n_work / arckv::kListItems));
#define ARCKV_LAUNCH(DD, GG)                                                                   \
  do {                                                                                         \
    if (tile_cols == arckv::kWideCols)                                                         \
      hipLaunchKernelGGL((prefill_attn_pp_kernel<DD, GG>), grid, dim3(512), 0, st, kp, vp, qp, op, \
                         block_tables, bt_stride, cu_q, seq_lens, n_reqs, wk, n_q, num_blocks, \
                         num_q_heads, num_kv_heads, scale_log2, ws_o, ws_lse, ws_slots);      \
    else                                                                                       \
      hipLaunchKernelGGL((prefill_attn_list_kernel<DD, GG>), list_grid, dim3(512), 0, st, kp, vp, qp, \
                         op, block_tables, bt_stride, cu_q, seq_lens, n_reqs, wk, n_q, num_blocks, \
                         num_q_heads, num_kv_heads, scale_log2, ws_o, ws_lse, ws_slots);      \
  } while (0)
    if (head_dim == 64) {
      switch (G) {
        case 1: ARCKV_LAUNCH(64, 1); break;
        case 2: ARCKV_LAUNCH(64, 2); break;
        case 4: ARCKV_LAUNCH(64, 4); break;
        case 5: ARCKV_LAUNCH(64, 5); break;
        default: ARCKV_LAUNCH(64, 8); break;
      }
    } else {
      switch (G) {
        case 1: ARCKV_LAUNCH(128, 1); break;
        case 2: ARCKV_LAUNCH(128, 2); break;
        case 4: ARCKV_LAUNCH(128, 4); break;
        case 5: ARCKV_LAUNCH(128, 5); break;
        default: ARCKV_LAUNCH(128, 8); break;
      }
    }
#undef ARCKV_LAUNCH
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
      return arckv::fail(ARCKV_EDEVICE, "prefill_attention: %s", hipGetErrorString(e));
  }
  if (!record(ev_mid)) return arckv::fail(ARCKV_EDEVICE, "prefill_attention: event record failed");
  if (n_combine > 0) {
    const dim3 grid(static_cast<unsigned>(n_combine), static_cast<unsigned>(tile_cols / kCombineCols));
    const Work* items = wk + n_work;
    if (head_dim == 64)
      hipLaunchKernelGGL(attn_combine_kernel<64>, grid, dim3(kCombineThreads), 0, st, op, items,
                         cu_q, n_reqs, n_q, num_q_heads, G, tile_cols, ws_o, ws_lse, ws_slots);
    else
      hipLaunchKernelGGL(attn_combine_kernel<128>, grid, dim3(kCombineThreads), 0, st, op, items,
                         cu_q, n_reqs, n_q, num_q_heads, G, tile_cols, ws_o, ws_lse, ws_slots);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
      return arckv::fail(ARCKV_EDEVICE, "attn_combine: %s", hipGetErrorString(e));
  }
  if (!record(ev_end)) return arckv::fail(ARCKV_EDEVICE, "prefill_attention: event record failed");
  return ARCKV_OK;
}

}  // namespace

ARCKV_DEFINE_CHECK_READER(read_attention_checks)

extern "C" int32_t arckv_device_checks(int32_t* bits, int64_t* count, int32_t reset, void* stream) {
  if (bits == nullptr || count == nullptr) return arckv::fail(ARCKV_EINVAL, "device_checks: NULL output");
  uint32_t b1 = 0, c1 = 0, b2 = 0, c2 = 0;
  int32_t st = arckv::read_scatter_checks(stream, reset != 0, &b1, &c1);
  if (st != ARCKV_OK) return st;
  st = arckv::read_attention_checks(stream, reset != 0, &b2, &c2);
  if (st != ARCKV_OK) return st;
  *bits = static_cast<int32_t>(b1 | b2);
  *count = static_cast<int64_t>(c1) + c2;
  return ARCKV_OK;
}

extern "C" int32_t arckv_prefill_attention(const void* k_pool, const void* v_pool, const void* q,
                                           void* out, const int32_t* block_tables,
                                           int32_t bt_stride, const int32_t* cu_q,
                                           const int32_t* seq_lens, int32_t n_reqs, int64_t n_q,
                                           int64_t num_blocks, const int32_t* work,
                                           int64_t n_work, int64_t n_combine, int32_t tile_cols,
                                           int32_t num_q_heads, int32_t num_kv_heads,
                                           int32_t head_dim, float scale, void* workspace,
                                           int64_t ws_bytes, void* stream) {
  return prefill_attention(k_pool, v_pool, q, out, block_tables, bt_stride, cu_q, seq_lens, n_reqs,
                           n_q, num_blocks, work, n_work, n_combine, tile_cols, num_q_heads,
                           num_kv_heads, head_dim, scale, workspace, ws_bytes, stream, nullptr,
                           nullptr, nullptr);
}

extern "C" int32_t arckv_prefill_attention_timed(
    const void* k_pool, const void* v_pool, const void* q, void* out, const int32_t* block_tables,
    int32_t bt_stride, const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs, int64_t n_q,
    int64_t num_blocks, const int32_t* work, int64_t n_work, int64_t n_combine, int32_t tile_cols,
    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float scale, void* workspace,
    int64_t ws_bytes, void* stream, void* ev_begin, void* ev_mid, void* ev_end) {
  return prefill_attention(k_pool, v_pool, q, out, block_tables, bt_stride, cu_q, seq_lens, n_reqs,
                           n_q, num_blocks, work, n_work, n_combine, tile_cols, num_q_heads,
                           num_kv_heads, head_dim, scale, workspace, ws_bytes, stream,
                           static_cast<hipEvent_t>(ev_begin), static_cast<hipEvent_t>(ev_mid),
                           static_cast<hipEvent_t>(ev_end));
}

// ---- the entry point that allocates nothing -------------------------------------------------
// The split pieces' partials go to a file-scope device array instead of a caller workspace.
// Each device holds its own copy (for as long as the process runs); its address is looked up
// once per device with hipGetSymbolAddress, with that device current, and kept: in host code
// the array's name is only a host-side stand-in, never a device address.  Every call on one
// device shares that device's copy, so calls that overlap in time on one device race.  Nothing
// in it needs clearing: every split piece writes its own slot before the combine reads it.
namespace {

constexpr int64_t kStaticScratchBytes = ARCKV_NOALLOC_MAX_WS_BYTES;
static_assert(kStaticScratchBytes % 256 == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Address of `scratch` on the device the stream belongs to (the current device for the null
// stream), looked up on the first call for that device.
int32_t device_scratch(hipStream_t st, void** ptr) {
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess)
    return arckv::fail(ARCKV_EDEVICE, "prefill_attention_noalloc: hipGetDevice failed");
  int dev = cur;
  if (st != nullptr && hipStreamGetDevice(st, &dev) != hipSuccess)
    return arckv::fail(ARCKV_EDEVICE, "prefill_attention_noalloc: hipStreamGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices)
    return arckv::fail(ARCKV_EUNSUPPORTED, "prefill_attention_noalloc: device %d >= %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess)
      return arckv::fail(ARCKV_EDEVICE, "prefill_attention_noalloc: hipSetDevice(%d) failed", dev);
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) (void)hipSetDevice(cur);
    if (e != hipSuccess || p == nullptr)
      return arckv::fail(ARCKV_EDEVICE, "prefill_attention_noalloc: hipGetSymbolAddress: %s",
                         hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return ARCKV_OK;
}

}  // namespace

extern "C" int32_t arckv_prefill_attention_noalloc(
    const void* k_pool, const void* v_pool, const void* q, void* out, const int32_t* block_tables,
    int32_t bt_stride, const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs, int64_t n_q,
    int64_t num_blocks, const int32_t* work, int64_t n_work, int64_t n_combine, int32_t tile_cols,
    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim, float scale, int64_t ws_bytes,
    void* stream) {
  if (ws_bytes < 0 || ws_bytes > kStaticScratchBytes)
    return arckv::fail(ARCKV_ENOSPC,
                       "prefill_attention_noalloc: the plan needs %lld bytes of workspace; the static "
                       "scratch holds %lld",
                       static_cast<long long>(ws_bytes), static_cast<long long>(kStaticScratchBytes));
  void* ws = nullptr;
  if (ws_bytes > 0) {
    const int32_t rc = device_scratch(static_cast<hipStream_t>(stream), &ws);
    if (rc != ARCKV_OK) return rc;
  }
  return prefill_attention(k_pool, v_pool, q, out, block_tables, bt_stride, cu_q, seq_lens, n_reqs,
                           n_q, num_blocks, work, n_work, n_combine, tile_cols, num_q_heads,
                           num_kv_heads, head_dim, scale, ws, ws_bytes, stream, nullptr, nullptr,
                           nullptr);
}
