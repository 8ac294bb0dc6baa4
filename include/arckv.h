/*
 * arckv.h -- C ABI of libarckv: prefix-cached paged prefill attention with an
 * ARC (or LRU) KV-block cache, for AMD Instinct MI355X (gfx950).
 *
 * The library covers the path whose work a higher prefix-cache hit rate cuts:
 * for every request of a batch, the computed (uncached) suffix tokens attend,
 * through a block table, to the KV blocks the cache kept and, causally, to
 * themselves; their new K/V are scattered into physical blocks first.  The
 * host side decides hits and evictions with ARC over chained block hashes.
 * Paper: "Recency/Frequency Adaptive KV Caching for Large Language Model
 * Serving" -- Sec. 2 (prefill, prefix caching, paged attention with
 * fixed-size KV blocks), Sec. 3 and Fig. 2 (ARC evictor: T1/T2/B1/B2 and the
 * adaptive target p, block-level decisions), Sec. 4 (16-token blocks, batched
 * offline prefill).
 *
 * Conventions
 *  - Every call returns an int32 status: ARCKV_OK (0) or a negative ARCKV_E*
 *    code; arckv_last_error() then returns a thread-local message.  No C++
 *    exception crosses this boundary.
 *  - Host objects are opaque and owned by the library (create/destroy pairs).
 *  - Device memory is always owned by the caller.  The library never
 *    allocates or frees device memory itself; device pointers are borrowed
 *    until the work queued on the given stream has completed.  The library
 *    links no other GPU library: every device step is a kernel of its own.
 *  - Device calls enqueue asynchronously on the caller's HIP stream (passed as
 *    void*, NULL = the null stream).  Argument checks are synchronous; a launch
 *    failure returns ARCKV_EDEVICE.  Nothing synchronises implicitly.
 *  - bf16 values are passed as 16-bit patterns; arrays are row-major, C order.
 *  - Block size is 16 tokens.  Pool layout version 1 (ARCKV_LAYOUT_V1):
 *      K pool: [num_blocks][num_kv_heads][16][head_dim]   (token-major block)
 *      V pool: [num_blocks][num_kv_heads][head_dim][16]   (dim-major block)
 *    Token j of a request lives in block table[j / 16] at offset j % 16; its
 *    slot is table[j / 16] * 16 + j % 16.
 */
#ifndef ARCKV_H
#define ARCKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ARCKV_BLOCK_TOKENS 16
#define ARCKV_LAYOUT_V1 1
/* largest planned workspace arckv_prefill_attention_noalloc accepts (its static scratch) */
#define ARCKV_NOALLOC_MAX_WS_BYTES (64LL << 20)

/* status codes */
#define ARCKV_OK 0
#define ARCKV_EINVAL (-1)       /* malformed arguments                                  */
#define ARCKV_ENOSPC (-2)       /* batch does not fit: capacity, scratch or buffer caps */
#define ARCKV_EDEVICE (-3)      /* a HIP call failed (message holds the HIP error)      */
#define ARCKV_ESTATE (-4)       /* call order violated (plan/release)                   */
#define ARCKV_EUNSUPPORTED (-5) /* head_dim / group size / block size not supported     */
#define ARCKV_ECOLLISION (-6)   /* two different blocks share one identity (check mode)  */

/* policies and reference order */
#define ARCKV_POLICY_ARC 0
#define ARCKV_POLICY_LRU 1
#define ARCKV_POLICY_DBL 2 /* ARC with p fixed at c/2 (Sec. 4's static two-queue variant) */
#define ARCKV_POLICY_FRC 3 /* ARC with p fixed at cfg.frc_p (the fixed-target form FRC_p)  */
#define ARCKV_REF_TAIL_FIRST 0
#define ARCKV_REF_HEAD_FIRST 1

/* decision-log case codes (ARC cases I..IV of the published algorithm, plus LRU) */
#define ARCKV_CASE_I 0          /* hit in T1 or T2 -> MRU of T2                      */
#define ARCKV_CASE_II 1         /* ghost hit in B1: p grows, REPLACE, -> T2           */
#define ARCKV_CASE_III 2        /* ghost hit in B2: p shrinks, REPLACE, -> T2         */
#define ARCKV_CASE_IVA 3        /* new, |T1|+|B1| = c, |T1| < c: drop B1 LRU, REPLACE */
#define ARCKV_CASE_IVA_T1DEL 4  /* new, |T1| = c: drop the T1 LRU page (no ghost)     */
#define ARCKV_CASE_IVB 5        /* new, |T1|+|B1| < c (REPLACE once the cache is full) */
#define ARCKV_CASE_LRU_HIT 6
#define ARCKV_CASE_LRU_MISS 7
/* list tags used in the log and in snapshots */
#define ARCKV_LIST_NONE 0
#define ARCKV_LIST_T1 1
#define ARCKV_LIST_T2 2
#define ARCKV_LIST_B1 3
#define ARCKV_LIST_B2 4

/* Device checks (a debug build: paper_2606_21238_amd.build with checked=True writes
 * lib/libarckv_checked.so, its kernels compiled with ARCKV_DEVICE_CHECKS).  Where a kernel
 * clamps or skips an out-of-range index it also records the kind, per device:
 *   ARCKV_CHECK_SLOT   a KV scatter slot outside [0, 16 num_blocks) (the token is skipped);
 *   ARCKV_CHECK_BLOCK  an attention block-table entry outside [0, num_blocks) among the blocks
 *                      of a request (block 0 is read in its place);
 *   ARCKV_CHECK_WORK   an attention or combine work item naming no request, KV head or
 *                      column of the batch (skipped; the idle items of a plan are not this).
 * arckv_device_checks waits for `stream`, stores the OR of the kinds recorded on the current
 * device since the last reset and the number of records (a bad index may be recorded by
 * several waves), and clears them when reset != 0 (not for use under graph capture).  In a
 * build without device checks it returns EUNSUPPORTED; nothing in the kernels traps. */
#define ARCKV_CHECK_SLOT 1
#define ARCKV_CHECK_BLOCK 2
#define ARCKV_CHECK_WORK 4
int32_t arckv_device_checks(int32_t* bits, int64_t* count, int32_t reset, void* stream);

/* Thread-local message describing the last failing call on this thread. */
const char* arckv_last_error(void);
/* Library ABI version (the pool layout version is ARCKV_LAYOUT_V1). */
int32_t arckv_version(void);

/* ---------------------------------------------------------------------------------------
 * Block hashing (host).  Block-level identity of cached KV (Sec. 3, last paragraph) under
 * prefix caching (Sec. 2): h_i = FNV-1a-64(le64(h_{i-1}) || le32 token ids of block i),
 * h_{-1} = root, for every full 16-token block; a trailing partial block is not hashed.
 * tokens: n_tokens int32 ids (host).  out: capacity out_cap (host, caller-owned).
 * *n_full receives n_tokens / 16.  ENOSPC if out_cap < n_tokens / 16; EINVAL on NULL /
 * negative sizes.
 * ------------------------------------------------------------------------------------- */
int32_t arckv_hash_blocks(const int32_t* tokens, int64_t n_tokens, uint64_t root,
                          uint64_t* out, int64_t out_cap, int64_t* n_full);
/* The same for n_seqs sequences at once (several chains advance together, which hides the
 * serial multiply latency).  tokens[r]: n_tokens[r] ids.  out: all identities, sequence after
 * sequence; offsets (n_seqs + 1 entries, host) receives where each sequence's run starts.
 * ENOSPC if the total exceeds out_cap (offsets are still filled). */
int32_t arckv_hash_blocks_batch(const int32_t* const* tokens, const int64_t* n_tokens,
                                int32_t n_seqs, uint64_t root, uint64_t* out, int64_t out_cap,
                                int64_t* offsets);

/* Block digests for collision checks: a second chained 64-bit value per full block, from a
 * different function than the identity (splitmix64's finaliser, Steele, Lea and Flood 2014,
 * applied per token): d_i = F(d_{i-1}, tokens of block i), d_{-1} = F0(root).  Two blocks
 * with the same identity but different token prefixes have equal digests only by a second,
 * independent accident.  Same arguments and errors as arckv_hash_blocks.  The cache keeps
 * them when created with check_blocks (see arckv_plan_batch). */
int32_t arckv_digest_blocks(const int32_t* tokens, int64_t n_tokens, uint64_t root,
                            uint64_t* out, int64_t out_cap, int64_t* n_full);

/* TEST ONLY.  Every identity the library computes from now on (arckv_hash_blocks, _batch,
 * arckv_prepare_batch) is ANDed with mask, process-wide; the chains themselves run
 * unmasked.  A narrow mask forces identity collisions, which lets tests exercise the
 * check mode.  ~0 (the default) restores normal identities.  *previous (may be NULL)
 * receives the mask in force before the call.  Not for serving. */
int32_t arckv_test_set_hash_mask(uint64_t mask, uint64_t* previous);

/* ---------------------------------------------------------------------------------------
 * Block cache: ARC(c) or LRU over block identities, with physical placement (host).
 * ARC per Sec. 3 / Fig. 2 (resident T1 "seen once", T2 "seen again", ghost lists B1/B2,
 * adaptive target p for |T1|; ghost hits steer p), with the published case rules and
 * real-valued p in IEEE binary64.  Pages used by the batch in flight are pinned: a victim
 * is the LRU-most unpinned page of the list the rule selects, else of the other list (it
 * then goes to the ghost list of the list it left).  A new page takes the physical block
 * of the page its reference evicted, else the head of a FIFO free list.
 * DBL (Sec. 4: a fixed 1:1 split between the recency and the frequency queue) runs the same
 * rules with p held at c/2: ghost hits move the page and call REPLACE but do not steer p.
 * FRC holds p at any given value in [0, c] the same way (DBL is FRC at c/2).
 * A page is "born" in a batch when a reference of that batch creates it (a miss) or brings
 * it back from a ghost list; with no_intra_batch_reuse, the prefix lookup of a request stops
 * at the first such page (it is then referenced as usual, an orphan whose KV is rewritten).
 * Length-aware victims (Sec. 6 proposes weighing prompt length beside recency and
 * frequency): with victim_window W > 1, wherever a policy evicts from a resident list
 * (REPLACE, ARC's IV-A T1 drop, LRU), it takes, among the W least recently used unpinned
 * pages of that list, the one at the greatest depth (block index in its prompt; ties: the
 * less recent one).  The list, the ghost bookkeeping and p are unchanged.  Losing a block at
 * depth k costs the next request on its chain the recompute of blocks k onwards, so deeper
 * blocks are the cheaper losses.
 * ------------------------------------------------------------------------------------- */
typedef struct arckv_cache arckv_cache;

typedef struct {
  int32_t policy;                    /* ARCKV_POLICY_ARC, _LRU, _DBL or _FRC             */
  int32_t ref_order;                 /* ARCKV_REF_TAIL_FIRST (default) or HEAD_FIRST     */
  int64_t capacity_blocks;           /* c >= 1: cacheable pages                          */
  int64_t num_phys_blocks;           /* pool size; >= capacity_blocks + scratch_blocks   */
  int64_t scratch_blocks;            /* blocks for partial last blocks of requests       */
  const int32_t* initial_free_order; /* permutation of [0, num_phys_blocks) or NULL for  */
                                     /* ascending; the first num_phys - scratch entries  */
                                     /* are the page free list, the rest the scratch FIFO */
  int32_t victim_window;             /* W in [1, 4096] (0 = 1): length-aware victims, see */
                                     /* below; 1 = the LRU-most unpinned page            */
  int32_t no_intra_batch_reuse;      /* 0 (default): a request may reuse blocks an earlier */
                                     /* request of its batch created; 1: its prefix stops */
                                     /* at such a block (engines that cache a block only  */
                                     /* once its step has run)                            */
  double frc_p;                      /* ARCKV_POLICY_FRC: the fixed target p, in [0, c]   */
  int32_t check_blocks;              /* 0 (default) or 1: resident pages keep each block's */
                                     /* digest and every plan verifies digests (below)     */
} arckv_cache_cfg;

/* Creates a cache (host memory only).  EINVAL on a bad configuration. */
int32_t arckv_cache_create(const arckv_cache_cfg* cfg, arckv_cache** out);
int32_t arckv_cache_destroy(arckv_cache* cache);

/* One request of a batch: its chained hashes (n_full = n_tokens / 16) and length, and
 * optionally its block digests (arckv_digest_blocks, n_full of them; NULL = unchecked). */
typedef struct {
  const uint64_t* hashes;
  int64_t n_full;
  int64_t n_tokens;
  const uint64_t* digests;
} arckv_req;

/* Caller-allocated host output arrays of arckv_plan_batch, with their capacities. */
typedef struct {
  int32_t* block_tables;   /* [n_reqs][bt_stride]: physical block of every logical block */
                           /* (full and partial), -1 padded                              */
  int32_t bt_stride;       /* >= max over requests of ceil(n_tokens / 16)                */
  int32_t* cu_q;           /* [n_reqs + 1]: prefix sums of computed tokens S             */
  int32_t* seq_lens;       /* [n_reqs]: prompt length L                                   */
  int32_t* prefix_lens;    /* [n_reqs]: cached prefix P = 16 k (L - S)                    */
  int32_t* hit_blocks;     /* [n_reqs]: k, the leading resident blocks reused             */
  int32_t* slot_mapping;   /* [slot_cap]: slot of every computed token, request order    */
  int64_t slot_cap;
  /* filled by the call */
  int64_t n_slots;         /* sum of S                                                    */
  int32_t max_q_len;       /* max S                                                       */
  int32_t max_seq_len;     /* max L                                                       */
} arckv_plan;

/* Number of consecutive requests (from the start of n_tokens[0..n_avail)) that form the next
 * batch: at most max_batch, while the sum of full blocks stays <= capacity and partial last
 * blocks <= scratch.  *n_take = 0 with ENOSPC if the first request alone does not fit. */
int32_t arckv_next_batch(const int64_t* n_tokens, int32_t n_avail, int32_t max_batch,
                         int64_t capacity, int64_t scratch, int32_t* n_take);

/* Plans one batch, requests in order (Sec. 2 prefix reuse; Sec. 3 miss handling):
 *  1. k = leading full blocks resident; if 16 k == L then k -= 1 (one block recomputed);
 *  2. pin the k prefix pages; 3. reference every full block once, tail first, and pin it;
 *  4. a partial last block takes a scratch block; 5. fill table row, cu_q, lengths and the
 *  slots of tokens [P, L).  A later request may hit blocks an earlier one created.
 * ESTATE if a batch is in flight; ENOSPC if the batch needs more than c full blocks, more
 * scratch blocks than free, or outputs exceed their capacities (state is then unchanged);
 * EINVAL on inconsistent requests.
 * Check mode (cfg.check_blocks = 1), for the requests that carry digests: before any state
 * changes, every block whose identity is resident must carry the digest stored with that page
 * (when one is stored), and blocks of the batch that share an identity must share the digest;
 * otherwise ECOLLISION (message: request, block, identity) and nothing changes.  Every page
 * a checked request references then stores its digest.  Without check mode a collision goes
 * unnoticed: the page's KV would be reused for different tokens. */
int32_t arckv_plan_batch(arckv_cache* cache, const arckv_req* reqs, int32_t n_reqs,
                         arckv_plan* plan);

/* Ends the batch in flight: unpins its pages, returns its scratch blocks (FIFO tail). */
int32_t arckv_release_batch(arckv_cache* cache);

typedef struct {
  int64_t t1, t2, b1, b2;   /* list sizes (LRU policy: t1 = resident pages)          */
  double p;                 /* ARC target for |T1| (c/2 for DBL, 0 for LRU)          */
  int64_t capacity;
  int64_t references;       /* policy references issued                              */
  int64_t requests, prompt_tokens, prefix_hit_tokens, computed_tokens;
  int64_t case_counts[8];   /* per ARCKV_CASE_*                                      */
  int64_t free_blocks, scratch_free;
  int32_t in_flight;
  int32_t policy;
} arckv_stats;

int32_t arckv_cache_stats(const arckv_cache* cache, arckv_stats* out);

/* One policy reference, in issue order. */
typedef struct {
  uint64_t key;          /* identity referenced                                      */
  uint64_t evicted;      /* page moved to a ghost list (or evicted, LRU) by it, or 0 */
  uint64_t dropped;      /* ghost dropped from B1/B2, or T1 page dropped (IV-A), or 0 */
  double p_after;        /* ARC target after the reference                           */
  int32_t kase;          /* ARCKV_CASE_*                                             */
  int32_t evicted_from;  /* ARCKV_LIST_T1 / T2 / NONE                                */
  int32_t dropped_from;  /* ARCKV_LIST_B1 / B2 / T1 / NONE                           */
  int32_t phys_block;    /* physical block of the referenced page afterwards         */
} arckv_event;

/* Routes the decision log into buf (host, caller-owned, cap events); references after the
 * buffer is full are counted but not stored.  buf = NULL switches the log off. */
int32_t arckv_cache_set_log(arckv_cache* cache, arckv_event* buf, int64_t cap);
/* Events issued since the last set_log (may exceed the capacity). */
int32_t arckv_cache_log_count(const arckv_cache* cache, int64_t* n);

/* Contents of one list (ARCKV_LIST_T1..B2), LRU to MRU: keys and physical blocks (-1 for
 * ghosts).  *n receives the list size; ENOSPC if it exceeds cap (nothing written). */
int32_t arckv_cache_snapshot(const arckv_cache* cache, int32_t list, uint64_t* keys,
                             int32_t* phys, int64_t cap, int64_t* n);

/* Checkpoint / resume, so that a long replay (e.g. the 10,000-request trace) can stop and go
 * on.  arckv_cache_save writes the whole state of a cache with no batch in flight into buf
 * (host, caller-owned, cap bytes): its configuration, p, the four lists from LRU to MRU with
 * each entry's identity, physical block, prompt depth and digest, the page free list, the
 * scratch FIFO and the counters, as a self-contained image of little-endian 64-bit words.
 * *n receives the image size in bytes (buf = NULL: size only).  ESTATE if a batch is in
 * flight; ENOSPC if cap < *n.  arckv_cache_restore creates a cache from such an image; every
 * later call on it behaves exactly as on the cache that was saved (the same decisions,
 * placements, plans and statistics).  The decision-log buffer is not part of the state, nor
 * are the device pools: their physical block numbers are what the image refers to, so a caller
 * that checkpoints a serving process keeps the pools (or copies of them) beside the image.
 * EINVAL if the image is malformed or inconsistent (nothing is created then). */
int32_t arckv_cache_save(const arckv_cache* cache, void* buf, int64_t cap, int64_t* n);
int32_t arckv_cache_restore(const void* buf, int64_t n, arckv_cache** out);

/* ---------------------------------------------------------------------------------------
 * Device: KV scatter (Sec. 3: a missed block's K/V is recomputed and stored again).
 * ------------------------------------------------------------------------------------- */

/* Bytes of one pool (K or V) in layout V1. */
int64_t arckv_pool_bytes(int64_t num_blocks, int32_t num_kv_heads, int32_t head_dim);

/* pool[slot[t]] <- (k_new[t], v_new[t]) for t < n_tokens, as an exact bit copy.
 * k_pool, v_pool: device, layout V1, num_blocks blocks.  k_new, v_new: device bf16
 * [n_tokens][num_kv_heads][head_dim].  slot_mapping: device int32 [n_tokens]; a slot
 * outside [0, 16 num_blocks) is skipped.  The two pools and the two row arrays must be
 * 16-byte aligned (EINVAL).  Two tokens with the same slot: one of their rows is written
 * (callers give equal bytes, as for a block recomputed twice in one batch).  head_dim in
 * {64, 128} (else EUNSUPPORTED).  Enqueued on stream. */
int32_t arckv_kv_scatter(void* k_pool, void* v_pool, const void* k_new, const void* v_new,
                         const int32_t* slot_mapping, int64_t n_tokens, int64_t num_blocks,
                         int32_t num_kv_heads, int32_t head_dim, void* stream);

/* ---------------------------------------------------------------------------------------
 * Device: prefix-cached paged prefill attention (Sec. 2: prefill runs the uncached part of
 * the prompt; its queries attend to the reused prefix KV and causally to each other).
 * For request r with L tokens, P cached, S = L - P computed, query head h, position j in
 * [P, L):  o = softmax(scale * q . K[0..j]^T) V[0..j], KV head h / (num_q_heads /
 * num_kv_heads); K/V read through the block table.  bf16 in, fp32 accumulate, bf16 out.
 * ------------------------------------------------------------------------------------- */

/* Work decomposition (host): one work item is a query tile of *tile_cols (column = token x
 * query head of one KV group, token-major) of one (request, KV head) over a key range.
 * 256-column tiles: one work-group per item; long key ranges are split when the batch has too
 * few tiles to fill num_cus compute units (into one round of at most num_cus items).
 * 128-column tiles: the items are grouped into lists of 8 entries (the list's items, then idle
 * entries with request -1), one list per work-group, balanced over at most num_cus lists;
 * key ranges are cut where a list's share ends.  Split tiles are merged by a log-sum-exp
 * combine pass.
 * cu_q, seq_lens: HOST copies of the plan's arrays.  work: host int32 buffer of
 * ARCKV_WORK_INTS * work_cap entries or NULL to query sizes.
 * Outputs: *n_work attention items, *n_combine combine items (both stored in work, the
 * combine items after the attention items), *ws_bytes device workspace needed, *tile_cols
 * the tile width (256; 128 when every request has at most 128 columns, e.g. short suffixes
 * and decode batches of one token per request).
 * ENOSPC if n_work + n_combine > work_cap (sizes still reported). */
#define ARCKV_WORK_INTS 8
int32_t arckv_attention_plan(const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs,
                             int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                             int32_t num_cus, int32_t* work, int64_t work_cap,
                             int64_t* n_work, int64_t* n_combine, int64_t* ws_bytes,
                             int32_t* tile_cols);

/* ---------------------------------------------------------------------------------------
 * Host: one batch's whole preparation in one call (Sec. 2 prefix caching and paged KV, Sec. 3
 * block-level eviction): arckv_hash_blocks_batch of every prompt (root `root`),
 * arckv_plan_batch on `cache`, then arckv_attention_plan, with the same results as those
 * calls in sequence.  Everything the device steps read is written into `packed` (host
 * int32; pinned memory lets one asynchronous copy move it), at the offsets reported:
 *   block_tables [n_reqs][bt_stride] | cu_q [n_reqs + 1] | seq_lens [n_reqs] |
 *   slot_mapping [n_slots] | work items [n_work + n_combine][ARCKV_WORK_INTS]
 * prefix_lens and hit_blocks (host, [n_reqs]) receive P and k per request.  bt_stride is the
 * smallest that fits (max ceil(n_tokens / 16)).  packed_cap must reach an upper bound that
 * depends only on the prompt lengths, heads and num_cus: if it does not, ENOSPC with the
 * bound in out->n_packed and the cache unchanged.  n_reqs >= 1 and every n_tokens >= 1 (else
 * EINVAL).  Other errors as for the three calls (a plan error leaves the cache unchanged; the
 * batch is in flight on success, to be ended with arckv_release_batch).  With a cache in
 * check mode the block digests (arckv_digest_blocks, same root) are computed too and every
 * request is checked (ECOLLISION as for arckv_plan_batch). */
typedef struct {
  int32_t n_reqs, bt_stride;
  int64_t off_block_tables, off_cu_q, off_seq_lens, off_slots, off_work; /* in int32 units  */
  int64_t n_packed;        /* ints written (on ENOSPC: the capacity needed)                */
  int64_t n_slots;         /* sum of S                                                     */
  int64_t n_work, n_combine, ws_bytes;  /* as from arckv_attention_plan                    */
  int32_t tile_cols, max_q_len, max_seq_len;
} arckv_batch;

int32_t arckv_prepare_batch(arckv_cache* cache, const int32_t* const* tokens,
                            const int64_t* n_tokens, int32_t n_reqs, uint64_t root,
                            int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                            int32_t num_cus, int32_t* packed, int64_t packed_cap,
                            int32_t* prefix_lens, int32_t* hit_blocks, arckv_batch* out);

/* arckv_prepare_batch for callers that keep their requests' chained hashes (a serving loop
 * holding a running request's block hashes): hashes[r] holds n_tokens[r] / 16 identities
 * (as arckv_hash_blocks gives; may be NULL when there are none); no hashing is done.  Same
 * outputs and errors as arckv_prepare_batch; the requests carry no digests, so check mode
 * does not verify them (their pages' stored digests are left as they were). */
int32_t arckv_prepare_batch_hashed(arckv_cache* cache, const uint64_t* const* hashes,
                                   const int64_t* n_tokens, int32_t n_reqs,
                                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                   int32_t num_cus, int32_t* packed, int64_t packed_cap,
                                   int32_t* prefix_lens, int32_t* hit_blocks, arckv_batch* out);

/* Runs attention for one planned batch.
 * k_pool, v_pool: device, layout V1 (num_blocks blocks).  q: device bf16
 * [n_q][num_q_heads][head_dim], rows ordered by cu_q.  out: device bf16, same shape.
 * block_tables: device int32 [n_reqs][bt_stride]; cu_q: device [n_reqs + 1]; seq_lens:
 * device [n_reqs] (the same values given to arckv_attention_plan).  work: device copy of
 * the plan's items, tile_cols: the plan's tile width.  workspace: device, >= the planned
 * ws_bytes (may be NULL if 0).  Calls that overlap in time must not share a workspace.
 * A block-table entry outside [0, num_blocks) is never dereferenced: the kernel reads block 0
 * in its place, so the keys it covers get unspecified (finite or not) values; entries past a
 * request's last block (the -1 padding of a plan's rows) are not read at all.
 * head_dim in {64, 128}; num_q_heads / num_kv_heads in {1, 2, 4, 5, 8}. */
int32_t arckv_prefill_attention(const void* k_pool, const void* v_pool, const void* q, void* out,
                                const int32_t* block_tables, int32_t bt_stride,
                                const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs,
                                int64_t n_q, int64_t num_blocks, const int32_t* work,
                                int64_t n_work, int64_t n_combine, int32_t tile_cols,
                                int32_t num_q_heads,
                                int32_t num_kv_heads, int32_t head_dim, float scale,
                                void* workspace, int64_t ws_bytes, void* stream);

/* Same as arckv_prefill_attention, for callers that time its two kernels: hipEvent_t handles
 * (each may be NULL) recorded on stream right before the attention kernel (ev_begin), between
 * it and the split-KV combine (ev_mid) and after the combine (ev_end).  The events must have
 * been created by the caller, which keeps ownership. */
int32_t arckv_prefill_attention_timed(const void* k_pool, const void* v_pool, const void* q,
                                      void* out, const int32_t* block_tables, int32_t bt_stride,
                                      const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs,
                                      int64_t n_q, int64_t num_blocks, const int32_t* work,
                                      int64_t n_work, int64_t n_combine, int32_t tile_cols,
                                      int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                      float scale, void* workspace, int64_t ws_bytes, void* stream,
                                      void* ev_begin, void* ev_mid, void* ev_end);

/* For callers that cannot allocate device memory (code under HIP graph capture, serving
 * loops or harnesses that forbid hipMalloc): arckv_prefill_attention with no workspace
 * argument.  ws_bytes is the plan's workspace size (arckv_attention_plan / arckv_batch); the
 * split partials go to a static device array of ARCKV_NOALLOC_MAX_WS_BYTES (64 MiB) per device,
 * held until the process ends, found on this call's first use of the stream's device.  Nothing
 * is allocated or freed.  Every call on one device shares that array: calls that overlap in
 * time on one device race (serialise them, e.g. on one stream).  Other arguments, results and
 * errors as arckv_prefill_attention; ENOSPC if ws_bytes > ARCKV_NOALLOC_MAX_WS_BYTES. */
int32_t arckv_prefill_attention_noalloc(const void* k_pool, const void* v_pool, const void* q,
                                        void* out, const int32_t* block_tables, int32_t bt_stride,
                                        const int32_t* cu_q, const int32_t* seq_lens,
                                        int32_t n_reqs, int64_t n_q, int64_t num_blocks,
                                        const int32_t* work, int64_t n_work, int64_t n_combine,
                                        int32_t tile_cols, int32_t num_q_heads,
                                        int32_t num_kv_heads, int32_t head_dim, float scale,
                                        int64_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------------------
 * Device: the producer of the computed tokens' Q/K/V (the attention inputs of a prefill;
 * Sec. 4 serves Qwen3-14B, whose public configuration fixes the details): projection of the
 * hidden states and rotary position embedding.
 *   y = x W^T (bf16 in, fp32 accumulate, y rounded to bf16), then for every query and key head
 *   at the token's absolute position p (request r's suffix token i: L_r - S_r + i) and
 *   i < head_dim / 2, angle a = p * rope_theta^(-2 i / head_dim):
 *   out[i] = u[i] cos a - u[i + D/2] sin a,  out[i + D/2] = u[i + D/2] cos a + u[i] sin a
 *   (angles in fp64, reduced mod 2 pi, then fp32 sine / cosine and rotation); values pass
 *   through.  Outputs bf16, round to nearest even.
 * x: device bf16 [n_tokens][hidden], rows ordered by cu_q.  w_qkv: device bf16
 * [(num_q_heads + 2 num_kv_heads) head_dim][hidden] (query heads, then key heads, then value
 * heads).  cu_q [n_reqs + 1], seq_lens [n_reqs]: device, as for the attention call
 * (n_tokens = cu_q[n_reqs]).  workspace: device, >= 4 n_tokens head_dim bytes (the (cos, sin)
 * pairs of every token as fp32), caller-owned.  q_out: device bf16 [n_tokens][num_q_heads]
 * [head_dim]; k_out, v_out: device bf16 [n_tokens][num_kv_heads][head_dim] (the layout
 * arckv_kv_scatter takes).  x, w_qkv, workspace, q_out, k_out and v_out must be 16-byte
 * aligned.  One fused kernel (GEMM tile + rotation in its epilogue) after a small table
 * pass; y never goes to memory.  Stream-ordered on `stream`.  head_dim in {64, 128}, hidden a
 * multiple of 32 (at most 2^22) and (num_q_heads + 2 num_kv_heads) head_dim a multiple of 128: else
 * EUNSUPPORTED; EINVAL on bad sizes, NULL or misaligned pointers or rope_theta <= 1; ENOSPC if
 * the workspace is too small; EDEVICE if a launch fails.  n_tokens = 0 is a no-op. */
int32_t arckv_qkv_rope(const void* x, const void* w_qkv, int64_t n_tokens, int32_t hidden,
                       int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                       const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs,
                       double rope_theta, void* workspace, int64_t ws_bytes, void* q_out,
                       void* k_out, void* v_out, void* stream);

/* The same producer with the KV scatter fused into it: Q as arckv_qkv_rope writes it, and K
 * and V of token t written straight into the paged pools at slot_mapping[t] (layout V1, as
 * arckv_kv_scatter writes them: pool[slot] <- the token's rotated K row and its V row), so
 * the scatter launch and the [n_tokens][num_kv_heads][head_dim] K/V rows disappear (Sec. 3:
 * the K/V of blocks that missed the cache are computed again and stored in the pool).
 * k_pool, v_pool: device, num_blocks blocks,
 * 16-byte aligned.  slot_mapping: device int32 [n_tokens]; a slot outside
 * [0, 16 num_blocks) is skipped.  The bytes written equal arckv_qkv_rope followed by
 * arckv_kv_scatter on the same slots (two tokens with the same slot: one of them wins).
 * Other arguments, requirements and errors as arckv_qkv_rope; EINVAL also for num_blocks
 * outside [1, 2^27] or a NULL slot_mapping. */
int32_t arckv_qkv_rope_to_pool(const void* x, const void* w_qkv, int64_t n_tokens, int32_t hidden,
                               int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                               const int32_t* cu_q, const int32_t* seq_lens, int32_t n_reqs,
                               double rope_theta, void* workspace, int64_t ws_bytes, void* q_out,
                               void* k_pool, void* v_pool, int64_t num_blocks,
                               const int32_t* slot_mapping, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* ARCKV_H */
