"""arckv: prefix-cached paged prefill attention with an ARC KV-block cache on MI355X.

Thin Python binding over libarckv (include/arckv.h).  Every step of the path runs in the
library: the host cache/planner in C++, scatter and attention in HIP kernels for gfx950.
This module only converts arguments (numpy arrays and torch device tensors to pointers) and
raises on error statuses; if the library has not been built it raises -- there is no
fallback implementation.
"""

from __future__ import annotations

import ctypes as C
from dataclasses import dataclass

import numpy as np

from . import _lib
from ._lib import ArckvError, SYMBOLS, WORK_INTS  # noqa: F401

BLOCK_TOKENS = 16
NOALLOC_MAX_WS_BYTES = 64 << 20     # ARCKV_NOALLOC_MAX_WS_BYTES: the static scratch of prefill_attention_noalloc
LIST_T1, LIST_T2, LIST_B1, LIST_B2 = 1, 2, 3, 4
# ARCKV_CASE_*: indices of stats()["case_counts"] and Event.kase
CASE_I, CASE_II, CASE_III, CASE_IVA, CASE_IVA_T1DEL, CASE_IVB, CASE_LRU_HIT, CASE_LRU_MISS = range(8)


def lib():
    return _lib.load()


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


# ------------------------------------------------------------------------------------------
# host: hashing and the block cache
# ------------------------------------------------------------------------------------------

def hash_blocks(tokens, root: int = 0) -> np.ndarray:
    """Chained identities (uint64) of the full 16-token blocks of one token sequence."""
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    out = np.empty(len(t) // BLOCK_TOKENS, dtype=np.uint64)
    nf = _lib.i64()
    _lib.check(lib().arckv_hash_blocks(_ptr(t, _lib.i32), len(t), C.c_uint64(root), _ptr(out, _lib.u64),
                                       len(out), C.byref(nf)), "arckv_hash_blocks")
    return out


def digest_blocks(tokens, root: int = 0) -> np.ndarray:
    """Chained block digests (uint64) for collision checks: an independent second hash of
    every full 16-token block (arckv_digest_blocks)."""
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    out = np.empty(len(t) // BLOCK_TOKENS, dtype=np.uint64)
    nf = _lib.i64()
    _lib.check(lib().arckv_digest_blocks(_ptr(t, _lib.i32), len(t), C.c_uint64(root), _ptr(out, _lib.u64),
                                         len(out), C.byref(nf)), "arckv_digest_blocks")
    return out


class forced_identity_mask:
    """TEST ONLY: while active, every block identity the library computes is ANDed with
    `mask` (arckv_test_set_hash_mask), which forces identity collisions."""

    def __init__(self, mask: int):
        self.mask = int(mask)
        self._prev = None

    def __enter__(self):
        prev = _lib.u64()
        _lib.check(lib().arckv_test_set_hash_mask(C.c_uint64(self.mask), C.byref(prev)), "arckv_test_set_hash_mask")
        self._prev = int(prev.value)
        return self

    def __exit__(self, *exc):
        lib().arckv_test_set_hash_mask(C.c_uint64(self._prev), None)
        return False


def hash_blocks_batch(token_lists, root: int = 0):
    """Chained identities of several sequences in one call -> list of uint64 arrays (views)."""
    toks = [np.ascontiguousarray(t, dtype=np.int32) for t in token_lists]
    n = len(toks)
    lens = np.array([len(t) for t in toks], dtype=np.int64)
    ptrs = (_lib.P_i32 * max(n, 1))(*[_ptr(t, _lib.i32) for t in toks])
    total = int(np.sum(lens // BLOCK_TOKENS))
    out = np.empty(max(total, 1), dtype=np.uint64)
    offs = np.empty(n + 1, dtype=np.int64)
    _lib.check(lib().arckv_hash_blocks_batch(ptrs, _ptr(lens, _lib.i64), n, C.c_uint64(root),
                                             _ptr(out, _lib.u64), len(out), _ptr(offs, _lib.i64)),
               "arckv_hash_blocks_batch")
    return [out[offs[r]:offs[r + 1]] for r in range(n)]


def next_batch(n_tokens, max_batch: int, capacity: int, scratch: int) -> int:
    a = np.ascontiguousarray(n_tokens, dtype=np.int64)
    n = _lib.i32()
    _lib.check(lib().arckv_next_batch(_ptr(a, _lib.i64), len(a), max_batch, capacity, scratch,
                                      C.byref(n)), "arckv_next_batch")
    return int(n.value)


@dataclass
class BatchPlan:
    block_tables: np.ndarray   # int32 [n_reqs, bt_stride], -1 padded
    cu_q: np.ndarray           # int32 [n_reqs + 1]
    seq_lens: np.ndarray       # int32 [n_reqs]
    prefix_lens: np.ndarray    # int32 [n_reqs]
    hit_blocks: np.ndarray     # int32 [n_reqs]
    slot_mapping: np.ndarray   # int32 [n_slots]
    max_q_len: int
    max_seq_len: int

    @property
    def n_reqs(self) -> int:
        return len(self.seq_lens)


@dataclass
class PreparedBatch:
    """What arckv_prepare_batch wrote: the plan and the attention work plan (copies), and the
    packed int32 metadata (`packed[:n_packed]`, the caller's buffer) in the device layout."""
    plan: BatchPlan
    attn: "AttnPlan"
    info: dict                 # bt_stride, off_* (int32 offsets into packed), n_packed, ...
    packed: np.ndarray


class BlockCache:
    """Host ARC (or LRU) cache with physical block placement; plans batches."""

    def __init__(self, policy: str, capacity: int, num_phys: int, scratch: int,
                 initial_order=None, ref_order: str = "tail_first", victim_window: int = 1,
                 intra_batch_reuse: bool = True, frc_p: float = 0.0, check_blocks: bool = False):
        """policy: arc, lru, dbl (p fixed at c/2) or frc (p fixed at frc_p).
        victim_window W > 1: length-aware victims (the deepest of the W least recently used
        unpinned pages of the list a policy evicts from); 1 is the plain policy.
        intra_batch_reuse False: a request's prefix stops at a block an earlier request of the
        same batch created.
        check_blocks True: check mode (pages keep block digests; plans verify them and raise
        ArckvError ECOLLISION when two different blocks share an identity)."""
        self._order = None if initial_order is None else np.ascontiguousarray(initial_order, dtype=np.int32)
        cfg = _lib.CacheCfg(_lib.POLICY[policy], _lib.REF_ORDER[ref_order], capacity, num_phys, scratch,
                            None if self._order is None else _ptr(self._order, _lib.i32), victim_window,
                            0 if intra_batch_reuse else 1, float(frc_p), 1 if check_blocks else 0)
        h = C.c_void_p()
        _lib.check(lib().arckv_cache_create(C.byref(cfg), C.byref(h)), "arckv_cache_create")
        self._h = h
        self._log = None
        self.capacity = capacity

    def save(self) -> bytes:
        """The cache's whole state between batches as a byte image (arckv_cache_save)."""
        n = _lib.i64()
        _lib.check(lib().arckv_cache_save(self._h, None, 0, C.byref(n)), "arckv_cache_save")
        buf = C.create_string_buffer(n.value)
        _lib.check(lib().arckv_cache_save(self._h, buf, n.value, C.byref(n)), "arckv_cache_save")
        return buf.raw[: n.value]

    @classmethod
    def restore(cls, image: bytes) -> "BlockCache":
        """A cache that continues exactly where the saved one stopped (arckv_cache_restore)."""
        h = C.c_void_p()
        buf = C.create_string_buffer(bytes(image), len(image))
        _lib.check(lib().arckv_cache_restore(buf, len(image), C.byref(h)), "arckv_cache_restore")
        self = cls.__new__(cls)
        self._order = None
        self._h = h
        self._log = None
        st = _lib.Stats()
        _lib.check(lib().arckv_cache_stats(h, C.byref(st)), "arckv_cache_stats")
        self.capacity = int(st.capacity)
        return self

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().arckv_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def plan_batch(self, reqs, bt_stride: int | None = None) -> BatchPlan:
        """reqs: sequence of (hashes uint64 array, n_tokens) or (hashes, n_tokens, digests)."""
        n = len(reqs)
        keep = [np.ascontiguousarray(rq[0], dtype=np.uint64) for rq in reqs]
        dig = [None if len(rq) < 3 or rq[2] is None else np.ascontiguousarray(rq[2], dtype=np.uint64)
               for rq in reqs]
        arr = (_lib.Req * max(n, 1))()
        for i, (rq, h, d) in enumerate(zip(reqs, keep, dig)):
            if d is not None and len(d) != len(h):
                raise ValueError(f"request {i}: {len(d)} digests for {len(h)} blocks")
            arr[i] = _lib.Req(_ptr(h, _lib.u64), len(h), int(rq[1]), None if d is None else _ptr(d, _lib.u64))
        lens = [int(rq[1]) for rq in reqs]
        stride = bt_stride or max([(x + BLOCK_TOKENS - 1) // BLOCK_TOKENS for x in lens] + [1])
        bt = np.empty((n, stride), dtype=np.int32)
        cu = np.empty(n + 1, dtype=np.int32)
        sl = np.empty(n, dtype=np.int32)
        pl = np.empty(n, dtype=np.int32)
        hb = np.empty(n, dtype=np.int32)
        cap = max(sum(lens), 1)
        slots = np.empty(cap, dtype=np.int32)
        pc = _lib.PlanC(_ptr(bt, _lib.i32), stride, _ptr(cu, _lib.i32), _ptr(sl, _lib.i32), _ptr(pl, _lib.i32),
                        _ptr(hb, _lib.i32), _ptr(slots, _lib.i32), cap, 0, 0, 0)
        _lib.check(lib().arckv_plan_batch(self._h, arr, n, C.byref(pc)), "arckv_plan_batch")
        return BatchPlan(bt, cu, sl, pl, hb, slots[: pc.n_slots].copy(), pc.max_q_len, pc.max_seq_len)

    def prepare_native(self, token_lists, num_q_heads: int, num_kv_heads: int, head_dim: int,
                       num_cus: int, packed: np.ndarray, root: int = 0, hashes=None, n_tokens=None):
        """One call of arckv_prepare_batch into `packed` (contiguous writable int32), or, with
        `hashes` (uint64 arrays) and `n_tokens`, of arckv_prepare_batch_hashed (token_lists is
        then unused).  Returns (status, info dict, prefix_lens, hit_blocks) without raising; on
        ENOSPC info["n_packed"] is the capacity needed (the cache is then unchanged)."""
        if hashes is None:
            seqs = [t if (t.dtype == np.int32 and t.flags.c_contiguous) else np.ascontiguousarray(t, dtype=np.int32)
                    for t in token_lists]
            lens = np.fromiter((t.shape[0] for t in seqs), dtype=np.int64, count=len(seqs))
            n = len(seqs)
            addrs = np.fromiter((t.__array_interface__["data"][0] for t in seqs), dtype=np.uint64, count=n)
        else:
            # one contiguous copy of every request's hashes and vectorised row pointers into it:
            # far cheaper per request than taking each array's own address
            n = len(hashes)
            lens = np.ascontiguousarray(n_tokens, dtype=np.int64)
            sizes = np.fromiter((len(h) for h in hashes), dtype=np.int64, count=n)
            if lens.shape != (n,) or (sizes < lens // BLOCK_TOKENS).any():
                raise ValueError("prepare_native: each request needs n_tokens // 16 hashes")
            # (a list of Python ints is converted on its own: exact for values >= 2^63)
            flat = (np.concatenate([h if isinstance(h, np.ndarray) else np.array(h, dtype=np.uint64)
                                    for h in hashes], dtype=np.uint64, casting="unsafe") if n
                    else np.zeros(0, dtype=np.uint64))
            starts = np.zeros(n, dtype=np.uint64)
            np.cumsum(sizes[:-1], out=starts[1:])
            addrs = np.uint64(flat.__array_interface__["data"][0]) + np.uint64(8) * starts
        pl = np.empty(max(n, 1), dtype=np.int32)
        hb = np.empty(max(n, 1), dtype=np.int32)
        info = _lib.BatchC()
        cap = 0 if packed is None else packed.size
        pk = None if packed is None else packed.__array_interface__["data"][0]
        a, ln = addrs.__array_interface__["data"][0], lens.__array_interface__["data"][0]
        if hashes is None:
            st = lib().arckv_prepare_batch(self._h, a, ln, n, root, num_q_heads, num_kv_heads, head_dim,
                                           num_cus, pk, cap, pl.__array_interface__["data"][0],
                                           hb.__array_interface__["data"][0], C.byref(info))
        else:
            st = lib().arckv_prepare_batch_hashed(self._h, a, ln, n, num_q_heads, num_kv_heads, head_dim,
                                                  num_cus, pk, cap, pl.__array_interface__["data"][0],
                                                  hb.__array_interface__["data"][0], C.byref(info))
        d = {k: getattr(info, k) for k, _ in _lib.BatchC._fields_}
        return st, d, pl[:n], hb[:n]

    def prepare_batch(self, token_lists, num_q_heads: int, num_kv_heads: int, head_dim: int,
                      num_cus: int = 256, packed: np.ndarray | None = None, root: int = 0) -> PreparedBatch:
        """Hash, plan and work-plan one batch in one native call; `packed` grows if too small."""
        while True:
            st, d, pl, hb = self.prepare_native(token_lists, num_q_heads, num_kv_heads, head_dim,
                                                num_cus, packed, root)
            if st == _lib.ENOSPC and (packed is None or d["n_packed"] > packed.size):
                packed = np.empty(d["n_packed"], dtype=np.int32)
                continue
            _lib.check(st, "arckv_prepare_batch")
            break
        return PreparedBatch(*unpack_prepared(packed, d, pl, hb), d, packed)

    def release_batch(self):
        _lib.check(lib().arckv_release_batch(self._h), "arckv_release_batch")

    def stats(self) -> dict:
        s = _lib.Stats()
        _lib.check(lib().arckv_cache_stats(self._h, C.byref(s)), "arckv_cache_stats")
        d = {k: getattr(s, k) for k, _ in _lib.Stats._fields_}
        d["case_counts"] = list(s.case_counts)
        return d

    def set_log(self, cap: int):
        """Start recording up to `cap` policy decisions (0 switches the log off)."""
        if cap <= 0:
            self._log = None
            _lib.check(lib().arckv_cache_set_log(self._h, None, 0), "arckv_cache_set_log")
            return
        self._log = (_lib.Event * cap)()
        _lib.check(lib().arckv_cache_set_log(self._h, self._log, cap), "arckv_cache_set_log")

    def log(self) -> list:
        """Recorded decisions as tuples (key, case, evicted, evicted_from, dropped, dropped_from,
        phys, p_after)."""
        n = _lib.i64()
        _lib.check(lib().arckv_cache_log_count(self._h, C.byref(n)), "arckv_cache_log_count")
        if self._log is None:
            return []
        m = min(n.value, len(self._log))
        return [(e.key, e.kase, e.evicted, e.evicted_from, e.dropped, e.dropped_from, e.phys_block,
                 e.p_after) for e in self._log[:m]]

    def log_array(self) -> np.ndarray:
        """Recorded decisions as one numpy structured array (fields of ``arckv_event``)."""
        if self._log is None:
            return np.ctypeslib.as_array((_lib.Event * 1)())[:0].copy()
        m = min(self.log_count(), len(self._log))
        return np.ctypeslib.as_array(self._log)[:m].copy()

    def log_count(self) -> int:
        n = _lib.i64()
        _lib.check(lib().arckv_cache_log_count(self._h, C.byref(n)), "arckv_cache_log_count")
        return int(n.value)

    def snapshot(self, which: int):
        n = _lib.i64()
        lib().arckv_cache_snapshot(self._h, which, None, None, 0, C.byref(n))
        keys = np.empty(n.value, dtype=np.uint64)
        phys = np.empty(n.value, dtype=np.int32)
        _lib.check(lib().arckv_cache_snapshot(self._h, which, _ptr(keys, _lib.u64), _ptr(phys, _lib.i32),
                                              n.value, C.byref(n)), "arckv_cache_snapshot")
        return keys, phys


# ------------------------------------------------------------------------------------------
# device: pool, scatter, attention
# ------------------------------------------------------------------------------------------

def pool_bytes(num_blocks: int, num_kv_heads: int, head_dim: int) -> int:
    return int(lib().arckv_pool_bytes(num_blocks, num_kv_heads, head_dim))


def _stream(stream):
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _dev(t, dtype_bits: int | None = None, name: str = "tensor"):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype_bits is not None and t.element_size() * 8 != dtype_bits:
        raise ValueError(f"{name} must have {dtype_bits}-bit elements")
    return C.c_void_p(t.data_ptr())


def device_checks(reset: bool = True, stream=None, library=None):
    """(bits, count) of the out-of-range indices the kernels recorded on the current device
    (arckv_device_checks; CHECK_SLOT | CHECK_BLOCK | CHECK_WORK) and clears them if `reset`.
    `library`: a handle from _lib.load() of the checked build (lib/libarckv_checked.so);
    default the loaded library.  Raises EUNSUPPORTED for a build without device checks."""
    L = library or lib()
    bits, count = _lib.i32(), _lib.i64()
    _lib.check(L.arckv_device_checks(C.byref(bits), C.byref(count), 1 if reset else 0,
                                     C.c_void_p(_stream(stream))), "arckv_device_checks")
    return int(bits.value), int(count.value)


def kv_scatter(k_pool, v_pool, k_new, v_new, slot_mapping, stream=None):
    """pool[slot[t]] <- (k_new[t], v_new[t]); pools [blocks, Hkv, 16, D] / [blocks, Hkv, D, 16]."""
    nb, hkv = int(k_pool.shape[0]), int(k_pool.shape[1])
    d = int(k_new.shape[-1])
    n = int(k_new.shape[0])
    if tuple(k_new.shape) != (n, hkv, d) or tuple(v_new.shape) != (n, hkv, d):
        raise ValueError("k_new / v_new must be [n_tokens, num_kv_heads, head_dim]")
    if tuple(k_pool.shape) != (nb, hkv, 16, d) or tuple(v_pool.shape) != (nb, hkv, d, 16):
        raise ValueError("pools must be [blocks, Hkv, 16, D] (K) and [blocks, Hkv, D, 16] (V)")
    if slot_mapping.numel() != n:
        raise ValueError("slot_mapping must hold one slot per token")
    _lib.check(lib().arckv_kv_scatter(_dev(k_pool, 16, "k_pool"), _dev(v_pool, 16, "v_pool"),
                                      _dev(k_new, 16, "k_new"), _dev(v_new, 16, "v_new"),
                                      _dev(slot_mapping, 32, "slot_mapping"), int(k_new.shape[0]), nb,
                                      hkv, d, C.c_void_p(_stream(stream))), "arckv_kv_scatter")


def qkv_rope(x, w_qkv, cu_q, seq_lens, num_q_heads: int, num_kv_heads: int, rope_theta: float,
             q_out, k_out, v_out, workspace, stream=None):
    """Projection + rotary embedding of the computed tokens (arckv_qkv_rope).  Device tensors:
    x [T, H] bf16, w_qkv [(Hq + 2 Hkv) D, H] bf16, cu_q [n+1], seq_lens [n] int32, q_out
    [T, Hq, D], k_out / v_out [T, Hkv, D] bf16, workspace >= 4 T D bytes (the rotary table)."""
    t, h = int(x.shape[0]), int(x.shape[1])
    d = int(q_out.shape[2])
    n_out = (num_q_heads + 2 * num_kv_heads) * d
    if tuple(w_qkv.shape) != (n_out, h):
        raise ValueError(f"w_qkv must be [{n_out}, {h}]")
    if tuple(q_out.shape) != (t, num_q_heads, d) or tuple(k_out.shape) != (t, num_kv_heads, d) \
            or tuple(v_out.shape) != (t, num_kv_heads, d):
        raise ValueError("q_out / k_out / v_out shapes do not match x and the head counts")
    if cu_q.numel() != seq_lens.numel() + 1:
        raise ValueError("cu_q must have len(seq_lens) + 1 entries")
    _lib.check(lib().arckv_qkv_rope(
        _dev(x, 16, "x"), _dev(w_qkv, 16, "w_qkv"), t, h, num_q_heads, num_kv_heads, d,
        _dev(cu_q, 32, "cu_q"), _dev(seq_lens, 32, "seq_lens"), int(seq_lens.numel()), float(rope_theta),
        _dev(workspace, None, "workspace"), int(workspace.numel() * workspace.element_size()),
        _dev(q_out, 16, "q_out"), _dev(k_out, 16, "k_out"), _dev(v_out, 16, "v_out"),
        C.c_void_p(_stream(stream))), "arckv_qkv_rope")


def qkv_rope_to_pool(x, w_qkv, cu_q, seq_lens, num_q_heads: int, num_kv_heads: int, rope_theta: float,
                     q_out, k_pool, v_pool, slot_mapping, workspace, stream=None):
    """qkv_rope with the KV scatter fused in (arckv_qkv_rope_to_pool): Q into q_out [T, Hq, D],
    K and V into the paged pools (layout V1, k_pool [N][Hkv][16][D], v_pool [N][Hkv][D][16]) at
    slot_mapping [T] int32."""
    t, h = int(x.shape[0]), int(x.shape[1])
    d = int(q_out.shape[2])
    n_out = (num_q_heads + 2 * num_kv_heads) * d
    if tuple(w_qkv.shape) != (n_out, h):
        raise ValueError(f"w_qkv must be [{n_out}, {h}]")
    if tuple(q_out.shape) != (t, num_q_heads, d):
        raise ValueError("q_out shape does not match x and the head counts")
    nb = int(k_pool.shape[0])
    if tuple(k_pool.shape) != (nb, num_kv_heads, 16, d) or tuple(v_pool.shape) != (nb, num_kv_heads, d, 16):
        raise ValueError("k_pool / v_pool must be layout V1 with matching heads and head_dim")
    if slot_mapping.numel() != t or cu_q.numel() != seq_lens.numel() + 1:
        raise ValueError("slot_mapping must have one slot per token, cu_q len(seq_lens) + 1 entries")
    _lib.check(lib().arckv_qkv_rope_to_pool(
        _dev(x, 16, "x"), _dev(w_qkv, 16, "w_qkv"), t, h, num_q_heads, num_kv_heads, d,
        _dev(cu_q, 32, "cu_q"), _dev(seq_lens, 32, "seq_lens"), int(seq_lens.numel()), float(rope_theta),
        _dev(workspace, None, "workspace"), int(workspace.numel() * workspace.element_size()),
        _dev(q_out, 16, "q_out"), _dev(k_pool, 16, "k_pool"), _dev(v_pool, 16, "v_pool"), nb,
        _dev(slot_mapping, 32, "slot_mapping"), C.c_void_p(_stream(stream))), "arckv_qkv_rope_to_pool")


@dataclass
class AttnPlan:
    work: np.ndarray     # int32 [n_work + n_combine, 8]
    n_work: int
    n_combine: int
    ws_bytes: int
    tile_cols: int       # query columns per work item (256, or 128 for short suffixes)


def attention_plan(cu_q, seq_lens, num_q_heads: int, num_kv_heads: int, head_dim: int,
                   num_cus: int = 256) -> AttnPlan:
    cu = np.ascontiguousarray(cu_q, dtype=np.int32)
    sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
    nw, nc, ws, tc = _lib.i64(), _lib.i64(), _lib.i64(), _lib.i32()
    L = lib()
    _lib.check(L.arckv_attention_plan(_ptr(cu, _lib.i32), _ptr(sl, _lib.i32), len(sl), num_q_heads,
                                      num_kv_heads, head_dim, num_cus, None, 0, C.byref(nw), C.byref(nc),
                                      C.byref(ws), C.byref(tc)), "arckv_attention_plan")
    work = np.zeros((max(nw.value + nc.value, 1), WORK_INTS), dtype=np.int32)
    _lib.check(L.arckv_attention_plan(_ptr(cu, _lib.i32), _ptr(sl, _lib.i32), len(sl), num_q_heads,
                                      num_kv_heads, head_dim, num_cus, _ptr(work, _lib.i32), len(work),
                                      C.byref(nw), C.byref(nc), C.byref(ws), C.byref(tc)),
               "arckv_attention_plan")
    return AttnPlan(work, int(nw.value), int(nc.value), int(ws.value), int(tc.value))


def unpack_prepared(packed: np.ndarray, d: dict, prefix_lens, hit_blocks):
    """(BatchPlan, AttnPlan) copies out of a packed buffer written by arckv_prepare_batch."""
    n, stride = d["n_reqs"], d["bt_stride"]
    o = d["off_block_tables"]
    bt = packed[o:o + n * stride].reshape(n, stride).copy()
    cu = packed[d["off_cu_q"]:d["off_cu_q"] + n + 1].copy()
    sl = packed[d["off_seq_lens"]:d["off_seq_lens"] + n].copy()
    slots = packed[d["off_slots"]:d["off_slots"] + d["n_slots"]].copy()
    nw = d["n_work"] + d["n_combine"]
    work = packed[d["off_work"]:d["off_work"] + nw * WORK_INTS].reshape(nw, WORK_INTS).copy()
    if nw == 0:
        work = np.zeros((1, WORK_INTS), dtype=np.int32)
    plan = BatchPlan(bt, cu, sl, np.array(prefix_lens, dtype=np.int32), np.array(hit_blocks, dtype=np.int32),
                     slots, d["max_q_len"], d["max_seq_len"])
    return plan, AttnPlan(work, d["n_work"], d["n_combine"], d["ws_bytes"], d["tile_cols"])


def _attention_args(k_pool, v_pool, q, out, block_tables, cu_q, seq_lens, work, n_work: int,
                    n_combine: int, tile_cols: int, scale: float):
    """Checked C arguments of the attention calls, up to (excluding) the workspace."""
    n_q, hq, d = int(q.shape[0]), int(q.shape[1]), int(q.shape[2])
    nb, hkv = int(k_pool.shape[0]), int(k_pool.shape[1])
    n_reqs = int(seq_lens.shape[0])
    if tuple(out.shape) != (n_q, hq, d):
        raise ValueError("out must have the shape of q")
    if tuple(k_pool.shape) != (nb, hkv, 16, d) or tuple(v_pool.shape) != (nb, hkv, d, 16):
        raise ValueError("pools must be [blocks, Hkv, 16, D] (K) and [blocks, Hkv, D, 16] (V)")
    if block_tables.dim() != 2 or int(block_tables.shape[0]) != n_reqs or cu_q.numel() != n_reqs + 1:
        raise ValueError("block_tables must be [n_reqs, stride] and cu_q [n_reqs + 1]")
    if work.dim() != 2 or int(work.shape[1]) != WORK_INTS or int(work.shape[0]) < n_work + n_combine:
        raise ValueError("work must be [>= n_work + n_combine, 8]")
    return (_dev(k_pool, 16, "k_pool"), _dev(v_pool, 16, "v_pool"), _dev(q, 16, "q"), _dev(out, 16, "out"),
            _dev(block_tables, 32, "block_tables"), int(block_tables.shape[1]), _dev(cu_q, 32, "cu_q"),
            _dev(seq_lens, 32, "seq_lens"), n_reqs, n_q, nb, _dev(work, 32, "work"), n_work, n_combine,
            int(tile_cols), hq, hkv, d, float(scale))


def prefill_attention(k_pool, v_pool, q, out, block_tables, cu_q, seq_lens, work, n_work: int,
                      n_combine: int, tile_cols: int, scale: float, workspace=None, ws_bytes: int = 0,
                      stream=None):
    """Device tensors: pools (layout V1), q/out [n_q, Hq, D] bf16, block_tables [n, stride] int32,
    cu_q [n+1], seq_lens [n], work [n_work + n_combine, 8] int32, workspace (bytes >= ws_bytes)."""
    args = _attention_args(k_pool, v_pool, q, out, block_tables, cu_q, seq_lens, work, n_work, n_combine,
                           tile_cols, scale)
    if ws_bytes and (workspace is None or workspace.numel() * workspace.element_size() < ws_bytes):
        raise ValueError("workspace smaller than ws_bytes")
    ws = C.c_void_p(0) if workspace is None else _dev(workspace, None, "workspace")
    _lib.check(lib().arckv_prefill_attention(*args, ws, int(ws_bytes), C.c_void_p(_stream(stream))),
               "arckv_prefill_attention")


def prefill_attention_noalloc(k_pool, v_pool, q, out, block_tables, cu_q, seq_lens, work, n_work: int,
                              n_combine: int, tile_cols: int, scale: float, ws_bytes: int = 0, stream=None):
    """prefill_attention without a workspace: the library's static per-device scratch holds the
    split partials (ws_bytes: the plan's size, at most NOALLOC_MAX_WS_BYTES).  Calls that overlap
    in time on one device must not be issued (they share the scratch)."""
    args = _attention_args(k_pool, v_pool, q, out, block_tables, cu_q, seq_lens, work, n_work, n_combine,
                           tile_cols, scale)
    _lib.check(lib().arckv_prefill_attention_noalloc(*args, int(ws_bytes), C.c_void_p(_stream(stream))),
               "arckv_prefill_attention_noalloc")
