"""PrefillEngine: the per-batch hot path wired over libarckv.

prepare (hash blocks, plan the batch on the host cache, plan the attention work, pack the
metadata: one native call) -> copy metadata to the device -> [project Q/K/V] -> scatter the
computed tokens' K/V -> prefix-cached prefill attention -> release.
Every step is a libarckv call; this class owns the device buffers (PyTorch tensors used
only as device memory) and the host cache handle.  plan() + upload() are the same first
steps as separate calls.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import (BlockCache, BatchPlan, attention_plan, hash_blocks_batch, lib, unpack_prepared)
from . import _lib


@dataclass
class DeviceBatch:
    plan: BatchPlan
    block_tables: object
    cu_q: object
    seq_lens: object
    slot_mapping: object
    work: object
    n_work: int
    n_combine: int
    ws_bytes: int
    tile_cols: int
    n_tokens: int = 0          # computed (suffix) tokens of the batch: rows of q / k_new / v_new
    work_ptr: int = 0          # device address of the work array


class PrefillEngine:
    def __init__(self, num_q_heads: int, num_kv_heads: int, head_dim: int, capacity: int,
                 num_phys: int, scratch: int, policy: str = "arc", initial_order=None,
                 ref_order: str = "tail_first", device: str = "cuda", num_cus: int | None = None,
                 pool_fill: int = -1, victim_window: int = 1, intra_batch_reuse: bool = True,
                 frc_p: float = 0.0):
        import torch
        self.hq, self.hkv, self.d = num_q_heads, num_kv_heads, head_dim
        self.scale = head_dim ** -0.5
        self.device = torch.device(device)
        self.num_phys = num_phys
        # pools hold bf16 bit patterns; the fill (0xFFFF, a NaN pattern) marks untouched slots
        self.k_pool = torch.full((num_phys, num_kv_heads, 16, head_dim), pool_fill, dtype=torch.int16,
                                 device=self.device)
        self.v_pool = torch.full((num_phys, num_kv_heads, head_dim, 16), pool_fill, dtype=torch.int16,
                                 device=self.device)
        self.cache = BlockCache(policy, capacity, num_phys, scratch, initial_order, ref_order, victim_window,
                                intra_batch_reuse, frc_p)
        if num_cus is None:
            num_cus = torch.cuda.get_device_properties(self.device).multi_processor_count
        self.num_cus = int(num_cus)
        self._ws = torch.empty(0, dtype=torch.uint8, device=self.device)
        self._y = None          # rotary (cos, sin) table of the batch (arckv_qkv_rope workspace)
        # a ring of reusable pinned staging buffers and device metadata buffers, with the events
        # that mark their copies done: the host may prepare up to four batches ahead of the GPU
        # (a slow host step is then absorbed), and no pinned memory is allocated per batch
        self._ring = 4
        self._stage = [None] * self._ring
        self._stage_ev = [None] * self._ring
        self._dev_meta = [None] * self._ring
        self._turn = 0

    # ---- host steps ----------------------------------------------------------------------
    def plan(self, token_lists) -> BatchPlan:
        """Hashes and the cache plan only (prepare() does these and the rest in one call)."""
        hashes = hash_blocks_batch(token_lists)
        return self.cache.plan_batch([(h, len(t)) for h, t in zip(hashes, token_lists)])

    def release(self):
        self.cache.release_batch()

    def prepare(self, token_lists, stream=None, hashes=None, n_tokens=None) -> DeviceBatch:
        """plan() + upload() in one native call (arckv_prepare_batch): hashes, the cache plan
        and the attention work plan are written straight into the next pinned staging buffer of
        the ring, then one asynchronous copy on `stream` moves them to the device.  A caller that
        keeps its requests' block hashes passes `hashes` and `n_tokens` instead of token lists."""
        import torch
        ts = self._torch_stream(stream)
        t = self._turn
        self._turn = (t + 1) % self._ring
        if self._stage_ev[t] is not None:
            self._stage_ev[t].synchronize()          # the copy that last read this buffer is done
        while True:
            host = None if self._stage[t] is None else self._stage[t].numpy()
            st, d, pl, hb = self.cache.prepare_native(token_lists, self.hq, self.hkv, self.d, self.num_cus, host,
                                                      hashes=hashes, n_tokens=n_tokens)
            if st == _lib.ENOSPC and (host is None or d["n_packed"] > host.size):
                cap = max(d["n_packed"], 1 << 16) * 2
                self._stage[t] = torch.empty(cap, dtype=torch.int32, pin_memory=True)
                with torch.cuda.stream(ts):
                    self._dev_meta[t] = torch.empty(cap, dtype=torch.int32, device=self.device)
                continue
            _lib.check(st, "arckv_prepare_batch")
            break
        n_int = d["n_packed"]
        dev = self._copy_meta(t, n_int, ts)
        plan, ap = unpack_prepared(host, d, pl, hb)
        n, stride = d["n_reqs"], d["bt_stride"]
        bt = dev[d["off_block_tables"]:d["off_block_tables"] + n * stride].view(n, stride)
        cu = dev[d["off_cu_q"]:d["off_cu_q"] + n + 1]
        sl = dev[d["off_seq_lens"]:d["off_seq_lens"] + n]
        sm = dev[d["off_slots"]:d["off_slots"] + d["n_slots"]]
        wk = dev[d["off_work"]:d["off_work"] + (d["n_work"] + d["n_combine"]) * 8].view(-1, 8)
        self._ensure_ws(d["ws_bytes"], ts)
        return DeviceBatch(plan, bt, cu, sl, sm, wk, d["n_work"], d["n_combine"], d["ws_bytes"],
                           d["tile_cols"], int(d["n_slots"]), wk.data_ptr())

    def upload(self, plan: BatchPlan, stream=None) -> DeviceBatch:
        """The metadata of a plan() result to the device, copied on `stream`."""
        import torch
        ts = self._torch_stream(stream)
        ap = attention_plan(plan.cu_q, plan.seq_lens, self.hq, self.hkv, self.d, self.num_cus)
        parts = [plan.block_tables.ravel(), plan.cu_q, plan.seq_lens, plan.slot_mapping, ap.work.ravel()]
        n_int = sum(p.size for p in parts)
        t = self._turn
        self._turn = (t + 1) % self._ring
        if self._stage_ev[t] is not None:
            self._stage_ev[t].synchronize()          # the copy that last read this buffer is done
        if self._stage[t] is None or self._stage[t].numel() < n_int:
            cap = max(n_int, 1 << 16) * 2
            self._stage[t] = torch.empty(cap, dtype=torch.int32, pin_memory=True)
            with torch.cuda.stream(ts):
                self._dev_meta[t] = torch.empty(cap, dtype=torch.int32, device=self.device)
        host = self._stage[t].numpy()
        o = 0
        for p in parts:
            host[o:o + p.size] = p
            o += p.size
        dev = self._copy_meta(t, n_int, ts)
        n = plan.n_reqs
        o = 0
        bt = dev[o:o + plan.block_tables.size].view(n, plan.block_tables.shape[1]); o += plan.block_tables.size
        cu = dev[o:o + n + 1]; o += n + 1
        sl = dev[o:o + n]; o += n
        sm = dev[o:o + len(plan.slot_mapping)]; o += len(plan.slot_mapping)
        wk = dev[o:o + ap.work.size].view(-1, 8)
        self._ensure_ws(ap.ws_bytes, ts)
        return DeviceBatch(plan, bt, cu, sl, sm, wk, ap.n_work, ap.n_combine, ap.ws_bytes, ap.tile_cols,
                           int(plan.cu_q[-1]), wk.data_ptr())

    # ---- streams ---------------------------------------------------------------------------
    # `stream` is None (torch's current stream), a torch.cuda.Stream or a raw hipStream_t
    # handle.  The metadata copy, its event and every (re)allocation of a device buffer run on
    # that stream, the stream the kernels then run on: the kernels are ordered after the copy,
    # and the caching allocator hands out a replaced buffer's memory again only in that
    # stream's order, after the kernels that read it.
    def _torch_stream(self, stream):
        import torch
        if stream is None:
            return torch.cuda.current_stream(self.device)
        if isinstance(stream, torch.cuda.Stream):
            return stream
        return torch.cuda.ExternalStream(int(stream), device=self.device)

    def _stream(self, stream):
        if stream is None:
            import torch
            return torch.cuda.current_stream(self.device).cuda_stream
        return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)

    def _copy_meta(self, t: int, n_int: int, ts):
        """Staging buffer t -> its device buffer on stream ts; the event marks the copy done, so
        that the host refills the staging buffer only after the copy has read it."""
        import torch
        dev = self._dev_meta[t][:n_int]
        with torch.cuda.stream(ts):
            dev.copy_(self._stage[t][:n_int], non_blocking=True)
            ev = torch.cuda.Event()
            ev.record(ts)
        self._stage_ev[t] = ev
        return dev

    def _ensure_ws(self, nbytes: int, ts):
        if nbytes > self._ws.numel():
            import torch
            with torch.cuda.stream(ts):
                self._ws = torch.empty(nbytes, dtype=torch.uint8, device=self.device)

    # ---- device steps --------------------------------------------------------------------
    # The engine built every device buffer itself, so these calls skip the binding's per-call
    # tensor checks and pass raw addresses straight to the C ABI (the library still validates
    # sizes); they only check the shapes of the caller's q / k / v / out.

    def scatter(self, db: DeviceBatch, k_new, v_new, stream=None):
        shape = (db.n_tokens, self.hkv, self.d)
        if tuple(k_new.shape) != shape or tuple(v_new.shape) != shape or not (
                k_new.is_contiguous() and v_new.is_contiguous()) or k_new.element_size() != 2:
            raise ValueError(f"k_new / v_new must be contiguous 16-bit {shape}")
        _lib.check(lib().arckv_kv_scatter(self.k_pool.data_ptr(), self.v_pool.data_ptr(), k_new.data_ptr(),
                                          v_new.data_ptr(), db.slot_mapping.data_ptr(), db.n_tokens,
                                          self.num_phys, self.hkv, self.d, self._stream(stream)),
                   "arckv_kv_scatter")

    def project(self, db: DeviceBatch, x, w_qkv, q, k_new, v_new, rope_theta: float, stream=None):
        """Q/K/V of the batch's computed tokens from their hidden states x [n_tokens, H]
        (projection by w_qkv [(Hq + 2 Hkv) D, H] and rotary embedding, arckv_qkv_rope);
        k_new / v_new then go to scatter()."""
        import torch
        t, h = db.n_tokens, int(x.shape[1])
        n_out = (self.hq + 2 * self.hkv) * self.d
        if tuple(x.shape) != (t, h) or tuple(w_qkv.shape) != (n_out, h) or x.element_size() != 2 or \
                not (x.is_contiguous() and w_qkv.is_contiguous()):
            raise ValueError(f"x must be contiguous 16-bit [{t}, H] and w_qkv [{n_out}, H]")
        for a, c in ((q, self.hq), (k_new, self.hkv), (v_new, self.hkv)):
            if tuple(a.shape) != (t, c, self.d) or not a.is_contiguous() or a.element_size() != 2:
                raise ValueError("q / k_new / v_new must be contiguous 16-bit [n_tokens, heads, D]")
        need = 4 * t * self.d
        if self._y is None or self._y.numel() < need:
            with torch.cuda.stream(self._torch_stream(stream)):
                self._y = torch.empty(max(need, 1), dtype=torch.uint8, device=self.device)
        _lib.check(lib().arckv_qkv_rope(x.data_ptr(), w_qkv.data_ptr(), t, h, self.hq, self.hkv, self.d,
                                        db.cu_q.data_ptr(), db.seq_lens.data_ptr(), db.plan.n_reqs,
                                        float(rope_theta), self._y.data_ptr(), self._y.numel(),
                                        q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), self._stream(stream)),
                   "arckv_qkv_rope")

    def project_to_pool(self, db: DeviceBatch, x, w_qkv, q, rope_theta: float, stream=None):
        """project() with the KV scatter fused in (arckv_qkv_rope_to_pool): Q into q, the batch's
        K and V straight into the engine's pools at the plan's slots; no scatter() follows."""
        import torch
        t, h = db.n_tokens, int(x.shape[1])
        n_out = (self.hq + 2 * self.hkv) * self.d
        if tuple(x.shape) != (t, h) or tuple(w_qkv.shape) != (n_out, h) or x.element_size() != 2 or \
                not (x.is_contiguous() and w_qkv.is_contiguous()):
            raise ValueError(f"x must be contiguous 16-bit [{t}, H] and w_qkv [{n_out}, H]")
        if tuple(q.shape) != (t, self.hq, self.d) or not q.is_contiguous() or q.element_size() != 2:
            raise ValueError("q must be contiguous 16-bit [n_tokens, heads, D]")
        need = 4 * t * self.d
        if self._y is None or self._y.numel() < need:
            with torch.cuda.stream(self._torch_stream(stream)):
                self._y = torch.empty(max(need, 1), dtype=torch.uint8, device=self.device)
        _lib.check(lib().arckv_qkv_rope_to_pool(
            x.data_ptr(), w_qkv.data_ptr(), t, h, self.hq, self.hkv, self.d, db.cu_q.data_ptr(),
            db.seq_lens.data_ptr(), db.plan.n_reqs, float(rope_theta), self._y.data_ptr(), self._y.numel(),
            q.data_ptr(), self.k_pool.data_ptr(), self.v_pool.data_ptr(), self.num_phys,
            db.slot_mapping.data_ptr(), self._stream(stream)), "arckv_qkv_rope_to_pool")

    def attention(self, db: DeviceBatch, q, out, stream=None, events=None):
        """Prefill attention of the batch.  `events`: optional (begin, mid, end) torch.cuda.Event
        triple (already recorded once, so that each has its HIP handle), recorded by the library
        right before the attention kernel, between it and the split-KV combine, and after it."""
        shape = (db.n_tokens, self.hq, self.d)
        if tuple(q.shape) != shape or tuple(out.shape) != shape or not (
                q.is_contiguous() and out.is_contiguous()) or q.element_size() != 2:
            raise ValueError(f"q / out must be contiguous 16-bit {shape}")
        args = (self.k_pool.data_ptr(), self.v_pool.data_ptr(), q.data_ptr(), out.data_ptr(),
                db.block_tables.data_ptr(), int(db.block_tables.shape[1]), db.cu_q.data_ptr(),
                db.seq_lens.data_ptr(), db.plan.n_reqs, db.n_tokens, self.num_phys, db.work_ptr,
                db.n_work, db.n_combine, db.tile_cols, self.hq, self.hkv, self.d, self.scale,
                self._ws.data_ptr() if db.ws_bytes else None, db.ws_bytes, self._stream(stream))
        if events is None:
            _lib.check(lib().arckv_prefill_attention(*args), "arckv_prefill_attention")
        else:
            _lib.check(lib().arckv_prefill_attention_timed(*args, *(e.cuda_event for e in events)),
                       "arckv_prefill_attention_timed")

    def step(self, token_lists, qkv_for_plan, stream=None, release: bool = True):
        """One batch: plan, upload, scatter, attend, release (release=False: the caller calls
        release()).  qkv_for_plan(plan) returns the computed tokens' (q, k_new, v_new) device
        tensors, ready on `stream`.  Returns (plan, out), out allocated on `stream`."""
        import torch
        db = self.prepare(token_lists, stream)
        plan = db.plan
        try:
            q, k_new, v_new = qkv_for_plan(plan)
            with torch.cuda.stream(self._torch_stream(stream)):
                out = torch.empty_like(q)
            self.scatter(db, k_new, v_new, stream)
            self.attention(db, q, out, stream)
        finally:
            if release:
                self.release()
        return plan, out
