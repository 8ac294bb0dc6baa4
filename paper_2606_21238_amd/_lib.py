"""ctypes declarations of the libarckv C ABI (include/arckv.h).  Marshalling only."""

from __future__ import annotations

import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "lib", "libarckv.so")

OK, EINVAL, ENOSPC, EDEVICE, ESTATE, EUNSUPPORTED, ECOLLISION = 0, -1, -2, -3, -4, -5, -6
STATUS_NAMES = {0: "OK", -1: "EINVAL", -2: "ENOSPC", -3: "EDEVICE", -4: "ESTATE", -5: "EUNSUPPORTED",
                -6: "ECOLLISION"}
POLICY = {"arc": 0, "lru": 1, "dbl": 2, "frc": 3}
REF_ORDER = {"tail_first": 0, "head_first": 1}
WORK_INTS = 8
CHECK_SLOT, CHECK_BLOCK, CHECK_WORK = 1, 2, 4

i32, i64, u64, f32, f64, vp = C.c_int32, C.c_int64, C.c_uint64, C.c_float, C.c_double, C.c_void_p
P_i32, P_i64, P_u64 = C.POINTER(i32), C.POINTER(i64), C.POINTER(u64)


class CacheCfg(C.Structure):
    _fields_ = [("policy", i32), ("ref_order", i32), ("capacity_blocks", i64),
                ("num_phys_blocks", i64), ("scratch_blocks", i64), ("initial_free_order", P_i32),
                ("victim_window", i32), ("no_intra_batch_reuse", i32), ("frc_p", f64),
                ("check_blocks", i32)]


class Req(C.Structure):
    _fields_ = [("hashes", P_u64), ("n_full", i64), ("n_tokens", i64), ("digests", P_u64)]


class PlanC(C.Structure):
    _fields_ = [("block_tables", P_i32), ("bt_stride", i32), ("cu_q", P_i32), ("seq_lens", P_i32),
                ("prefix_lens", P_i32), ("hit_blocks", P_i32), ("slot_mapping", P_i32),
                ("slot_cap", i64), ("n_slots", i64), ("max_q_len", i32), ("max_seq_len", i32)]


class BatchC(C.Structure):
    _fields_ = [("n_reqs", i32), ("bt_stride", i32), ("off_block_tables", i64), ("off_cu_q", i64),
                ("off_seq_lens", i64), ("off_slots", i64), ("off_work", i64), ("n_packed", i64),
                ("n_slots", i64), ("n_work", i64), ("n_combine", i64), ("ws_bytes", i64),
                ("tile_cols", i32), ("max_q_len", i32), ("max_seq_len", i32)]


class Stats(C.Structure):
    _fields_ = [("t1", i64), ("t2", i64), ("b1", i64), ("b2", i64), ("p", f64), ("capacity", i64),
                ("references", i64), ("requests", i64), ("prompt_tokens", i64),
                ("prefix_hit_tokens", i64), ("computed_tokens", i64), ("case_counts", i64 * 8),
                ("free_blocks", i64), ("scratch_free", i64), ("in_flight", i32), ("policy", i32)]


class Event(C.Structure):
    _fields_ = [("key", u64), ("evicted", u64), ("dropped", u64), ("p_after", f64), ("kase", i32),
                ("evicted_from", i32), ("dropped_from", i32), ("phys_block", i32)]


_SIGS = {
    "arckv_last_error": (C.c_char_p, []),
    "arckv_version": (i32, []),
    "arckv_hash_blocks": (i32, [P_i32, i64, u64, P_u64, i64, P_i64]),
    "arckv_hash_blocks_batch": (i32, [C.POINTER(P_i32), P_i64, i32, u64, P_u64, i64, P_i64]),
    "arckv_digest_blocks": (i32, [P_i32, i64, u64, P_u64, i64, P_i64]),
    "arckv_device_checks": (i32, [C.POINTER(i32), P_i64, i32, vp]),
    "arckv_cache_save": (i32, [vp, vp, i64, P_i64]),
    "arckv_cache_restore": (i32, [vp, i64, C.POINTER(vp)]),
    "arckv_test_set_hash_mask": (i32, [u64, P_u64]),
    "arckv_cache_create": (i32, [C.POINTER(CacheCfg), C.POINTER(vp)]),
    "arckv_cache_destroy": (i32, [vp]),
    "arckv_next_batch": (i32, [P_i64, i32, i32, i64, i64, P_i32]),
    "arckv_plan_batch": (i32, [vp, C.POINTER(Req), i32, C.POINTER(PlanC)]),
    "arckv_release_batch": (i32, [vp]),
    "arckv_cache_stats": (i32, [vp, C.POINTER(Stats)]),
    "arckv_cache_set_log": (i32, [vp, C.POINTER(Event), i64]),
    "arckv_cache_log_count": (i32, [vp, P_i64]),
    "arckv_cache_snapshot": (i32, [vp, i32, P_u64, P_i32, i64, P_i64]),
    "arckv_pool_bytes": (i64, [i64, i32, i32]),
    "arckv_kv_scatter": (i32, [vp, vp, vp, vp, vp, i64, i64, i32, i32, vp]),
    "arckv_qkv_rope": (i32, [vp, vp, i64, i32, i32, i32, i32, vp, vp, i32, f64, vp, i64, vp, vp, vp, vp]),
    "arckv_qkv_rope_to_pool": (i32, [vp, vp, i64, i32, i32, i32, i32, vp, vp, i32, f64, vp, i64, vp, vp, vp,
                                      i64, vp, vp]),
    "arckv_attention_plan": (i32, [P_i32, P_i32, i32, i32, i32, i32, i32, P_i32, i64, P_i64, P_i64,
                                   P_i64, P_i32]),
    "arckv_prepare_batch": (i32, [vp, vp, vp, i32, u64, i32, i32, i32, i32, vp, i64, vp, vp,
                                  C.POINTER(BatchC)]),
    "arckv_prepare_batch_hashed": (i32, [vp, vp, vp, i32, i32, i32, i32, i32, vp, i64, vp, vp,
                                         C.POINTER(BatchC)]),
    "arckv_prefill_attention": (i32, [vp, vp, vp, vp, vp, i32, vp, vp, i32, i64, i64, vp, i64, i64,
                                      i32, i32, i32, i32, f32, vp, i64, vp]),
    "arckv_prefill_attention_timed": (i32, [vp, vp, vp, vp, vp, i32, vp, vp, i32, i64, i64, vp, i64,
                                            i64, i32, i32, i32, i32, f32, vp, i64, vp, vp, vp, vp]),
    "arckv_prefill_attention_noalloc": (i32, [vp, vp, vp, vp, vp, i32, vp, vp, i32, i64, i64, vp, i64,
                                              i64, i32, i32, i32, i32, f32, i64, vp]),
}

SYMBOLS = tuple(_SIGS)

_lib = None


class ArckvError(RuntimeError):
    def __init__(self, status: int, fn: str, msg: str):
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status
        self.code = STATUS_NAMES.get(status, str(status))


def load(path: str | None = None):
    """Loads libarckv.so (built in-tree; the environment variable ARCKV_LIBRARY names another
    build of it, e.g. the sanitizer build of the host code).  Raises if it has not been built:
    there is no fallback."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or os.environ.get("ARCKV_LIBRARY") or LIB_PATH
    try:
        # torch ships its own libamdhip64.so.7; loading it first makes libarckv bind to that same
        # runtime (one HIP runtime per process; two copies do not share devices or streams)
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(p):
        raise RuntimeError(f"libarckv not built: {p} missing; run `python -m paper_2606_21238_amd.build`")
    lib = C.CDLL(p)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _lib = lib
    return lib


def check(status: int, fn: str) -> int:
    if status != OK:
        msg = load().arckv_last_error().decode(errors="replace")
        raise ArckvError(status, fn, msg)
    return status
