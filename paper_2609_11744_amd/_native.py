"""ctypes declarations for libkvx.so (include/kvx.h). Marshalling only."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvx.so")

c_i32, c_i64, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p


class KvxCache(ctypes.Structure):
    _fields_ = [("k", ctypes.POINTER(c_vp)), ("v", ctypes.POINTER(c_vp)),
                ("num_layers", c_i32), ("num_blocks", c_i32), ("block_size", c_i32),
                ("num_kv_heads", c_i32), ("head_dim", c_i32), ("elem_bytes", c_i32),
                ("layout", c_i32)]


class KvxPiece(ctypes.Structure):
    _fields_ = [("src_offset", c_i64), ("bytes", c_i64), ("bt_first", c_i32),
                ("n_blocks", c_i32), ("l_begin", c_i32), ("l_end", c_i32),
                ("chunk_tokens", c_i32), ("n_spans", c_i32)]


class KvxChunkRef(ctypes.Structure):
    _fields_ = [("packed_offset", c_i64), ("bt_offset", c_i32), ("n_blocks", c_i32)]


class KvxHostChunk(ctypes.Structure):
    _fields_ = [("host", c_vp), ("bt_offset", c_i32), ("n_blocks", c_i32)]


class KvxRingStats(ctypes.Structure):
    _fields_ = [("pieces", c_i64), ("bytes", c_i64), ("fill_ms", ctypes.c_double),
                ("wait_fill_ms", ctypes.c_double), ("enqueue_ms", ctypes.c_double),
                ("dma", c_i32), ("dma_engine", c_i32)]


class KvxTraceEvent(ctypes.Structure):
    _fields_ = [("kind", c_i32), ("piece", c_i32), ("lane", c_i32), ("slot", c_i32),
                ("bytes", c_i64), ("t0_ns", c_i64), ("t1_ns", c_i64)]


class KvxFileChunk(ctypes.Structure):
    _fields_ = [("path", ctypes.c_char_p), ("bt_offset", c_i32), ("n_blocks", c_i32)]


class KvxFileIo(ctypes.Structure):
    _fields_ = [("path", ctypes.c_char_p), ("buf", c_vp), ("offset", c_i64), ("bytes", c_i64)]


class KvxPreloadStats(ctypes.Structure):
    _fields_ = [(n, c_i64) for n in ("hints", "spec_deduped", "spec_dropped", "spec_reads",
                                     "demand_fetches", "hits_ready", "hits_inflight",
                                     "demand_reads", "evictions", "spec_preempted", "bytes_read",
                                     "staged", "held")]


class KvxWalk(ctypes.Structure):
    _fields_ = [("work_items", c_i64), ("parts", c_i32), ("ordered", c_i32), ("linear", c_i32),
                ("pair_slices", c_i32), ("fronts", c_i32), ("reserved", c_i32)]


class KvxCurve(ctypes.Structure):
    _fields_ = [("tokens", ctypes.POINTER(ctypes.c_double)),
                ("seconds", ctypes.POINTER(ctypes.c_double)), ("n", c_i32)]


class KvxStepRequest(ctypes.Structure):
    _fields_ = [("block_hashes", c_vp), ("resident", c_vp), ("n_blocks", c_i32),
                ("n_resident", c_i32), ("new_blocks", c_i32), ("reserved", c_i32)]


class KvxStepRestore(ctypes.Structure):
    _fields_ = [("key", ctypes.c_uint64), ("n_blocks", c_i32), ("request", c_i32),
                ("chunk", c_i32), ("bt_offset", c_i32)]


class KvxStepOffload(ctypes.Structure):
    _fields_ = [("request", c_i32), ("chunk", c_i32), ("n_blocks", c_i32), ("bt_offset", c_i32),
                ("new_first", c_i32)]


class KvxStepPlan(ctypes.Structure):
    _fields_ = [("restore", ctypes.POINTER(KvxStepRestore)),
                ("offload", ctypes.POINTER(KvxStepOffload)),
                ("chunk_states", ctypes.POINTER(c_i32)), ("declined", ctypes.POINTER(c_i32)),
                ("restore_cap", c_i32), ("offload_cap", c_i32), ("chunk_states_cap", c_i32),
                ("declined_cap", c_i32), ("n_restore", c_i32), ("n_offload", c_i32),
                ("n_chunk_states", c_i32), ("n_declined", c_i32), ("resident_hits", c_i32),
                ("reserved", c_i32), ("restore_blocks", c_i64), ("offload_blocks", c_i64),
                ("recompute_blocks", c_i64)]


# name -> (restype, argtypes); every symbol include/kvx.h declares.
SIGNATURES = {
    "kvx_bytes_per_token": (c_i64, [c_i32, c_i32, c_i32, c_i32]),
    "kvx_packed_bytes": (c_i64, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32]),
    "kvx_chunk_stride": (c_i64, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32]),
    "kvx_gather_blocks": (ctypes.c_int, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_vp, c_i32,
                                         c_i32, c_vp, c_vp]),
    "kvx_scatter_blocks": (ctypes.c_int, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_vp, c_i32,
                                          c_i32, c_vp, c_vp]),
    "kvx_scatter_blocks_noalloc": (ctypes.c_int, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_vp,
                                                  c_i32, c_i32, c_vp, c_vp]),
    "kvx_gather_chunks": (ctypes.c_int, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_vp, c_i32,
                                         c_vp, c_i32, c_i32, c_vp, c_i64, c_vp]),
    "kvx_scatter_chunks": (ctypes.c_int, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_vp, c_i32,
                                          c_vp, c_i32, c_i32, c_vp, c_i64, c_vp]),
    "kvx_copy_walk": (ctypes.c_int, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32, c_i32, c_i32,
                                     ctypes.POINTER(KvxWalk)]),
    "kvx_check": (ctypes.c_int, [c_vp]),
    "kvx_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "kvx_plan_pieces": (ctypes.c_int, [ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32, c_i32,
                                       c_i64, c_i32, ctypes.POINTER(KvxPiece), c_i32,
                                       ctypes.POINTER(c_i32)]),
    "kvx_ring_create": (ctypes.c_int, [ctypes.c_int, c_i32, c_i64, c_vp, ctypes.POINTER(c_vp)]),
    "kvx_ring_bind": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32, c_i32,
                                     c_vp, c_i32]),
    "kvx_restore_from_staging": (ctypes.c_int, [c_vp, c_vp, c_vp]),
    "kvx_ring_bind_chunks": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32,
                                            ctypes.POINTER(KvxHostChunk), c_i32, c_i32]),
    "kvx_ring_bind_offload": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32,
                                             ctypes.POINTER(KvxHostChunk), c_i32, c_i32]),
    "kvx_offload_to_staging": (ctypes.c_int, [c_vp, c_vp, c_vp]),
    "kvx_offload_begin": (ctypes.c_int, [c_vp, c_vp, c_vp]),
    "kvx_offload_wait": (ctypes.c_int, [c_vp]),
    "kvx_restore_begin": (ctypes.c_int, [c_vp, c_vp, c_vp]),
    "kvx_restore_wait": (ctypes.c_int, [c_vp, c_vp]),
    "kvx_ring_stats_get": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxRingStats)]),
    "kvx_ring_set_trace": (ctypes.c_int, [c_vp, c_i32]),
    "kvx_ring_trace_get": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxTraceEvent), c_i32,
                                          ctypes.POINTER(c_i32)]),
    "kvx_ring_abort": (ctypes.c_int, [c_vp]),
    "kvx_ring_set_test_hooks": (ctypes.c_int, [c_vp, c_i32, c_i32]),
    "kvx_ring_destroy": (ctypes.c_int, [c_vp]),
    "kvx_block_hashes": (c_i64, [c_vp, c_i64, c_i32, ctypes.c_uint64, c_vp]),
    "kvx_dedupe_keys": (ctypes.c_int, [c_vp, c_i32, c_vp]),
    "kvx_plan_step": (ctypes.c_int, [ctypes.POINTER(KvxStepRequest), c_i32, c_i32, c_i32, c_i64,
                                     ctypes.POINTER(KvxStepPlan)]),
    "kvx_curve_eval": (ctypes.c_int, [ctypes.POINTER(KvxCurve), ctypes.c_double,
                                      ctypes.POINTER(ctypes.c_double)]),
    "kvx_load_beats_recompute": (ctypes.c_int, [ctypes.POINTER(KvxCurve), ctypes.POINTER(KvxCurve),
                                                c_i64, c_i64, ctypes.POINTER(c_i32)]),
    "kvx_break_even_prefix": (ctypes.c_int, [ctypes.POINTER(KvxCurve), ctypes.POINTER(KvxCurve),
                                             c_i64, c_i32, ctypes.POINTER(c_i64)]),
    "kvx_break_even_tokens": (ctypes.c_int, [ctypes.POINTER(KvxCurve), ctypes.POINTER(KvxCurve),
                                             c_i64, c_i32, ctypes.POINTER(c_i64)]),
    "kvx_max_io": (ctypes.c_int, [ctypes.POINTER(KvxCurve), ctypes.POINTER(KvxCurve),
                                  ctypes.POINTER(KvxCurve), c_i64,
                                  ctypes.POINTER(ctypes.c_double)]),
    "kvx_hit_curve_from_rate": (ctypes.c_int, [ctypes.POINTER(KvxCurve), c_i64, ctypes.c_double,
                                               ctypes.POINTER(ctypes.c_double)]),
    "kvx_required_GBps": (ctypes.c_int, [ctypes.POINTER(KvxCurve), ctypes.POINTER(KvxCurve),
                                         ctypes.POINTER(KvxCurve), c_i64, c_i64,
                                         ctypes.POINTER(ctypes.c_double)]),
    "kvx_tier_threshold": (ctypes.c_int, [ctypes.POINTER(KvxCurve), ctypes.POINTER(KvxCurve),
                                          c_i64, ctypes.c_double, c_i64, c_i32,
                                          ctypes.POINTER(c_i64)]),
    "kvx_probe_stream": (ctypes.c_int, [c_vp, c_vp, c_i64, c_i32, c_vp]),
    "kvx_ring_bind_files": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32,
                                           ctypes.POINTER(KvxFileChunk), c_i32, c_i32]),
    "kvx_ring_bind_offload_files": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxCache), c_i32, c_i32,
                                                   c_i32, ctypes.POINTER(KvxFileChunk), c_i32,
                                                   c_i32]),
    "kvx_chunk_path": (c_i32, [ctypes.c_char_p, ctypes.c_char_p, ctypes.c_uint64,
                               ctypes.c_char_p, c_i32]),
    "kvx_read_files": (ctypes.c_int, [ctypes.POINTER(KvxFileIo), c_i32, c_i32]),
    "kvx_write_files": (ctypes.c_int, [ctypes.POINTER(KvxFileIo), c_i32, c_i32]),
    "kvx_preloader_create": (ctypes.c_int, [c_i32, c_i64, c_i32, c_i32, c_i32,
                                            ctypes.POINTER(c_vp)]),
    "kvx_preload_hint": (ctypes.c_int, [c_vp, ctypes.POINTER(ctypes.c_char_p), c_i32]),
    "kvx_preload_fetch": (ctypes.c_int, [c_vp, ctypes.POINTER(ctypes.c_char_p), c_i32,
                                         ctypes.POINTER(c_vp), ctypes.POINTER(c_i64)]),
    "kvx_preload_release": (ctypes.c_int, [c_vp, ctypes.POINTER(ctypes.c_char_p), c_i32]),
    "kvx_preload_wait_idle": (ctypes.c_int, [c_vp]),
    "kvx_preload_stats_get": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxPreloadStats)]),
    "kvx_preload_set_test_hooks": (ctypes.c_int, [c_vp, c_i32]),
    "kvx_ring_bind_preloaded": (ctypes.c_int, [c_vp, ctypes.POINTER(KvxCache), c_i32, c_i32, c_i32,
                                               c_vp, ctypes.POINTER(KvxFileChunk), c_i32]),
    "kvx_preloader_destroy": (ctypes.c_int, [c_vp]),
    "kvx_pinned_alloc": (ctypes.c_int, [c_i64, ctypes.POINTER(c_vp)]),
    "kvx_pinned_free": (ctypes.c_int, [c_vp]),
}

_lib = None


def lib():
    """Load libkvx.so; raise if it is not built (there is no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libkvx.so not found at {LIB_PATH}; build it with "
                               "__graft_entry__.build() (there is no non-HIP fallback)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(handle, name)
            f.restype = res
            f.argtypes = args
        _lib = handle
    return _lib
