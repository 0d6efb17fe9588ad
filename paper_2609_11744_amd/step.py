"""Step planning for a batch of requests: marshalling over kvx_plan_step.

One engine step moves two chunk lists (computed by the library, include/kvx.h):
  * the restore list: every distinct chunk that some loading request needs
    and the GPU does not hold, once (identical prefixes share one read and one
    staging slot, Sec. 6.5);
  * the offload list: every request's newly computed blocks, cut into chunks
    (the store path, Sec. 6.4).
Chunks are identified by the prefix-hash chain of Sec. 2.1 (kvx_block_hashes:
the hash of a chunk's last full block covers the whole prefix through it).
With a gate threshold (the tier's break-even prefix, Sec. 6.6) a request whose
load is shorter declines it, and its missing chunks are recomputed unless
another request of the step loads them. The lists feed one fused chunk-list
copy per staging slot (kvx_ring_bind_chunks / kvx_ring_bind_offload).

A request is any object with
  tokens      int32 prompt tokens,
  resident    per chunk of the prompt: whether the GPU already holds it (the
              outcome of the engine's prefix-cache lookup),
  new_blocks  number of newly computed blocks to offload.
"""
from __future__ import annotations

import ctypes
import dataclasses

import numpy as np

from . import _native, _ok, kvx_block_hashes
from ._native import KvxStepOffload, KvxStepPlan, KvxStepRequest, KvxStepRestore

CHUNK_RESIDENT, CHUNK_RECOMPUTE = -1, -2


@dataclasses.dataclass
class RestoreChunk:
    key: int            # hash of the chunk's last block
    n_blocks: int
    origin: tuple       # (request, chunk index) of the first loading request needing it
    bt_offset: int      # first entry in the restore block table


@dataclasses.dataclass
class OffloadChunk:
    request: int
    chunk: int          # chunk index within the request's new blocks
    n_blocks: int
    bt_offset: int      # first entry in the offload block table
    new_first: int      # first new block of the request in this chunk


@dataclasses.dataclass
class StepPlan:
    restore: list
    offload: list
    resident_hits: int              # distinct chunks the GPU already holds
    request_chunks: list            # per (request, chunk): ("resident",), ("restore", i)
                                    # or ("recompute",)
    restore_blocks: int
    offload_blocks: int
    declined: list = dataclasses.field(default_factory=list)  # requests under the gate
    recompute_blocks: int = 0       # blocks of declined loads that no one restores


def plan_step(requests, block_size: int, chunk_tokens: int, gate_tokens: int = 0) -> StepPlan:
    keep = []
    arr = (KvxStepRequest * max(len(requests), 1))()
    for i, r in enumerate(requests):
        h = np.ascontiguousarray(kvx_block_hashes(r.tokens, block_size), dtype=np.uint64)
        res = np.ascontiguousarray(np.asarray(r.resident, dtype=bool).astype(np.uint8))
        keep += [h, res]
        arr[i] = KvxStepRequest(h.ctypes.data if h.size else None,
                                res.ctypes.data if res.size else None, h.size, res.size,
                                int(r.new_blocks), 0)
    lib = _native.lib()
    p = KvxStepPlan()
    _ok(lib.kvx_plan_step(arr, len(requests), block_size, chunk_tokens, gate_tokens,
                          ctypes.byref(p)), "kvx_plan_step")
    rs = (KvxStepRestore * max(p.n_restore, 1))()
    of = (KvxStepOffload * max(p.n_offload, 1))()
    cs = (ctypes.c_int32 * max(p.n_chunk_states, 1))()
    dc = (ctypes.c_int32 * max(p.n_declined, 1))()
    p.restore, p.offload, p.chunk_states, p.declined = rs, of, cs, dc
    p.restore_cap, p.offload_cap = max(p.n_restore, 1), max(p.n_offload, 1)
    p.chunk_states_cap, p.declined_cap = max(p.n_chunk_states, 1), max(p.n_declined, 1)
    _ok(lib.kvx_plan_step(arr, len(requests), block_size, chunk_tokens, gate_tokens,
                          ctypes.byref(p)), "kvx_plan_step")
    restore = [RestoreChunk(rs[i].key, rs[i].n_blocks, (rs[i].request, rs[i].chunk),
                            rs[i].bt_offset) for i in range(p.n_restore)]
    offload = [OffloadChunk(of[i].request, of[i].chunk, of[i].n_blocks, of[i].bt_offset,
                            of[i].new_first) for i in range(p.n_offload)]
    states = [("resident",) if v == CHUNK_RESIDENT else ("recompute",) if v == CHUNK_RECOMPUTE
              else ("restore", v) for v in cs[:p.n_chunk_states]]
    return StepPlan(restore, offload, p.resident_hits, states, p.restore_blocks,
                    p.offload_blocks, list(dc[:p.n_declined]), p.recompute_blocks)
