"""Step planning for a batch of requests (host side).

Turns a batch of prompts into the two chunk lists one engine step moves:
  * the restore list: every distinct chunk that some request needs and the
    GPU does not hold, once (identical prefixes share one read and one
    staging slot, Sec. 6.5);
  * the offload list: every request's newly computed blocks, cut into chunks
    (the store path, Sec. 6.4).
Chunks are identified by the prefix-hash chain of Sec. 2.1 (the hash of a
chunk's last full block covers the whole prefix through it), computed and
deduplicated by the library (kvx_block_hashes, kvx_dedupe_keys). The lists
feed one fused chunk-list copy per staging slot (kvx_ring_bind_chunks /
kvx_ring_bind_offload), which is how the ready mappings of several requests
move in one launch.

With a gate threshold (breakeven.break_even_tokens for the staging tier,
Sec. 6.6), a request whose load from the tier (its chunks the GPU does not
hold) is shorter than the threshold declines the load: its missing chunks are
recomputed by the engine, unless another request of the step loads them (a
chunk's KV depends only on its prefix, so a restored chunk serves every
request that shares it).

A request is any object with
  tokens      int32 prompt tokens (a whole number of blocks),
  resident    per chunk of the prompt: whether the GPU already holds it (the
              outcome of the engine's prefix-cache lookup),
  new_blocks  number of newly computed blocks to offload.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from . import kvx_block_hashes, kvx_dedupe_keys


@dataclasses.dataclass
class RestoreChunk:
    key: int            # hash of the chunk's last block
    n_blocks: int
    origin: tuple       # (request, chunk index) of its first occurrence
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
    request_chunks: list            # per (request, chunk): ("resident", key), ("restore", i)
                                    # or ("recompute", key)
    restore_blocks: int
    offload_blocks: int
    declined: list = dataclasses.field(default_factory=list)  # requests under the gate
    recompute_blocks: int = 0       # blocks of declined loads that no one restores


def plan_step(requests, block_size: int, chunk_tokens: int, gate_tokens: int = 0) -> StepPlan:
    if chunk_tokens % block_size:
        raise ValueError("chunk_tokens must be a multiple of block_size")
    bpc = chunk_tokens // block_size
    keys, nblocks, resident, origin = [], [], [], []
    for ri, r in enumerate(requests):
        h = kvx_block_hashes(r.tokens, block_size)
        n_chunks = (h.size + bpc - 1) // bpc
        if len(r.resident) != n_chunks:
            raise ValueError(f"request {ri}: {len(r.resident)} residency flags for "
                             f"{n_chunks} chunks")
        for k in range(n_chunks):
            last = min((k + 1) * bpc, h.size) - 1
            keys.append(int(h[last]))
            nblocks.append(last - k * bpc + 1)
            resident.append(bool(r.resident[k]))
            origin.append((ri, k))
    first_of = kvx_dedupe_keys(np.array(keys, dtype=np.uint64)) if keys else np.zeros(0, np.int32)
    load_blocks = [0] * len(requests)  # blocks each request would load from the tier
    for i in range(len(keys)):
        if not resident[int(first_of[i])]:
            load_blocks[origin[i][0]] += nblocks[i]
    accepts = [lb * block_size >= gate_tokens for lb in load_blocks]
    declined = [ri for ri, lb in enumerate(load_blocks) if lb and not accepts[ri]]
    restore, index_of, bt = [], {}, 0
    hits = sum(1 for i in range(len(keys)) if first_of[i] == i and resident[i])
    for i in range(len(keys)):
        j = int(first_of[i])
        if resident[j] or j in index_of or not accepts[origin[i][0]]:
            continue
        index_of[j] = len(restore)
        restore.append(RestoreChunk(keys[i], nblocks[i], origin[i], bt))
        bt += nblocks[i]
    request_chunks, recompute = [], 0
    for i in range(len(keys)):
        j = int(first_of[i])
        if resident[j]:
            request_chunks.append(("resident", keys[i]))
        elif j in index_of:
            request_chunks.append(("restore", index_of[j]))
        else:
            request_chunks.append(("recompute", keys[i]))
            recompute += nblocks[i]
    offload, obt = [], 0
    for ri, r in enumerate(requests):
        for c, first in enumerate(range(0, r.new_blocks, bpc)):
            nb = min(bpc, r.new_blocks - first)
            offload.append(OffloadChunk(ri, c, nb, obt, first))
            obt += nb
    return StepPlan(restore, offload, hits, request_chunks, bt, obt, declined, recompute)
