"""Seeded batched-request workload: token prompts that share prefixes along a
random prefix tree, as in multi-turn or document-QA serving.

Recipe (per request r = 0 .. n-1, one seeded numpy Generator):
  * prompt length L_r = block_size * floor(exp(U(ln lo, ln hi)) / block_size)
    tokens (log-uniform between lo and hi, whole blocks);
  * a child cap b_r ~ U{1..max_children};
  * a parent p drawn uniformly among earlier requests with fewer than b_p
    children; none left -> r is a new root;
  * a shared prefix s_r = g * floor(U(0,1) * min(L_r, L_p) / g) tokens, copied
    from the parent, with g = chunk_tokens (share="chunk": whole transfer
    chunks) or g = block_size (share="block": a shared prefix may end inside a
    chunk, as when a multi-turn prompt extends the previous turn); the rest of
    the prompt is fresh random token ids;
  * each chunk of the tree (identified by the request that introduced it and
    its index) is GPU-resident with probability `resident_p`; requests that
    share a chunk see the same flag. A child's chunk k is its parent's chunk k
    when it ends at the same block as the parent's and inside the shared
    prefix (same last block, same tokens through it); otherwise it is a new
    chunk of the child, also when it only extends a partial chunk of the
    parent;
  * q_r ~ U{new_lo..new_hi} newly computed blocks to offload.

This module only draws inputs; how chunks are identified, deduplicated and
moved is the library's business.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


@dataclasses.dataclass
class Request:
    tokens: np.ndarray          # int32 prompt tokens, a whole number of blocks
    parent: int                 # -1 for a root
    shared_tokens: int          # prefix copied from the parent
    chunk_owner: list           # per chunk: (request that introduced it, chunk index)
    resident: np.ndarray        # per chunk: GPU-resident (bool)
    new_blocks: int             # newly computed blocks to offload


def make_requests(seed: int, n: int = 64, block_size: int = 16, chunk_tokens: int = 256,
                  lo: int = 1024, hi: int = 32768, max_children: int = 4,
                  resident_p: float = 0.5, new_lo: int = 16, new_hi: int = 64,
                  share: str = "chunk"):
    if share not in ("chunk", "block"):
        raise ValueError("share must be 'chunk' or 'block'")
    grain = chunk_tokens if share == "chunk" else block_size
    rng = np.random.default_rng(seed)
    reqs: list[Request] = []
    cap, children = [], []
    owner_resident = {}
    for r in range(n):
        length = block_size * int(math.exp(rng.uniform(math.log(lo), math.log(hi))) // block_size)
        cap.append(int(rng.integers(1, max_children + 1)))
        children.append(0)
        cands = [p for p in range(r) if children[p] < cap[p]]
        n_chunks = (length + chunk_tokens - 1) // chunk_tokens
        if cands:
            p = int(rng.choice(cands))
            children[p] += 1
            plen = len(reqs[p].tokens)
            shared = grain * int(rng.uniform() * min(length, plen) // grain)
            fresh = rng.integers(0, 2**31 - 1, size=length - shared, dtype=np.int64)
            tokens = np.concatenate([reqs[p].tokens[:shared], fresh.astype(np.int32)])
            owners = []
            for k in range(n_chunks):
                end = min(chunk_tokens * (k + 1), length)      # this chunk's last token + 1
                pend = min(chunk_tokens * (k + 1), plen)       # the parent's chunk k
                same = end <= shared and end == pend
                owners.append(reqs[p].chunk_owner[k] if same else (r, k))
        else:
            p, shared = -1, 0
            tokens = rng.integers(0, 2**31 - 1, size=length, dtype=np.int64).astype(np.int32)
            owners = [(r, k) for k in range(n_chunks)]
        for o in owners:
            if o not in owner_resident:
                owner_resident[o] = bool(rng.uniform() < resident_p)
        resident = np.array([owner_resident[o] for o in owners], dtype=bool)
        new_blocks = int(rng.integers(new_lo, new_hi + 1))
        reqs.append(Request(tokens, p, shared, owners, resident, new_blocks))
    return reqs


def chunk_stream(owner) -> int:
    """Generator stream id of a chunk's stored KV image."""
    r, k = owner
    return (0x4348 << 48) | (r << 24) | k


def new_block_stream(request: int) -> int:
    return (0x4E42 << 48) | request
