"""Oracle for the step planner: prefix identity of blocks and chunk dedupe.

TEST INFRASTRUCTURE ONLY.

Written from the definitions, with exact keys instead of hashes:
  * Sec. 2.1: a full block is identified by its tokens together with the
    identity of the block before it, i.e. by the whole token prefix up to its
    end; lookup walks blocks from the start of the prompt until the first
    block not in the cache; a trailing partial block is never cached.
    Here the key of block b is the tuple of all tokens through block b.
  * Sec. 6.5: identical prefixes share one read, so a step restores each
    distinct chunk once; a chunk is identified by the key of its last block.

Pinned by the worked prefix-tree example of Sec. 2.1 (Fig. "Prefix-hash
chaining"), stored in tests/golden/prefix_hash_example.json.
"""
from __future__ import annotations


def block_keys(tokens, block_size):
    """Exact key of every full block: the token prefix through that block."""
    toks = tuple(int(t) for t in tokens)
    return [toks[:(b + 1) * block_size] for b in range(len(toks) // block_size)]


def matched_blocks(tokens, block_size, cached):
    """Blocks reused from `cached` (a set of block keys): walk until the first miss."""
    n = 0
    for key in block_keys(tokens, block_size):
        if key not in cached:
            break
        n += 1
    return n


def chunk_keys(tokens, block_size, chunk_tokens):
    """(key, n_blocks) of every chunk of the full blocks of a prompt."""
    keys = block_keys(tokens, block_size)
    bpc = chunk_tokens // block_size
    out = []
    for first in range(0, len(keys), bpc):
        last = min(first + bpc, len(keys)) - 1
        out.append((keys[last], last - first + 1))
    return out


def dedupe(keys):
    """first_of[i] = index of the first occurrence of keys[i]."""
    seen = {}
    return [seen.setdefault(k, i) for i, k in enumerate(keys)]


def plan_step(requests, block_size, chunk_tokens, gate_tokens=0):
    """The chunk lists of one batched engine step, from exact keys.

    requests: objects with .tokens (a whole number of blocks), .resident (per
    chunk, whether the GPU holds it) and .new_blocks. Definitions:
      * every chunk of every prompt, in request order, keyed by chunk_keys;
        a chunk's residency is that of its first occurrence (the engine's
        lookup finds one copy of a chunk);
      * Sec. 6.6 gate (breakeven.plan_gate): a request loads when the tokens
        of its chunks the GPU does not hold reach gate_tokens;
      * Sec. 6.5: a missing chunk is restored once, the first time a loading
        request needs it, with that request as its origin; restore block
        table slices follow in restore order;
      * a missing chunk no loading request needs is recomputed, for every
        request that needs it;
      * Sec. 6.4 store path: each request's new blocks, cut into chunks of at
        most chunk_tokens / block_size blocks, in request order.
    Returns a dict; restore entries are (key, n_blocks, (request, chunk),
    bt_offset), offload entries (request, chunk, n_blocks, bt_offset,
    new_first), chunk_states per (request, chunk) ("resident",),
    ("restore", index) or ("recompute",).
    """
    from .breakeven import plan_gate

    bpc = chunk_tokens // block_size
    chunks = []  # (request, chunk index, key, n_blocks)
    for ri, r in enumerate(requests):
        ck = chunk_keys(r.tokens, block_size, chunk_tokens)
        assert len(ck) == len(r.resident), "one residency flag per chunk"
        for k, (key, nb) in enumerate(ck):
            chunks.append((ri, k, key, nb))
    first = dedupe([c[2] for c in chunks])
    resident = {}
    for i, (ri, k, key, nb) in enumerate(chunks):
        if first[i] == i:
            resident[key] = bool(requests[ri].resident[k])
    load = [0] * len(requests)
    for ri, k, key, nb in chunks:
        if not resident[key]:
            load[ri] += nb
    loads = plan_gate(load, block_size, gate_tokens)
    restore, index_of, bt = [], {}, 0
    for ri, k, key, nb in chunks:
        if not resident[key] and loads[ri] and key not in index_of:
            index_of[key] = len(restore)
            restore.append((key, nb, (ri, k), bt))
            bt += nb
    states, recompute = [], 0
    for ri, k, key, nb in chunks:
        if resident[key]:
            states.append(("resident",))
        elif key in index_of:
            states.append(("restore", index_of[key]))
        else:
            states.append(("recompute",))
            recompute += nb
    offload, obt = [], 0
    for ri, r in enumerate(requests):
        c = 0
        for first_new in range(0, r.new_blocks, bpc):
            nb = min(bpc, r.new_blocks - first_new)
            offload.append((ri, c, nb, obt, first_new))
            obt += nb
            c += 1
    return {"restore": restore, "offload": offload, "chunk_states": states,
            "resident_hits": sum(1 for v in resident.values() if v),
            "restore_blocks": bt, "offload_blocks": obt,
            "declined": [ri for ri in range(len(requests)) if not loads[ri]],
            "recompute_blocks": recompute}
