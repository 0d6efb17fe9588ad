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
