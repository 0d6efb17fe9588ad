"""Element-wise oracle (O1) for gather and scatter, in plain Python loops.

TEST INFRASTRUCTURE ONLY; for tiny shapes. Written independently of the C
slab oracle (kvx_oracle.c): it walks every (chunk, layer, K|V, token, head)
and moves one head's vector of head_dim words at a time, computing each
index from the element-level statement of the mapping:

    packed token t of chunk c, layer l, K|V kv, head h, dim d
      <->  cache[l][kv][ block_table[c*bpc + t // block_size] ][ t % block_size ][h][d]

with the readings listed in kvx_oracle.c (layer-major chunk, K before V,
compact last chunk). Blocks of fixed token count: Sec. 2.1; storage blocks
grouping several GPU blocks: Sec. 6.4.

Arrays: ``k[l]`` and ``v[l]`` are numpy arrays of shape
[num_blocks, block_size, kv_heads, head_dim] with an unsigned integer dtype of
the element width, so values are moved as raw words.
"""
from __future__ import annotations

import numpy as np


def _check(k, l0, l1, block_table, chunk_tokens):
    nb, bs, _, _ = k[0].shape
    if chunk_tokens <= 0 or chunk_tokens % bs:
        raise ValueError("chunk_tokens must be a positive multiple of block_size")
    if not 0 <= l0 <= l1 <= len(k):
        raise ValueError("bad layer range")
    for b in block_table:
        if not 0 <= int(b) < nb:
            raise IndexError(f"block id {b} out of range")


def gather_elementwise(k, v, l0, l1, block_table, chunk_tokens):
    """Return the packed image as a flat array of element words."""
    _check(k, l0, l1, block_table, chunk_tokens)
    nb, bs, heads, dim = k[0].shape
    n = len(block_table)
    bpc = chunk_tokens // bs
    lr = l1 - l0
    out = np.zeros(n * bs * lr * 2 * heads * dim, dtype=k[0].dtype)
    chunk_elems = lr * 2 * chunk_tokens * heads * dim
    c = 0
    while c * bpc < n:
        nc = min(bpc, n - c * bpc)
        tc = nc * bs
        for li in range(lr):
            for kv, tensors in ((0, k), (1, v)):
                src = tensors[l0 + li]
                for t in range(tc):
                    blk = int(block_table[c * bpc + t // bs])
                    slot = t % bs
                    for h in range(heads):
                        pos = c * chunk_elems + ((li * 2 + kv) * tc + t) * heads * dim + h * dim
                        for d in range(dim):
                            out[pos + d] = src[blk, slot, h, d]
        c += 1
    return out


def scatter_elementwise(k, v, l0, l1, block_table, chunk_tokens, packed):
    """Write the packed image (flat element words) into k / v in place."""
    _check(k, l0, l1, block_table, chunk_tokens)
    nb, bs, heads, dim = k[0].shape
    n = len(block_table)
    bpc = chunk_tokens // bs
    lr = l1 - l0
    if packed.size != n * bs * lr * 2 * heads * dim:
        raise ValueError("packed image has the wrong size")
    chunk_elems = lr * 2 * chunk_tokens * heads * dim
    c = 0
    while c * bpc < n:
        nc = min(bpc, n - c * bpc)
        tc = nc * bs
        for li in range(lr):
            for kv, tensors in ((0, k), (1, v)):
                dst = tensors[l0 + li]
                for t in range(tc):
                    blk = int(block_table[c * bpc + t // bs])
                    slot = t % bs
                    for h in range(heads):
                        pos = c * chunk_elems + ((li * 2 + kv) * tc + t) * heads * dim + h * dim
                        for d in range(dim):
                            dst[blk, slot, h, d] = packed[pos + d]
        c += 1
