"""Shared helpers for the parity tests: workload shapes, seeded block ids,
device caches filled by the generator, sparse host mirrors for the oracle,
and readers that pull cache slabs back to the host."""
from __future__ import annotations

import dataclasses

import numpy as np

import kvsynth
import oracle
from oracle import Shape

# Workload shapes (bf16 elements): tiny, Llama-3-8B-shaped, Llama-70B-shaped.
TINY = Shape(2, 64, 16, 2, 64, 2)
L8B = dict(num_layers=32, block_size=16, kv_heads=8, head_dim=128, elem_bytes=2)
L70B = dict(num_layers=80, block_size=16, kv_heads=8, head_dim=128, elem_bytes=2)


def shape_8b(num_blocks: int) -> Shape:
    return Shape(num_blocks=num_blocks, **L8B)


def shape_70b(num_blocks: int) -> Shape:
    return Shape(num_blocks=num_blocks, **L70B)


def seeded_ids(seed: int, pool: int, *counts):
    """Disjoint random block ids: a seeded permutation of the pool, cut in order."""
    perm = np.random.default_rng(seed).permutation(pool).astype(np.int32)
    out, at = [], 0
    for c in counts:
        out.append(perm[at:at + c].copy())
        at += c
    return out


@dataclasses.dataclass
class Filled:
    seed: int
    role: int
    mode: int = kvsynth.MODE_NORMAL_BF16


def torch_dtype(elem_bytes: int):
    import torch

    return {1: torch.uint8, 2: torch.bfloat16, 4: torch.int32, 8: torch.int64}[elem_bytes]


def device_cache(shape: Shape, fill: Filled | None, device):
    """Allocate a PagedKVCache and fill every tensor from the generator."""
    import paper_2609_11744_amd as kvx

    cache = kvx.PagedKVCache.allocate(shape.num_layers, shape.num_blocks, shape.block_size,
                                      shape.kv_heads, shape.head_dim,
                                      torch_dtype(shape.elem_bytes), device, layout=shape.layout)
    if fill is not None:
        for l in range(shape.num_layers):
            kvsynth.fill_device(cache.k[l], fill.seed, kvsynth.cache_stream(fill.role, l, 0),
                                mode=fill.mode)
            kvsynth.fill_device(cache.v[l], fill.seed, kvsynth.cache_stream(fill.role, l, 1),
                                mode=fill.mode)
    return cache


def host_mirror(shape: Shape, fill: Filled, block_ids, layers=None, threads=16):
    """Host mirror (lazily zeroed arrays) holding generator content for the
    given blocks only: the same bytes the device fill put there."""
    k, v = oracle.new_mirror(shape)
    u = shape.slab_bytes
    offs = np.asarray(block_ids, dtype=np.uint64) * np.uint64(u)
    for l in (range(shape.num_layers) if layers is None else layers):
        kvsynth.fill_ranges(k[l], offs, u, fill.seed, kvsynth.cache_stream(fill.role, l, 0),
                            mode=fill.mode, threads=threads)
        kvsynth.fill_ranges(v[l], offs, u, fill.seed, kvsynth.cache_stream(fill.role, l, 1),
                            mode=fill.mode, threads=threads)
    return k, v


def read_slabs(cache, layer: int, kv: int, ids) -> np.ndarray:
    """Bytes of the given blocks of one cache tensor, as [len(ids), slab] uint8."""
    import torch

    t = cache.k[layer] if kv == 0 else cache.v[layer]
    idx = torch.as_tensor(np.asarray(ids, dtype=np.int64), device=t.device)
    rows = t.index_select(0, idx).contiguous().view(torch.uint8).cpu().numpy()
    return rows.reshape(len(ids), -1)


def mirror_slabs(mirror, shape: Shape, layer: int, kv: int, ids) -> np.ndarray:
    u = shape.slab_bytes
    buf = mirror[kv][layer].reshape(shape.num_blocks, u)
    return buf[np.asarray(ids, dtype=np.int64)]


def to_host(t) -> np.ndarray:
    import torch

    return t.contiguous().view(torch.uint8).cpu().numpy().ravel()


def first_mismatch(a: np.ndarray, b: np.ndarray, step: int = 1 << 28):
    """Index of the first differing byte of two equal-length arrays, or None.
    Compares in bounded pieces so multi-GB images need no full-size temporaries."""
    a, b = a.ravel(), b.ravel()
    if a.size != b.size:
        return min(a.size, b.size)
    for s in range(0, a.size, step):
        x, y = a[s:s + step], b[s:s + step]
        if not np.array_equal(x, y):
            return s + int(np.flatnonzero(x != y)[0])
    return None


def generator_tensor(shape: Shape, fill: Filled, layer: int, kv: int, threads=16) -> np.ndarray:
    """The whole cache tensor (layer, K|V) as the generator filled it."""
    buf = np.empty(shape.num_blocks * shape.slab_bytes, dtype=np.uint8)
    kvsynth.fill_host(buf, fill.seed, kvsynth.cache_stream(fill.role, layer, kv), mode=fill.mode,
                      threads=threads)
    return buf


def oracle_layer_after_scatters(shape: Shape, fill: Filled, layer: int, chunks,
                                chunk_tokens: int):
    """Expected cache tensors (layer, K) and (layer, V) after scattering a list
    of chunk images into a cache the generator filled: the generator's content
    of the whole tensor, then the oracle scatter of each chunk restricted to
    this layer. chunks: (image, block ids, l0) with image the packed image of
    one chunk (len(ids) blocks) over layers [l0, ...); a chunk's layer-l part
    is one contiguous run of its K then V slabs (the layer-major chunk
    layout), which is itself that chunk's image over [layer, layer + 1)
    (the layer-decomposition pin; tests/test_kvtest_util.py checks this
    function against the oracle's scatter of the whole chunks)."""
    dummy = np.zeros(16, dtype=np.uint8)
    k = [dummy] * shape.num_layers
    v = [dummy] * shape.num_layers
    k[layer] = generator_tensor(shape, fill, layer, 0)
    v[layer] = generator_tensor(shape, fill, layer, 1)
    u = shape.slab_bytes
    for img, ids, l0 in chunks:
        n = len(ids)
        part = img[(layer - l0) * 2 * n * u:(layer - l0 + 1) * 2 * n * u]
        oracle.scatter(shape, k, v, layer, layer + 1, ids, chunk_tokens, part)
    return k[layer], v[layer]


def check_layer_after_scatters(cache, shape: Shape, fill: Filled, layer: int, chunks,
                               chunk_tokens: int, what: str) -> None:
    """Every byte of cache tensors (layer, K) and (layer, V) on the device
    against oracle_layer_after_scatters: the scattered slabs, and every other
    block unchanged."""
    u = shape.slab_bytes
    exp = oracle_layer_after_scatters(shape, fill, layer, chunks, chunk_tokens)
    for kv in (0, 1):
        got = to_host((cache.k if kv == 0 else cache.v)[layer])
        bad = first_mismatch(got, exp[kv])
        if bad is not None:
            raise AssertionError(f"{what}: layer {layer} kv {kv} differs at byte {bad} "
                                 f"(block {bad // u})")
