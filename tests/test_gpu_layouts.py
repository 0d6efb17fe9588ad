"""GPU parity for the cache layouts that reorder a slab (moved head by head:
HND rows directly, paged attention through LDS): KVX_LAYOUT_HND
([head][token][dim]) and KVX_LAYOUT_PAGED_ATTN (keys in 16-byte groups
[head][dim/x][token][x], values [head][dim][token]), against the oracle, which
moves elements through the layout's index function. Heads of up to 256
vectors take the one-vector-per-thread kernels, larger ones the
twelve-vector kernels."""
import numpy as np
import pytest

import kvsynth
import oracle
from kvtest_util import (Filled, device_cache, first_mismatch, host_mirror, mirror_slabs,
                         read_slabs, seeded_ids, to_host)

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
HND, PA = oracle.LAYOUT_HND, oracle.LAYOUT_PAGED_ATTN


def _bt(ids):
    return torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(DEV)


def _check():
    torch.cuda.synchronize()
    kvx.kvx_check()


CASES = [
    # (layout, layers, BS, heads, dim, elem, l0, l1, n, chunk_tokens)
    (HND, 3, 16, 2, 64, 2, 0, 3, 13, 64),
    (HND, 2, 16, 8, 128, 2, 0, 2, 9, 32),     # 32 KiB slabs
    (HND, 2, 8, 3, 32, 4, 1, 2, 7, 24),
    (PA, 3, 16, 2, 64, 2, 0, 3, 13, 64),
    (PA, 2, 16, 8, 128, 2, 0, 2, 9, 32),      # the 8B/70B slab shape
    (PA, 2, 8, 2, 32, 4, 0, 2, 11, 16),       # 4-byte elements (x = 4)
    (PA, 2, 16, 2, 32, 1, 1, 2, 5, 48),       # 1-byte elements (x = 16)
    (PA, 2, 4, 1, 16, 8, 0, 2, 6, 8),         # 8-byte elements (x = 2)
    (PA, 2, 5, 2, 16, 2, 0, 2, 7, 15),        # block size not a multiple of x
    (PA, 2, 16, 12, 128, 2, 0, 2, 5, 32),     # 48 KiB slabs, the largest transposed
    (HND, 2, 16, 12, 128, 2, 0, 2, 5, 32),
    (PA, 2, 32, 4, 128, 2, 0, 2, 6, 64),      # 4 token vectors per value row
    (PA, 2, 8, 2, 64, 2, 0, 2, 9, 16),        # 1 token vector per value row
    (PA, 2, 24, 2, 64, 2, 0, 2, 7, 48),       # 3 token vectors per value row
    (PA, 2, 6, 3, 32, 2, 0, 2, 8, 12),        # even block size, not a multiple of 8
    (PA, 2, 16, 16, 96, 1, 0, 2, 5, 32),      # 1-byte elements, 24 KiB slabs
    (PA, 2, 1, 8, 64, 2, 0, 2, 9, 3),         # one token per block
    (PA, 2, 3, 5, 40, 2, 0, 2, 7, 9),         # odd block size and head count
    (HND, 2, 32, 2, 256, 2, 0, 2, 6, 64),     # heads of 1,024 vectors (several per thread)
    (PA, 2, 16, 1, 1536, 2, 0, 2, 5, 32),     # one 48 KiB head: 12 vectors per thread
    (HND, 2, 96, 1, 256, 2, 0, 2, 4, 96),     # one 48 KiB head, HND
]


@pytest.mark.parametrize("case", CASES, ids=[f"c{i}" for i in range(len(CASES))])
def test_layout_gather_scatter_bit_exact(case):
    layout, L, BS, H, D, e, l0, l1, n, ct = case
    NB = 3 * n + 4
    s = oracle.Shape(L, NB, BS, H, D, e, layout)
    seed = 200 + n + layout
    bt_src, bt_dst = seeded_ids(seed, NB, n, n)
    fill = Filled(seed, kvsynth.ROLE_SRC, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(NB))
    expect = oracle.gather(s, *mirror, l0, l1, bt_src, ct)
    dst = torch.full((expect.size + 4096,), 0xA5, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_blocks(cache, l0, l1, _bt(bt_src), n, ct, dst)
    _check()
    got = to_host(dst)
    bad = first_mismatch(got[:expect.size], expect)
    assert bad is None, f"gather differs at byte {bad}"
    assert (got[expect.size:] == 0xA5).all()
    kvx.kvx_scatter_blocks(cache, l0, l1, _bt(bt_dst), n, ct, dst)
    _check()
    oracle.scatter(s, *mirror, l0, l1, bt_dst, ct, expect)
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"


@pytest.mark.parametrize("layout,heads,dim", [(HND, 2, 64), (PA, 2, 64), (HND, 1, 128),
                                              (PA, 1, 128), (PA, 4, 32)],
                         ids=["hnd", "paged_attn", "hnd_one_head", "paged_attn_one_head",
                              "paged_attn_four_heads"])
def test_layout_ordered_scatter_and_chunk_lists(layout, heads, dim):
    """Large scatters (>= 1024 blocks: destination order, or with one head
    the default layout's linear image-order walk; paged-attention heads on 256
    threads, or on 128 threads x 2 vectors with four heads or more) and the
    chunk-list path (ring restore and offload) in a reordering layout."""
    s = oracle.Shape(2, 4000, 16, heads, dim, 2, layout)
    n = 1300
    seed = 210 + layout + heads
    walk = kvx.kvx_copy_walk(kvx.shape_only_cache(2, 4000, 16, heads, dim, 2, layout), 0, 2, n,
                             64, False)
    assert (walk["ordered"], walk["linear"]) == ((0, 1) if heads == 1 else (1, 0))
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, n, n)
    fill = Filled(seed, kvsynth.ROLE_SRC, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    expect = oracle.gather(s, *mirror, 0, 2, bt_src, 64)
    dst = torch.empty(expect.size, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_blocks(cache, 0, 2, _bt(bt_src), n, 64, dst)
    kvx.kvx_scatter_blocks(cache, 0, 2, _bt(bt_dst), n, 64, dst)
    _check()
    assert first_mismatch(to_host(dst), expect) is None
    oracle.scatter(s, *mirror, 0, 2, bt_dst, 64, expect)
    for l in range(2):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l])
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l])
    # ring: restore an image into the source blocks, offload it back out
    image = kvsynth.host_bytes(expect.size, seed, kvsynth.image_stream(9), mode=kvsynth.MODE_RAW)
    ring = kvx.StagingRing(DEV, 3, 48 << 10)
    try:
        ring.bind(cache, 0, 2, n, 64, image, fill_threads=2)
        kvx.kvx_restore_from_staging(ring, _bt(bt_src))
        _check()
        per_block = oracle.packed_bytes(s, 0, 2, 1)
        sinks = [(np.zeros(min(4, n - b) * per_block, np.uint8), b, min(4, n - b))
                 for b in range(0, n, 4)]
        ring.bind_offload(cache, 0, 2, 64, sinks, drain_threads=2)
        kvx.kvx_offload_to_staging(ring, _bt(bt_src))
        _check()
    finally:
        ring.close()
    assert np.array_equal(np.concatenate([x[0] for x in sinks]), image)
    oracle.restore(s, *mirror, 0, 2, bt_src, 64, image)
    for l in range(2):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l])
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l])


def test_paged_attn_80k_prefix_sampled_against_oracle():
    """The 80k-token prefix of the 8B-shaped cache in the paged-attention
    layout: every gathered byte checked by a round trip through a scatter into
    fresh blocks and a second gather, and a seeded sample of chunks against the
    oracle (which moves element by element)."""
    s = oracle.Shape(32, 20000, 16, 8, 128, 2, PA)
    seed = 7
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, 5000, 5000)
    fill = Filled(seed, kvsynth.ROLE_SRC)
    cache = device_cache(s, fill, DEV)
    nbytes = oracle.packed_bytes(s, 0, 32, 5000)
    a = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    b = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_blocks(cache, 0, 32, _bt(bt_src), 5000, 256, a)
    kvx.kvx_scatter_blocks(cache, 0, 32, _bt(bt_dst), 5000, 256, a)
    kvx.kvx_gather_blocks(cache, 0, 32, _bt(bt_dst), 5000, 256, b)
    _check()
    assert torch.equal(a, b)
    chunks = np.random.default_rng(3).choice(5000 // 16, 12, replace=False)
    per_chunk = oracle.packed_bytes(s, 0, 32, 16)
    for c in chunks:
        ids = bt_src[c * 16:(c + 1) * 16]
        mirror = host_mirror(s, fill, ids)
        exp = oracle.gather(s, *mirror, 0, 32, ids, 256)
        got = a[c * per_chunk:(c + 1) * per_chunk].cpu().numpy()
        assert np.array_equal(got, exp), f"chunk {c} differs"
    # and the scattered blocks on a sample of layers, against the oracle scatter
    dmirror = oracle.new_mirror(s)
    oracle.scatter(s, *dmirror, 0, 32, bt_dst[:64], 256, a[:4 * per_chunk].cpu().numpy())
    for l in (0, 13, 31):
        for kv in (0, 1):
            assert np.array_equal(read_slabs(cache, l, kv, bt_dst[:64]),
                                  mirror_slabs(dmirror, s, l, kv, bt_dst[:64]))
