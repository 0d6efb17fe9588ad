"""GPU parity: the HIP path through the C ABI, bit-exact against the CPU oracle
on the same seeded inputs.

Inputs come from the generator (kvsynth): device caches are filled on the GPU
and the oracle's host mirrors are regenerated from the same streams, so no
oracle input is ever read back from the device. Results are compared byte for
byte (integer views; never float comparisons, so NaN payloads and -0 count).
"""
import numpy as np
import pytest

import kvsynth
import oracle
from kvtest_util import (TINY, Filled, device_cache, first_mismatch, host_mirror, mirror_slabs,
                         read_slabs, seeded_ids, shape_8b, to_host)

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
SRC = lambda seed, mode=kvsynth.MODE_NORMAL_BF16: Filled(seed, kvsynth.ROLE_SRC, mode)  # noqa: E731
BKG = lambda seed, mode=kvsynth.MODE_NORMAL_BF16: Filled(seed, kvsynth.ROLE_DST, mode)  # noqa: E731


def _sync_check():
    torch.cuda.synchronize()
    kvx.kvx_check()


def _bt(ids):
    return torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(DEV)


def _packed(nbytes):
    return torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)


def _compare_paged(cache, shape, expect_mirror, layers, ids, what):
    for l in layers:
        for kv in (0, 1):
            got = read_slabs(cache, l, kv, ids)
            exp = mirror_slabs(expect_mirror, shape, l, kv, ids)
            bad = first_mismatch(got.ravel(), exp.ravel())
            assert bad is None, f"{what}: layer {l} kv {kv} differs at byte {bad}"


def _untouched_equal(cache, before, shape, layers_touched, ids_touched, what):
    all_ids = np.arange(shape.num_blocks)
    keep = torch.from_numpy(np.setdiff1d(all_ids, ids_touched)).to(DEV)
    for l in range(shape.num_layers):
        for kv in (0, 1):
            a = (cache.k if kv == 0 else cache.v)[l].view(torch.uint8)
            b = before[kv][l].view(torch.uint8)
            if l in layers_touched:
                ok = torch.equal(a.index_select(0, keep), b.index_select(0, keep))
            else:
                ok = torch.equal(a, b)
            assert ok, f"{what}: bytes outside the named slabs changed (layer {l} kv {kv})"


def _clone(cache):
    return ([t.clone() for t in cache.k], [t.clone() for t in cache.v])


# ---- the generator itself on the device -------------------------------------

@pytest.mark.parametrize("mode", [kvsynth.MODE_NORMAL_BF16, kvsynth.MODE_RAW])
def test_device_generator_matches_host(mode):
    t = torch.empty(3 << 20, dtype=torch.uint8, device=DEV)
    kvsynth.fill_device(t, 4, 999, byte_offset=8 * 1000, mode=mode)
    torch.cuda.synchronize()
    host = kvsynth.host_bytes(3 << 20, 4, 999, byte_offset=8 * 1000, mode=mode)
    assert np.array_equal(to_host(t), host)


# ---- tiny workload (2 layers, 64 blocks of 16 tokens, 2 heads, dim 64) ----------

def test_tiny_gather_scatter_bit_exact():
    s, seed = TINY, 1
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, 16, 16)
    k, v = host_mirror(s, SRC(seed), range(s.num_blocks))
    cache = kvx.PagedKVCache.from_host(k, v, s.num_blocks, s.block_size, s.kv_heads, s.head_dim,
                                       torch.bfloat16, DEV)
    expect = oracle.gather(s, k, v, 0, 2, bt_src, 256)
    ev = lambda m: [oracle.element_view(a, s) for a in m]  # noqa: E731
    assert np.array_equal(expect.view(np.uint16),
                          oracle.gather_elementwise(ev(k), ev(v), 0, 2, bt_src, 256))
    dst = _packed(expect.size)
    kvx.kvx_gather_blocks(cache, 0, 2, _bt(bt_src), 16, 256, dst)
    _sync_check()
    assert np.array_equal(to_host(dst)[:expect.size], expect)

    kvx.kvx_scatter_blocks(cache, 0, 2, _bt(bt_dst), 16, 256, dst)
    _sync_check()
    oracle.scatter(s, k, v, 0, 2, bt_dst, 256, expect)
    for l in range(2):
        assert np.array_equal(to_host(cache.k[l]), k[l])
        assert np.array_equal(to_host(cache.v[l]), v[l])


# ---- Llama-8B-shaped, 8,192-token prefix -------------------------------------

def test_8b_8k_prefix_gather_then_scatter_to_fresh_blocks():
    s, seed = shape_8b(4096), 2
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, 512, 512)
    cache = device_cache(s, SRC(seed), DEV)
    mirror = host_mirror(s, SRC(seed), bt_src)
    expect = oracle.gather(s, *mirror, 0, 32, bt_src, 256)
    assert expect.size == 1 << 30
    dst = _packed(expect.size)
    kvx.kvx_gather_blocks(cache, 0, 32, _bt(bt_src), 512, 256, dst)
    _sync_check()
    got = to_host(dst)
    bad = first_mismatch(got, expect)
    assert bad is None, f"gather differs at byte {bad}"
    del got

    before = _clone(cache)
    kvx.kvx_scatter_blocks(cache, 0, 32, _bt(bt_dst), 512, 256, dst)
    _sync_check()
    oracle.scatter(s, *mirror, 0, 32, bt_dst, 256, expect)
    _compare_paged(cache, s, mirror, range(32), bt_dst, "scatter")
    _untouched_equal(cache, before, s, set(range(32)), bt_dst, "scatter")


# ---- edge cases ---------------------------------------------------------------

EDGE = [
    # (layers, NB, BS, heads, dim, elem, l0, l1, n, chunk_tokens)
    (3, 40, 16, 2, 64, 2, 0, 3, 13, 64),      # ragged last chunk (13 = 3*4 + 1)
    (3, 40, 16, 2, 64, 2, 1, 2, 7, 1024),     # chunk longer than the prefix, one layer
    (4, 50, 4, 1, 8, 2, 1, 4, 17, 12),        # 64-byte slabs (vector tail path)
    (2, 30, 16, 8, 128, 2, 0, 2, 9, 16),      # 32 KiB slabs, one block per chunk
    (2, 20, 32, 8, 128, 2, 0, 2, 5, 96),      # 64 KiB slabs (wider unrolled path)
    (2, 30, 16, 1, 16, 1, 0, 2, 11, 32),      # 1-byte elements
    (2, 30, 8, 2, 32, 4, 0, 2, 11, 16),       # 4-byte elements
    (2, 30, 8, 1, 32, 8, 0, 2, 6, 24),        # 8-byte elements
    (5, 25, 2, 1, 8, 2, 2, 5, 1, 2),          # a single block
    (130, 12, 2, 1, 8, 2, 1, 129, 5, 4),      # the largest layer range a call takes (128)
    (3, 40, 16, 3, 128, 2, 0, 3, 7, 48),      # 12 KiB slabs: 3 parts; chunks of 3, 3, 1 blocks
    (2, 3000, 16, 3, 128, 2, 0, 2, 1100, 80), # the same, ordered scatter (1,100 blocks, 5 per chunk)
]


@pytest.mark.parametrize("case", EDGE, ids=[f"e{i}" for i in range(len(EDGE))])
def test_edge_shapes_bit_exact(case):
    L, NB, BS, H, D, e, l0, l1, n, ct = case
    s = oracle.Shape(L, NB, BS, H, D, e)
    seed = 100 + n
    bt_src, bt_dst = seeded_ids(seed, NB, n, n)
    cache = device_cache(s, SRC(seed, kvsynth.MODE_RAW), DEV)
    mirror = host_mirror(s, SRC(seed, kvsynth.MODE_RAW), range(NB))
    expect = oracle.gather(s, *mirror, l0, l1, bt_src, ct)
    guard = 4096
    dst = torch.full((expect.size + guard,), 0xA5, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_blocks(cache, l0, l1, _bt(bt_src), n, ct, dst)
    _sync_check()
    got = to_host(dst)
    assert np.array_equal(got[:expect.size], expect)
    assert (got[expect.size:] == 0xA5).all(), "gather wrote past the packed image"

    kvx.kvx_scatter_blocks(cache, l0, l1, _bt(bt_dst), n, ct, dst)
    _sync_check()
    oracle.scatter(s, *mirror, l0, l1, bt_dst, ct, expect)
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"


def test_empty_prefix_and_empty_layer_range_are_noops():
    s = oracle.Shape(2, 16, 16, 2, 64, 2)
    cache = device_cache(s, SRC(5), DEV)
    before = _clone(cache)
    dst = torch.full((4096,), 7, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_blocks(cache, 0, 2, _bt([1, 2]), 0, 16, dst)
    kvx.kvx_scatter_blocks(cache, 1, 1, _bt([1, 2]), 2, 16, dst)
    _sync_check()
    assert (to_host(dst) == 7).all()
    _untouched_equal(cache, before, s, set(), np.array([], np.int64), "no-op")


def test_bad_block_id_is_reported_and_skipped():
    s = oracle.Shape(2, 32, 16, 2, 64, 2)
    cache = device_cache(s, BKG(6), DEV)
    before = _clone(cache)
    img = torch.from_numpy(kvsynth.host_bytes(oracle.packed_bytes(s, 0, 2, 4), 6, 5)).to(DEV)
    bad_table = [3, 32, 5, -1]  # 32 == num_blocks and -1 are out of range
    kvx.kvx_scatter_blocks(cache, 0, 2, _bt(bad_table), 4, 32, img)
    torch.cuda.synchronize()
    with pytest.raises(kvx.KvxError) as ei:
        kvx.kvx_check()
    assert ei.value.status == kvx.KVX_EBADBLOCK
    kvx.kvx_check()  # the flag is cleared by the check that reported it
    # only the two valid destinations may have changed
    _untouched_equal(cache, before, s, {0, 1}, np.array([3, 5]), "bad-id scatter")


def test_host_rejects_bad_arguments_without_launching():
    s = oracle.Shape(2, 32, 16, 2, 64, 2)
    cache = device_cache(s, None, DEV)
    dst = _packed(1 << 20)
    with pytest.raises(kvx.KvxError) as ei:
        kvx.kvx_gather_blocks(cache, 0, 2, _bt([1, 2]), 2, 24, dst)  # not a whole block
    assert ei.value.status == kvx.KVX_EINVAL
    with pytest.raises(kvx.KvxError):
        kvx.kvx_gather_blocks(cache, 0, 3, _bt([1, 2]), 2, 16, dst)  # layer range
    with pytest.raises(ValueError):
        kvx.kvx_gather_blocks(cache, 0, 2, _bt([1, 2]), 2, 16, _packed(64))  # too small
    with pytest.raises(kvx.KvxError):
        kvx.kvx_gather_blocks(cache, 0, 2, _bt([1, 2]), 2, 16, cache.k[1].view(torch.uint8))


# ---- staged restore at small sizes --------------------------------------------

RESTORE = [
    # (layers, NB, n, chunk_tokens, slots, slot_bytes, fill_threads)
    (3, 64, 21, 32, 2, 64 << 10, 1),       # whole-chunk pieces, 2 slots reused many times
    (3, 64, 21, 64, 3, 128 << 10, 3),      # ragged last chunk, several fill threads
    (4, 80, 19, 128, 2, 64 << 10, 2),      # chunk larger than a slot -> layer pieces
    (3, 64, 21, 32, 4, 96 << 10, 0),       # no staging copy: H2D straight from pinned image
]


@pytest.mark.parametrize("case", RESTORE, ids=[f"r{i}" for i in range(len(RESTORE))])
def test_staged_restore_equals_oracle_scatter_of_image(case):
    L, NB, n, ct, slots, slot_bytes, threads = case
    s = oracle.Shape(L, NB, 16, 2, 64, 2)
    seed = 30 + n
    (bt,) = seeded_ids(seed, NB, n)
    cache = device_cache(s, BKG(seed), DEV)
    mirror = host_mirror(s, BKG(seed), range(NB))
    nbytes = oracle.packed_bytes(s, 0, L, n)
    pinned = kvx.PinnedBuffer(nbytes)
    kvsynth.fill_host(pinned.array, seed, kvsynth.image_stream(7))
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    try:
        ring.bind(cache, 0, L, n, ct, pinned if threads == 0 else pinned.array.copy(),
                  fill_threads=threads)
        for rep in range(2):  # twice in a row: slots and events carry over between calls
            kvx.kvx_restore_from_staging(ring, _bt(bt))
            _sync_check()
        st = ring.stats()
        assert st["bytes"] == nbytes and st["pieces"] >= 1
    finally:
        ring.close()
    oracle.restore(s, *mirror, 0, L, bt, ct, pinned.array)
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"
    pinned.free()


def test_aborted_ring_reports_closed():
    s = oracle.Shape(2, 32, 16, 2, 64, 2)
    cache = device_cache(s, BKG(8), DEV)
    img = kvsynth.host_bytes(oracle.packed_bytes(s, 0, 2, 8), 8, 1)
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    try:
        ring.bind(cache, 0, 2, 8, 32, img, fill_threads=1)
        ring.abort()
        with pytest.raises(kvx.KvxError) as ei:
            kvx.kvx_restore_from_staging(ring, _bt(np.arange(8)))
        assert ei.value.status == kvx.KVX_ECLOSED
    finally:
        ring.close()


# ---- large scatters (1024..8192 blocks) ----------------------------------------

@pytest.mark.parametrize("heads", [8, 2], ids=["ordered_16k_slabs", "linear_4k_slabs"])
@pytest.mark.parametrize("n", [1024, 1500, 8192])
def test_ordered_scatter_bit_exact(n, heads):
    """Scatters of 1,024 blocks or more: in destination order with 16 KiB
    slabs, in image order on a linear walk with 4 KiB slabs (48-token chunks,
    three blocks each)."""
    s = oracle.Shape(2, 3 * 8192, 16, heads, 64, 2)
    seed = 40 + n + heads
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, n, n)
    cache = device_cache(s, SRC(seed, kvsynth.MODE_RAW), DEV)
    mirror = host_mirror(s, SRC(seed, kvsynth.MODE_RAW), np.concatenate([bt_src, bt_dst]))
    expect = oracle.gather(s, *mirror, 0, 2, bt_src, 48)
    dst = _packed(expect.size)
    kvx.kvx_gather_blocks(cache, 0, 2, _bt(bt_src), n, 48, dst)
    _sync_check()
    assert np.array_equal(to_host(dst)[:expect.size], expect)
    before = _clone(cache)
    kvx.kvx_scatter_blocks(cache, 0, 2, _bt(bt_dst), n, 48, dst)
    _sync_check()
    oracle.scatter(s, *mirror, 0, 2, bt_dst, 48, expect)
    _compare_paged(cache, s, mirror, range(2), bt_dst, "ordered scatter")
    _untouched_equal(cache, before, s, {0, 1}, bt_dst, "ordered scatter")


# Geometries of the 2 MiB pairings: the gather walks a chunk's slices in pairs
# D apart, and the ordered scatter walks each XCD's range as two fronts paired
# D slices apart, where a slice's run in a chunk (blocks per chunk x slab) times
# D is 2 MiB, D a power of two (gather D <= 32, scatter D <= 16 for slabs above
# 8 KiB, else 4); the scatter also needs the slice count to be a multiple of 16
# (two halves per XCD range) and of 2 D, the gather of 2 D. (Scatters of slabs
# of at most 8 KiB in the default layout walk the image instead.)
PAIRED = [
    # (layers, NB, BS, heads, dim, elem, l0, l1, n, chunk_tokens), then the walks taken:
    # gather pair distance D, scatter (ordered, linear, fronts' D, fronts)
    ((8, 2300, 16, 8, 128, 2, 0, 8, 1100, 256), 4, (1, 0, 4, 2)),    # 32 KiB slabs x 16 blocks
    ((8, 2300, 16, 8, 128, 2, 0, 8, 1100, 1024), 1, (1, 0, 1, 2)),   # x 64 blocks
    ((8, 2300, 16, 8, 128, 2, 0, 8, 1100, 512), 2, (1, 0, 2, 2)),    # x 32 blocks
    ((40, 2100, 16, 2, 128, 2, 0, 40, 1030, 1024), 4, (0, 1, 0, 1)), # 8 KiB x 64: linear scatter
    ((40, 2100, 16, 4, 128, 2, 0, 40, 1030, 1024), 2, (1, 0, 2, 2)), # 16 KiB x 64: 10 slices per XCD
    ((12, 2300, 16, 8, 128, 2, 2, 10, 1100, 256), 4, (1, 0, 4, 2)),  # a partial layer range: 16 slices
    ((12, 2300, 16, 8, 128, 2, 0, 12, 1100, 256), 4, (1, 0, 0, 1)),  # 24 slices: scatter one front
    ((10, 2300, 16, 8, 128, 2, 0, 10, 1100, 256), 0, (1, 0, 0, 1)),  # 20 slices: neither paired
    ((8, 2300, 16, 8, 128, 2, 0, 8, 1100, 128), 8, (1, 0, 8, 2)),    # 32 KiB x 8 blocks
    ((16, 2300, 16, 8, 128, 2, 0, 16, 1101, 64), 16, (1, 0, 16, 2)), # x 4 blocks; ragged last chunk
    ((16, 2300, 16, 4, 128, 2, 0, 16, 1100, 256), 8, (1, 0, 8, 2)),  # 16 KiB x 16 blocks
    ((4, 2300, 16, 8, 128, 2, 0, 4, 1100, 64), 0, (1, 0, 0, 1)),     # D = 16 but 8 slices
    ((32, 2300, 16, 1, 128, 2, 0, 32, 1100, 256), 32, (0, 1, 0, 1)), # 4 KiB x 16 blocks
    ((16, 2300, 16, 2, 128, 2, 0, 16, 1103, 256), 16, (0, 1, 0, 1)), # 8 KiB x 16 blocks; ragged
    ((24, 2300, 16, 1, 128, 2, 0, 24, 1100, 256), 0, (0, 1, 0, 1)),  # D = 32 but 48 slices
]


@pytest.mark.parametrize("case,gather_d,scatter_walk", PAIRED,
                         ids=[f"p{i}" for i in range(len(PAIRED))])
def test_paired_walks_bit_exact(case, gather_d, scatter_walk):
    L, NB, BS, H, D, e, l0, l1, n, ct = case
    s = oracle.Shape(L, NB, BS, H, D, e)
    # the geometry takes the walk it is here for (kvx_copy_walk reports the launcher's choice)
    c = kvx.shape_only_cache(L, NB, BS, H, D, e)
    assert kvx.kvx_copy_walk(c, l0, l1, n, ct, True)["pair_slices"] == gather_d
    w = kvx.kvx_copy_walk(c, l0, l1, n, ct, False)
    assert (w["ordered"], w["linear"], w["pair_slices"], w["fronts"]) == scatter_walk
    seed = 300 + L + ct
    bt_src, bt_dst = seeded_ids(seed, NB, n, n)
    cache = device_cache(s, SRC(seed, kvsynth.MODE_RAW), DEV)
    mirror = host_mirror(s, SRC(seed, kvsynth.MODE_RAW), np.concatenate([bt_src, bt_dst]))
    expect = oracle.gather(s, *mirror, l0, l1, bt_src, ct)
    guard = 4096
    dst = torch.full((expect.size + guard,), 0xA5, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_blocks(cache, l0, l1, _bt(bt_src), n, ct, dst)
    _sync_check()
    got = to_host(dst)
    bad = first_mismatch(got[:expect.size], expect)
    assert bad is None, f"gather differs at byte {bad}"
    assert (got[expect.size:] == 0xA5).all(), "gather wrote past the packed image"
    del got
    before = _clone(cache)
    kvx.kvx_scatter_blocks(cache, l0, l1, _bt(bt_dst), n, ct, dst)
    _sync_check()
    oracle.scatter(s, *mirror, l0, l1, bt_dst, ct, expect)
    _compare_paged(cache, s, mirror, range(l0, l1), bt_dst, "ordered scatter")
    _untouched_equal(cache, before, s, set(range(l0, l1)), bt_dst, "ordered scatter")


@pytest.mark.parametrize("heads", [8, 2], ids=["ordered_16k_slabs", "linear_4k_slabs"])
def test_ordered_scatter_with_bad_ids_skips_only_those(heads):
    s = oracle.Shape(2, 6000, 16, heads, 64, 2)
    n = 2000
    bt, spare = seeded_ids(9, s.num_blocks, n, 3)
    bad_pos = [5, 777, 1999]
    bad = bt.copy()
    bad[bad_pos] = [6000, -3, 2**31 - 1]
    cache = device_cache(s, BKG(9), DEV)
    before = _clone(cache)
    img = kvsynth.host_bytes(oracle.packed_bytes(s, 0, 2, n), 9, 11)
    kvx.kvx_scatter_blocks(cache, 0, 2, _bt(bad), n, 32, torch.from_numpy(img).to(DEV))
    torch.cuda.synchronize()
    with pytest.raises(kvx.KvxError) as ei:
        kvx.kvx_check()
    assert ei.value.status == kvx.KVX_EBADBLOCK
    good = np.delete(bt, bad_pos)
    _untouched_equal(cache, before, s, {0, 1}, good, "bad-id ordered scatter")
    # Oracle: the same scatter with each bad id replaced by a spare block; the
    # valid destinations must match it (the spares' units were skipped on the GPU).
    mirror = host_mirror(s, BKG(9), range(s.num_blocks))
    subst = bt.copy()
    subst[bad_pos] = spare
    oracle.scatter(s, *mirror, 0, 2, subst, 32, img)
    _compare_paged(cache, s, mirror, range(2), good, "bad-id ordered scatter")


# ---- calls larger than one dispatch ---------------------------------------------

def test_launch_split_above_2_22_units():
    """A call of more than 2^22 units is split into several launches (a grid
    counts its work-items in 32 bits). 16-byte slabs (1 token x 1 head x 8 dims,
    bf16) over 64 layers and 40,000 blocks make 5,120,000 units per call: the
    gather, the destination-ordered scatter and the chunk-list gather, each
    bit-exact against the oracle."""
    s = oracle.Shape(64, 80004, 1, 1, 8, 2)
    n, ct, L = 40000, 16, 64
    assert n * L * 2 > 1 << 22
    seed = 123
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, n, n)
    fill = SRC(seed, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    expect = oracle.gather(s, *mirror, 0, L, bt_src, ct)
    dst = _packed(expect.size)
    kvx.kvx_gather_blocks(cache, 0, L, _bt(bt_src), n, ct, dst)
    _sync_check()
    bad = first_mismatch(to_host(dst)[:expect.size], expect)
    assert bad is None, f"split gather differs at byte {bad}"
    kvx.kvx_scatter_blocks(cache, 0, L, _bt(bt_dst), n, ct, dst)
    _sync_check()
    oracle.scatter(s, *mirror, 0, L, bt_dst, ct, expect)
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"
    # the same image through the chunk-list kernel: 2,500 chunks of 16 blocks
    per_block = oracle.packed_bytes(s, 0, L, 1)
    refs = [(b * per_block, b, min(16, n - b)) for b in range(0, n, 16)]
    packed = torch.full((expect.size + 4096,), 0x5A, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_chunks(cache, 0, L, _bt(bt_src), n, kvx.chunk_refs(refs, DEV), len(refs), ct,
                          packed)
    _sync_check()
    got = to_host(packed)
    bad = first_mismatch(got[:expect.size], expect)
    assert bad is None, f"split chunk-list gather differs at byte {bad}"
    assert (got[expect.size:] == 0x5A).all()


def test_probe_stream_copies_exactly():
    """The roofline probe's copy mode is a plain copy; the write mode writes
    every 16-byte vector; the read mode leaves its source alone."""
    n = 64 << 20
    src = torch.randint(0, 256, (n,), dtype=torch.uint8, device=DEV)
    keep = src.clone()
    dst = torch.zeros(n, dtype=torch.uint8, device=DEV)
    kvx.kvx_probe_stream(src, dst, n, 2)
    _sync_check()
    assert torch.equal(dst, src)
    kvx.kvx_probe_stream(src, None, n, 0)
    dst.zero_()
    kvx.kvx_probe_stream(None, dst, n, 1)
    _sync_check()
    assert torch.equal(src, keep)
    words = dst.view(torch.int32).view(-1, 4)
    assert bool((words[:, 2] == 0x9E3779B9 - 2**32).all()) and bool((words[:, 3] == 0x7F4A7C15).all())
