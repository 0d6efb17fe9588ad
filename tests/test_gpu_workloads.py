"""GPU parity at the full workload sizes, in the launch configuration the bench
times: the 8B-shaped 80k-token prefix (5,000 blocks of a 20,000-block pool,
10.49 GB moved per operation) and the 32k-token granularity sweep (chunks of
16/64/256/1024 tokens, rings of 2/4/8 slots of 64 MiB).

Every gathered image is compared with the oracle's image byte for byte.
Scatters and restores are compared with the oracle's result on every slab
they name (read back from the device), and every other block is checked
unchanged on the device against a copy taken before the call.
"""
import numpy as np
import pytest

import kvsynth
import oracle
from kvtest_util import (Filled, device_cache, first_mismatch, host_mirror, mirror_slabs,
                         read_slabs, seeded_ids, shape_8b, to_host)

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
NB = 20000
SLOT = 64 << 20
# Pieces of the ramped 80k restore plan (also checked on the CPU, test_abi).
RAMPED_80K_PIECES = 161


def _bt(ids):
    return torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(DEV)


def _check():
    torch.cuda.synchronize()
    kvx.kvx_check()


def _compare_named_slabs(cache, shape, mirror, ids, what):
    for l in range(shape.num_layers):
        for kv in (0, 1):
            got = read_slabs(cache, l, kv, ids)
            exp = mirror_slabs(mirror, shape, l, kv, ids)
            if not np.array_equal(got, exp):
                bad = first_mismatch(got.ravel(), exp.ravel())
                raise AssertionError(f"{what}: layer {l} kv {kv} differs at byte {bad} "
                                     f"(block {ids[bad // shape.slab_bytes]})")


def _unchanged_except(cache, before, shape, ids, what):
    keep = torch.from_numpy(np.setdiff1d(np.arange(shape.num_blocks), ids)).to(DEV)
    for l in range(shape.num_layers):
        for kv in (0, 1):
            a = (cache.k if kv == 0 else cache.v)[l].view(torch.uint8)
            b = before[kv][l].view(torch.uint8)
            assert torch.equal(a.index_select(0, keep), b.index_select(0, keep)), \
                f"{what}: a block outside the named set changed (layer {l} kv {kv})"


class Workload80k:
    """8B-shaped cache, 80,000-token prefix; shared by the tests below."""

    def __init__(self):
        self.shape = shape_8b(NB)
        self.seed = 3
        self.fill = Filled(self.seed, kvsynth.ROLE_SRC, kvsynth.MODE_NORMAL_BF16)
        self.bt_src, self.bt_dst, self.bt_rst = seeded_ids(self.seed, NB, 5000, 5000, 5000)
        self.cache = device_cache(self.shape, self.fill, DEV)
        self.mirror = host_mirror(self.shape, self.fill, self.bt_src)
        self.nbytes = oracle.packed_bytes(self.shape, 0, 32, 5000)


@pytest.fixture(scope="module")
def w80k():
    w = Workload80k()
    yield w
    del w.cache
    torch.cuda.empty_cache()


def test_80k_gather_full_image_bit_exact(w80k):
    w = w80k
    assert w.nbytes == 10_485_760_000
    expect = oracle.gather(w.shape, *w.mirror, 0, 32, w.bt_src, 256)
    dst = torch.empty(w.nbytes, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_blocks(w.cache, 0, 32, _bt(w.bt_src), 5000, 256, dst)
    _check()
    got = to_host(dst)
    bad = first_mismatch(got, expect)
    assert bad is None, f"80k gather differs at byte {bad}"
    w.packed = dst
    w.expect = expect


def test_80k_scatter_to_fresh_blocks(w80k):
    w = w80k
    if not hasattr(w, "packed"):
        pytest.skip("needs the gather of the previous test")
    before = ([t.clone() for t in w.cache.k], [t.clone() for t in w.cache.v])
    kvx.kvx_scatter_blocks(w.cache, 0, 32, _bt(w.bt_dst), 5000, 256, w.packed)
    _check()
    oracle.scatter(w.shape, *w.mirror, 0, 32, w.bt_dst, 256, w.expect)
    _compare_named_slabs(w.cache, w.shape, w.mirror, w.bt_dst, "80k scatter")
    _unchanged_except(w.cache, before, w.shape, w.bt_dst, "80k scatter")
    del before
    torch.cuda.empty_cache()


def test_80k_staged_restore_4x64MiB(w80k):
    w = w80k
    if not hasattr(w, "packed"):
        pytest.skip("needs the gather of the first test")
    del w.packed
    torch.cuda.empty_cache()
    image = kvx.PinnedBuffer(w.nbytes)
    kvsynth.fill_host(image.array, w.seed, kvsynth.image_stream(1), threads=16)
    before = ([t.clone() for t in w.cache.k], [t.clone() for t in w.cache.v])
    ring = kvx.StagingRing(DEV, 4, SLOT)
    try:
        ring.bind(w.cache, 0, 32, 5000, 256, image, fill_threads=8)
        kvx.kvx_restore_from_staging(ring, _bt(w.bt_rst))
        _check()
        # the restore's ramp (each piece at most twice the one before, from
        # 1/8 slot): 8, 16, 8 MiB of the first chunk, 16 + 16 of the second,
        # the third whole, then 155 two-chunk pieces (the last 32 + 16 MiB)
        assert ring.stats()["pieces"] == RAMPED_80K_PIECES
    finally:
        ring.close()
    # the oracle's restore: every restored slab, and every other block unchanged
    oracle.restore(w.shape, *w.mirror, 0, 32, w.bt_rst, 256, image.array)
    _compare_named_slabs(w.cache, w.shape, w.mirror, w.bt_rst, "80k restore")
    _unchanged_except(w.cache, before, w.shape, w.bt_rst, "80k restore")
    del before
    torch.cuda.empty_cache()
    image.free()
    del w.expect


# ---- 32k-token granularity sweep -------------------------------------------------

class Workload32k:
    def __init__(self):
        self.shape = shape_8b(NB)
        self.seed = 4
        self.fill = Filled(self.seed, kvsynth.ROLE_SRC, kvsynth.MODE_NORMAL_BF16)
        self.bt_src, self.bt_dst = seeded_ids(self.seed, NB, 2048, 2048)
        self.cache = device_cache(self.shape, self.fill, DEV)
        self.mirror = host_mirror(self.shape, self.fill, self.bt_src)
        self.nbytes = oracle.packed_bytes(self.shape, 0, 32, 2048)
        self.packed = torch.empty(self.nbytes, dtype=torch.uint8, device=DEV)
        # the cache as filled; the scatters and restores below write only the
        # bt_dst blocks, so every other block must keep this content
        self.before = ([t.clone() for t in self.cache.k], [t.clone() for t in self.cache.v])


@pytest.fixture(scope="module")
def w32k():
    w = Workload32k()
    yield w
    del w.cache, w.packed, w.before
    torch.cuda.empty_cache()


@pytest.mark.parametrize("chunk", [16, 64, 256, 1024])
def test_32k_gather_then_scatter_per_chunk_size(w32k, chunk):
    w = w32k
    expect = oracle.gather(w.shape, *w.mirror, 0, 32, w.bt_src, chunk)
    kvx.kvx_gather_blocks(w.cache, 0, 32, _bt(w.bt_src), 2048, chunk, w.packed)
    _check()
    bad = first_mismatch(to_host(w.packed), expect)
    assert bad is None, f"chunk {chunk}: gather differs at byte {bad}"
    # scatter into fresh blocks and compare every named slab with the oracle
    kvx.kvx_scatter_blocks(w.cache, 0, 32, _bt(w.bt_dst), 2048, chunk, w.packed)
    _check()
    # (the mirror's source blocks are disjoint from bt_dst, so later chunk
    # sizes still gather from unchanged sources)
    oracle.scatter(w.shape, *w.mirror, 0, 32, w.bt_dst, chunk, expect)
    _compare_named_slabs(w.cache, w.shape, w.mirror, w.bt_dst, f"chunk {chunk} scatter")
    _unchanged_except(w.cache, w.before, w.shape, w.bt_dst, f"chunk {chunk} scatter")


@pytest.mark.parametrize("chunk", [16, 64, 256, 1024])
@pytest.mark.parametrize("slots", [2, 4, 8])
def test_32k_staged_restore(w32k, chunk, slots):
    w = w32k
    image = kvx.PinnedBuffer(w.nbytes)
    kvsynth.fill_host(image.array, w.seed, kvsynth.image_stream(100 + chunk), threads=16)
    ring = kvx.StagingRing(DEV, slots, SLOT)
    try:
        ring.bind(w.cache, 0, 32, 2048, chunk, image, fill_threads=8)
        kvx.kvx_restore_from_staging(ring, _bt(w.bt_dst))
        _check()
    finally:
        ring.close()
    # every restored slab against the oracle's restore, every other block unchanged
    exp = oracle.new_mirror(w.shape)
    oracle.restore(w.shape, *exp, 0, 32, w.bt_dst, chunk, image.array)
    _compare_named_slabs(w.cache, w.shape, exp, w.bt_dst, f"chunk {chunk} slots {slots} restore")
    _unchanged_except(w.cache, w.before, w.shape, w.bt_dst, f"chunk {chunk} slots {slots} restore")
    image.free()
