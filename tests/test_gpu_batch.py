"""GPU parity of the batched path: fused chunk-list gather / scatter, chunk-list
staged restore, staged offload, and one batched step (restore of the distinct
missing chunks of a request batch concurrent with the offload of their new
blocks, both started from one thread with kvx_restore_begin and
kvx_offload_begin), against the oracle.

The oracle's side of a chunk list is the plain definition: chunk c is the
oracle gather of its own blocks, as one chunk, placed at its packed offset.
"""
import time

import numpy as np
import pytest

import kvsynth
import kvsynth.prefix_tree as pt
import oracle
import oracle.prefix as oracle_prefix
from kvtest_util import (Filled, check_layer_after_scatters, device_cache, first_mismatch,
                         host_mirror, mirror_slabs, read_slabs, seeded_ids, shape_70b, to_host)

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402
from paper_2609_11744_amd import step  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _bt(ids):
    return torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(DEV)


def _check():
    torch.cuda.synchronize()
    kvx.kvx_check()


def _oracle_chunk(s, mirror, l0, l1, bt, off, nb, ct):
    return oracle.gather(s, *mirror, l0, l1, bt[off:off + nb], ct)


def _compare_blocks(cache, s, mirror, ids, layers, what):
    for l in layers:
        for kv in (0, 1):
            got = read_slabs(cache, l, kv, ids)
            exp = mirror_slabs(mirror, s, l, kv, ids)
            bad = first_mismatch(got.ravel(), exp.ravel())
            assert bad is None, f"{what}: layer {l} kv {kv} differs at byte {bad}"


# ---- fused chunk-list gather / scatter ------------------------------------------

@pytest.mark.parametrize("l0,l1", [(0, 3), (1, 2)])
def test_chunk_list_gather_and_scatter_bit_exact(l0, l1):
    s = oracle.Shape(3, 200, 16, 2, 64, 2)
    ct = 64  # 4 blocks per chunk
    seed = 60 + l0
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, 40, 40)
    # chunks of 1..4 blocks over the table, placed out of order with gaps
    rng = np.random.default_rng(seed)
    sizes, at = [], 0
    while at < 40:
        nb = int(min(rng.integers(1, 5), 40 - at))
        sizes.append((at, nb))
        at += nb
    per_block = oracle.packed_bytes(s, l0, l1, 1)
    order = rng.permutation(len(sizes))
    refs, off = [None] * len(sizes), 4096
    for i in order:
        bt0, nb = sizes[i]
        refs[i] = (off, bt0, nb)
        off += nb * per_block + 16 * int(rng.integers(0, 4))
    total = off + 4096
    cache = device_cache(s, Filled(seed, kvsynth.ROLE_SRC, kvsynth.MODE_RAW), DEV)
    mirror = host_mirror(s, Filled(seed, kvsynth.ROLE_SRC, kvsynth.MODE_RAW), range(s.num_blocks))
    packed = torch.full((total,), 0x5A, dtype=torch.uint8, device=DEV)
    dref = kvx.chunk_refs(refs, DEV)
    kvx.kvx_gather_chunks(cache, l0, l1, _bt(bt_src), 40, dref, len(refs), ct, packed)
    _check()
    got = to_host(packed)
    expect = np.full(total, 0x5A, np.uint8)
    for (off, bt0, nb) in refs:
        img = _oracle_chunk(s, mirror, l0, l1, bt_src, bt0, nb, ct)
        expect[off:off + img.size] = img
    bad = first_mismatch(got, expect)
    assert bad is None, f"chunk-list gather differs at byte {bad}"

    kvx.kvx_scatter_chunks(cache, l0, l1, _bt(bt_dst), 40, dref, len(refs), ct, packed)
    _check()
    for (off, bt0, nb) in refs:
        oracle.scatter(s, *mirror, l0, l1, bt_dst[bt0:bt0 + nb], ct, expect[off:])
    for l in range(3):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"


def test_chunk_list_rejects_bad_refs_on_device():
    s = oracle.Shape(2, 64, 16, 2, 64, 2)
    cache = device_cache(s, Filled(3, kvsynth.ROLE_DST, kvsynth.MODE_RAW), DEV)
    before = [t.clone() for t in cache.k + cache.v]
    per_block = oracle.packed_bytes(s, 0, 2, 1)
    packed = torch.zeros(8 * per_block, dtype=torch.uint8, device=DEV)
    bad_refs = [(0, 0, 5),            # more blocks than a chunk holds (ct = 64 -> 4)
                (8, 0, 1),            # misaligned packed offset
                (0, 6, 4),            # block-table slice past table_len (8)
                (7 * per_block, 0, 2)]  # image past the packed buffer
    for ref in bad_refs:
        kvx.kvx_scatter_chunks(cache, 0, 2, _bt(np.arange(8)), 8, kvx.chunk_refs([ref], DEV), 1,
                               64, packed)
        torch.cuda.synchronize()
        with pytest.raises(kvx.KvxError) as ei:
            kvx.kvx_check()
        assert ei.value.status == kvx.KVX_EINVAL, ref
    for a, b in zip(cache.k + cache.v, before):
        assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))


# ---- chunk-list staged restore and staged offload ------------------------------

RING = [
    # (layers, chunk_tokens, slots, slot_bytes, threads)
    (4, 64, 2, 96 << 10, 2),    # several chunks per slot, 2 slots reused many times
    (4, 64, 3, 40 << 10, 1),    # 64 KiB chunks larger than a slot: layer pieces
    (4, 64, 4, 128 << 10, 0),   # no staging copy (pinned host images)
]


def _host_chunk_images(s, l0, l1, sizes, seed, pinned):
    """One host buffer per chunk (separate allocations, out of order)."""
    per_block = oracle.packed_bytes(s, l0, l1, 1)
    bufs = []
    for i, (bt0, nb) in enumerate(sizes):
        if pinned:
            b = kvx.PinnedBuffer(nb * per_block)
            kvsynth.fill_host(b.array, seed, 0x77000 + i)
            bufs.append(b)
        else:
            bufs.append(kvsynth.host_bytes(nb * per_block, seed, 0x77000 + i))
    return bufs


def _arr(b):
    return b.array if isinstance(b, kvx.PinnedBuffer) else b


@pytest.mark.parametrize("hip_copies", [False, True], ids=["dma", "hip"])
@pytest.mark.parametrize("case", RING, ids=[f"ring{i}" for i in range(len(RING))])
def test_chunk_list_restore_equals_oracle(case, hip_copies):
    """Both host-to-device paths: the DMA engine driven directly (default) and
    the HIP runtime copy on the side stream."""
    L, ct, slots, slot_bytes, threads = case
    s = oracle.Shape(L, 300, 16, 2, 64, 2)
    seed = 70 + slots
    (bt,) = seeded_ids(seed, s.num_blocks, 45)
    rng = np.random.default_rng(seed)
    sizes, at = [], 0
    while at < 45:
        nb = int(min(rng.integers(1, 5), 45 - at))
        sizes.append((at, nb))
        at += nb
    bufs = _host_chunk_images(s, 0, L, sizes, seed, pinned=threads == 0)
    cache = device_cache(s, Filled(seed, kvsynth.ROLE_DST), DEV)
    mirror = host_mirror(s, Filled(seed, kvsynth.ROLE_DST), range(s.num_blocks))
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    try:
        ring.set_test_hooks(hip_copies=hip_copies)
        ring.bind_chunks(cache, 0, L, ct, [(b, bt0, nb) for b, (bt0, nb) in zip(bufs, sizes)],
                         fill_threads=threads)
        for _ in range(2):
            kvx.kvx_restore_from_staging(ring, _bt(bt))
            _check()
        assert ring.stats()["dma"] == (0 if hip_copies else 1)
    finally:
        ring.close()
    for b, (bt0, nb) in zip(bufs, sizes):
        oracle.scatter(s, *mirror, 0, L, bt[bt0:bt0 + nb], ct, _arr(b))
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"


@pytest.mark.parametrize("hip_copies", [False, True], ids=["dma", "hip"])
@pytest.mark.parametrize("case", RING, ids=[f"ring{i}" for i in range(len(RING))])
def test_offload_equals_oracle_gather(case, hip_copies):
    """Both device-to-host paths: the DMA engine driven directly (default) and
    the HIP runtime copy on the side stream."""
    L, ct, slots, slot_bytes, threads = case
    s = oracle.Shape(L, 300, 16, 2, 64, 2)
    seed = 80 + slots
    (bt,) = seeded_ids(seed, s.num_blocks, 45)
    rng = np.random.default_rng(seed)
    sizes, at = [], 0
    while at < 45:
        nb = int(min(rng.integers(1, 5), 45 - at))
        sizes.append((at, nb))
        at += nb
    fill = Filled(seed, kvsynth.ROLE_NEW, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, bt)
    per_block = oracle.packed_bytes(s, 0, L, 1)
    if threads == 0:
        sinks = [kvx.PinnedBuffer(nb * per_block) for _, nb in sizes]
        for b in sinks:
            b.array[:] = 0xEE
    else:
        sinks = [np.full(nb * per_block, 0xEE, np.uint8) for _, nb in sizes]
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    try:
        ring.set_test_hooks(hip_copies=hip_copies)
        ring.bind_offload(cache, 0, L, ct, [(b, bt0, nb) for b, (bt0, nb) in zip(sinks, sizes)],
                          drain_threads=threads)
        for _ in range(2):
            kvx.kvx_offload_to_staging(ring, _bt(bt))
        _check()
        assert ring.stats()["dma"] == (0 if hip_copies else 1)
    finally:
        ring.close()
    for b, (bt0, nb) in zip(sinks, sizes):
        exp = oracle.gather(s, *mirror, 0, L, bt[bt0:bt0 + nb], ct)
        assert np.array_equal(_arr(b), exp), f"offloaded chunk at table entry {bt0} differs"


# ---- one batched step: restore distinct missing chunks || offload new blocks ----

def _run_step(s, reqs, plan, seed, slots=4, slot_bytes=64 << 20, threads=8, layers=None):
    """Execute a step plan: returns (cache, restore table, restore images,
    offload table, sinks, timings)."""
    L = s.num_layers
    per_block = oracle.packed_bytes(s, 0, L, 1)
    nb_needed = plan.restore_blocks + plan.offload_blocks
    ids = np.random.default_rng(seed).permutation(s.num_blocks).astype(np.int32)
    assert nb_needed <= s.num_blocks
    rbt, obt = ids[:plan.restore_blocks], ids[plan.restore_blocks:nb_needed]
    # the host store: one image per distinct missing chunk, drawn from its chunk stream
    store = np.empty(plan.restore_blocks * per_block, dtype=np.uint8)
    store_chunks = []
    for c in plan.restore:
        view = store[c.bt_offset * per_block:(c.bt_offset + c.n_blocks) * per_block]
        owner = reqs[c.origin[0]].chunk_owner[c.origin[1]]
        kvsynth.fill_host(view, seed, pt.chunk_stream(owner), threads=16)
        store_chunks.append((view, c.bt_offset, c.n_blocks))
    cache = device_cache(s, Filled(seed, kvsynth.ROLE_NEW), DEV)
    sinks = [np.zeros(c.n_blocks * per_block, dtype=np.uint8) for c in plan.offload]
    r_ring = kvx.StagingRing(DEV, slots, slot_bytes)
    o_ring = kvx.StagingRing(DEV, slots, slot_bytes)
    timings = {}
    try:
        r_ring.bind_chunks(cache, 0, L, 256, store_chunks, fill_threads=threads)
        o_ring.bind_offload(cache, 0, L, 256,
                            [(b, c.bt_offset, c.n_blocks) for b, c in zip(sinks, plan.offload)],
                            drain_threads=threads)
        rbt_d, obt_d = _bt(rbt), _bt(obt)
        s_r, s_o = torch.cuda.Stream(), torch.cuda.Stream()
        torch.cuda.synchronize()
        # both transfers run on the rings' own threads; this thread only
        # starts and collects them
        t0 = time.perf_counter()
        kvx.kvx_restore_begin(r_ring, rbt_d, stream=s_r)
        kvx.kvx_offload_begin(o_ring, obt_d, stream=s_o)
        kvx.kvx_offload_wait(o_ring)
        timings["offload_s"] = time.perf_counter() - t0
        kvx.kvx_restore_wait(r_ring, stream=s_r)
        s_r.synchronize()
        timings["restore_s"] = time.perf_counter() - t0
        _check()
        kvx.kvx_check(s_r)
        kvx.kvx_check(s_o)
    finally:
        r_ring.close()
        o_ring.close()
    return cache, rbt, store, store_chunks, obt, sinks, timings


@pytest.mark.parametrize("share", ["chunk", "block"])
def test_batched_step_small_shape_bit_exact(share):
    """The whole step at a small shape (4 layers, 4 KiB slabs), every byte
    checked; with share="block" shared prefixes end inside chunks, so a child
    that extends its parent's partial chunk restores a chunk of its own."""
    seed = 5
    reqs = pt.make_requests(seed, n=24, lo=256, hi=2048, share=share)
    plan = step.plan_step(reqs, 16, 256)
    if share == "block":
        assert any(r.shared_tokens % 256 for r in reqs)
        # the plan restores one chunk per distinct exact key (the oracle's plan)
        want = oracle_prefix.plan_step(reqs, 16, 256)
        assert [(c.n_blocks, c.origin, c.bt_offset) for c in plan.restore] == \
            [(nb, o, bt) for _, nb, o, bt in want["restore"]]
    s = oracle.Shape(4, plan.restore_blocks + plan.offload_blocks + 32, 16, 2, 64, 2)
    cache, rbt, store, store_chunks, obt, sinks, _ = _run_step(
        s, reqs, plan, seed, slots=2, slot_bytes=192 << 10, threads=3)  # 1 layer of a full chunk = 128 KiB
    fill = Filled(seed, kvsynth.ROLE_NEW, kvsynth.MODE_NORMAL_BF16)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    for (img, bt0, nb), c in zip(store_chunks, plan.restore):
        oracle.scatter(s, *mirror, 0, 4, rbt[bt0:bt0 + nb], 256, img)
    for l in range(4):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"
    src = host_mirror(s, fill, obt)
    for b, c in zip(sinks, plan.offload):
        assert np.array_equal(b, oracle.gather(s, *src, 0, 4, obt[c.bt_offset:c.bt_offset + c.n_blocks], 256))


@pytest.mark.timeout(900)
def test_batched_step_70b_64_requests():
    """The full batched workload: 64 requests on a prefix tree over a 70B-shaped
    cache (80 layers, 8 KV heads, head dim 128), distinct missing chunks restored
    through a 4 x 64 MiB ring while the new blocks are offloaded through another."""
    seed = 5
    reqs = pt.make_requests(seed, n=64)
    plan = step.plan_step(reqs, 16, 256)
    s = shape_70b(plan.restore_blocks + plan.offload_blocks + 64)
    print(f"\n70B batch: {len(plan.restore)} distinct missing chunks "
          f"({plan.restore_blocks} blocks), {plan.resident_hits} resident, "
          f"{plan.offload_blocks} new blocks; pool {s.num_blocks} blocks", flush=True)
    cache, rbt, store, store_chunks, obt, sinks, t = _run_step(s, reqs, plan, seed)
    per_block = oracle.packed_bytes(s, 0, 80, 1)
    rb, ob = plan.restore_blocks * per_block, plan.offload_blocks * per_block
    print(f"restore {rb / 1e9:.1f} GB in {t['restore_s']:.3f} s; offload {ob / 1e9:.1f} GB "
          f"in {t['offload_s']:.3f} s (concurrent)", flush=True)
    # every byte of every cache tensor against the oracle: the generator's
    # content with each restored chunk scattered into it (restored slabs
    # right, every other block unchanged), one layer at a time
    fill = Filled(seed, kvsynth.ROLE_NEW, kvsynth.MODE_NORMAL_BF16)
    chunks = [(img, rbt[bt0:bt0 + nb], 0) for img, bt0, nb in store_chunks]
    for l in range(80):
        check_layer_after_scatters(cache, s, fill, l, chunks, 256, "70B restore")
        if l % 16 == 15:
            print(f"70B restore: layers 0..{l} match the oracle", flush=True)
    # offload: every sink against the oracle gather of the new blocks
    src = host_mirror(s, fill, obt)
    for b, c in zip(sinks, plan.offload):
        exp = oracle.gather(s, *src, 0, 80, obt[c.bt_offset:c.bt_offset + c.n_blocks], 256)
        assert np.array_equal(b, exp), f"offload of request {c.request} chunk {c.chunk} differs"
