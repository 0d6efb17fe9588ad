"""Staging-ring protocol under host-forced stress: small rings reused many
times, random pauses in the fill / drain threads (varied interleavings), and
released host slots overwritten with poison before they are refilled, so a
copy that still read a released slot would deliver the poison into the cache.
Results must stay bit-exact against the oracle. Aborts are forced from another
thread while a transfer runs; the call must return KVX_ECLOSED and the ring
must close without hanging. Every condition is forced from the host; every
kernel exits normally."""
import threading
import time

import numpy as np
import pytest

import kvsynth
import oracle
from kvtest_util import Filled, device_cache, host_mirror, seeded_ids, to_host

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _bt(ids):
    return torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(DEV)


STRESS = [
    # (slots, slot_bytes, threads, max_delay_us, chunk_tokens)
    (2, 64 << 10, 3, 300, 32),
    (2, 32 << 10, 1, 200, 64),     # chunks larger than a slot: layer pieces
    (3, 128 << 10, 4, 500, 16),
    (1, 64 << 10, 2, 300, 32),     # one slot: each piece's scatter must drain it first
]


@pytest.mark.parametrize("hip_copies", [False, True], ids=["dma", "hip"])
@pytest.mark.parametrize("case", STRESS, ids=[f"s{i}" for i in range(len(STRESS))])
def test_restore_with_pauses_and_poisoned_slots(case, hip_copies):
    slots, slot_bytes, threads, delay, ct = case
    s = oracle.Shape(4, 400, 16, 2, 64, 2)
    n = 150
    seed = 90 + slots + threads
    (bt,) = seeded_ids(seed, s.num_blocks, n)
    cache = device_cache(s, Filled(seed, kvsynth.ROLE_DST), DEV)
    mirror = host_mirror(s, Filled(seed, kvsynth.ROLE_DST), range(s.num_blocks))
    image = kvsynth.host_bytes(oracle.packed_bytes(s, 0, 4, n), seed, kvsynth.image_stream(3),
                               mode=kvsynth.MODE_RAW)
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    try:
        ring.set_test_hooks(max_delay_us=delay, poison=True, hip_copies=hip_copies)
        ring.bind(cache, 0, 4, n, ct, image, fill_threads=threads)
        for _ in range(2):
            kvx.kvx_restore_from_staging(ring, _bt(bt))
        torch.cuda.synchronize()
        kvx.kvx_check()
        assert ring.stats()["pieces"] > 3 * slots  # every slot reused several times
        assert ring.stats()["dma"] == (0 if hip_copies else 1)
    finally:
        ring.close()
    oracle.restore(s, *mirror, 0, 4, bt, ct, image)
    for l in range(4):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"


@pytest.mark.parametrize("hip_copies", [False, True], ids=["dma", "hip"])
@pytest.mark.parametrize("case", STRESS, ids=[f"s{i}" for i in range(len(STRESS))])
def test_offload_with_pauses(case, hip_copies):
    slots, slot_bytes, threads, delay, ct = case
    s = oracle.Shape(4, 400, 16, 2, 64, 2)
    n = 150
    seed = 95 + slots + threads
    (bt,) = seeded_ids(seed, s.num_blocks, n)
    fill = Filled(seed, kvsynth.ROLE_NEW, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, bt)
    bpc = ct // 16
    per_block = oracle.packed_bytes(s, 0, 4, 1)
    chunks = [(np.zeros(min(bpc, n - b) * per_block, np.uint8), b, min(bpc, n - b))
              for b in range(0, n, bpc)]
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    try:
        ring.set_test_hooks(max_delay_us=delay, hip_copies=hip_copies)
        ring.bind_offload(cache, 0, 4, ct, chunks, drain_threads=threads)
        kvx.kvx_offload_to_staging(ring, _bt(bt))
        kvx.kvx_check()
        assert ring.stats()["dma"] == (0 if hip_copies else 1)
    finally:
        ring.close()
    image = np.concatenate([c[0] for c in chunks])
    assert np.array_equal(image, oracle.gather(s, *mirror, 0, 4, bt, ct))


def _abort_after(ring, seconds):
    def run():
        time.sleep(seconds)
        ring.abort()
    t = threading.Thread(target=run)
    t.start()
    return t


def test_abort_during_restore_returns_closed_and_ring_closes():
    s = oracle.Shape(2, 3000, 16, 2, 64, 2)
    n = 1200
    (bt,) = seeded_ids(11, s.num_blocks, n)
    cache = device_cache(s, Filled(11, kvsynth.ROLE_DST), DEV)
    image = kvsynth.host_bytes(oracle.packed_bytes(s, 0, 2, n), 11, 5)
    ring = kvx.StagingRing(DEV, 2, 64 << 10)  # 300 pieces of 64 KiB
    try:
        ring.set_test_hooks(max_delay_us=20000)
        ring.bind(cache, 0, 2, n, 64, image, fill_threads=2)
        t = _abort_after(ring, 0.05)
        t0 = time.perf_counter()
        with pytest.raises(kvx.KvxError) as ei:
            kvx.kvx_restore_from_staging(ring, _bt(bt))
        t.join()
        assert ei.value.status == kvx.KVX_ECLOSED
        assert time.perf_counter() - t0 < 5.0
        torch.cuda.synchronize()  # pieces already enqueued complete normally
        kvx.kvx_check()
        with pytest.raises(kvx.KvxError) as ei:  # the ring stays closed
            kvx.kvx_restore_from_staging(ring, _bt(bt))
        assert ei.value.status == kvx.KVX_ECLOSED
    finally:
        ring.close()


def test_abort_during_offload_returns_closed_and_ring_closes():
    s = oracle.Shape(2, 3000, 16, 2, 64, 2)
    n = 1200
    (bt,) = seeded_ids(12, s.num_blocks, n)
    cache = device_cache(s, Filled(12, kvsynth.ROLE_NEW), DEV)
    per_block = oracle.packed_bytes(s, 0, 2, 1)
    chunks = [(np.zeros(4 * per_block, np.uint8), b, 4) for b in range(0, n, 4)]
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    try:
        ring.set_test_hooks(max_delay_us=20000)
        ring.bind_offload(cache, 0, 2, 64, chunks, drain_threads=2)
        t = _abort_after(ring, 0.05)
        t0 = time.perf_counter()
        with pytest.raises(kvx.KvxError) as ei:
            kvx.kvx_offload_to_staging(ring, _bt(bt))
        t.join()
        assert ei.value.status == kvx.KVX_ECLOSED
        assert time.perf_counter() - t0 < 5.0
        torch.cuda.synchronize()
        kvx.kvx_check()
    finally:
        ring.close()
