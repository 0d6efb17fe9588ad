"""GPU parity of restores from preloaded chunk images (Sec. 6.5): chunk files
written by the ring's offload are read ahead into a pinned preloader pool;
the request's fetch claims the staged images and reads the others on demand;
the ring restores straight from the pool (fill_threads 0: host-to-device
copies out of the pinned slots), bit-exact against the oracle's scatter of
the file contents."""
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


CASES = [
    # (shape args, n blocks, chunk_tokens, files preloaded before the fetch, hip_copies)
    ((4, 400, 16, 2, 64, 2), 150, 64, 19, False),   # half staged, half on demand; ragged last chunk
    ((4, 400, 16, 2, 64, 2), 150, 64, 38, False),   # all staged: only the copy to the device left
    ((4, 400, 16, 2, 64, 2), 150, 64, 0, True),     # all on demand; copies through the runtime
    ((3, 300, 5, 2, 16, 2), 70, 15, 7, False),      # 320-byte slabs, 24 files of 2 KiB
]


@pytest.mark.parametrize("case", CASES, ids=[f"c{i}" for i in range(len(CASES))])
def test_restore_from_preloaded_images(tmp_path, case):
    shape_args, n, ct, n_pre, hip_copies = case
    s = oracle.Shape(*shape_args)
    L, BS = s.num_layers, s.block_size
    bpc = ct // BS
    seed = 500 + n + n_pre
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, n, n)
    fill = Filled(seed, kvsynth.ROLE_NEW, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    chunks = [(kvx.kvx_chunk_path(str(tmp_path), "p", 0x9E3779B97F4A7C15 * (i + 1)), b,
               min(bpc, n - b)) for i, b in enumerate(range(0, n, bpc))]
    paths = [c[0] for c in chunks]
    per_block = oracle.packed_bytes(s, 0, L, 1)
    slot = -(-bpc * per_block // 4096) * 4096
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    pre = kvx.Preloader(len(chunks) + 2, slot, io_depth=4, reserve=2, pinned=True)
    try:
        ring.set_test_hooks(hip_copies=hip_copies)
        ring.bind_offload_files(cache, 0, L, ct, chunks, io_depth=4)
        kvx.kvx_offload_to_staging(ring, _bt(bt_src))
        kvx.kvx_check()
        pre.hint(paths[:n_pre])
        pre.wait_idle()
        imgs = pre.fetch(paths)
        st = pre.stats()
        assert st["hits_ready"] == n_pre and st["demand_reads"] == len(paths) - n_pre
        for img, (path, _, _) in zip(imgs, chunks):
            assert np.array_equal(img, np.fromfile(path, np.uint8)), f"staged image of {path}"
        ring.bind_chunks(cache, 0, L, ct, [(img, b0, nb) for img, (_, b0, nb) in zip(imgs, chunks)],
                         fill_threads=0)
        for _ in range(2):
            kvx.kvx_restore_from_staging(ring, _bt(bt_dst))
        torch.cuda.synchronize()
        kvx.kvx_check()
        assert ring.stats()["dma"] == (0 if hip_copies else 1)
        pre.release(paths)
    finally:
        ring.close()
        pre.close()
    for path, b0, nb in chunks:
        oracle.scatter(s, *mirror, 0, L, bt_dst[b0:b0 + nb], ct, np.fromfile(path, np.uint8))
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"


def _offloaded_files(tmp_path, seed, s, n, ct):
    """Chunk files of n seeded blocks written by the ring's offload; returns
    (chunks, cache, mirror, bt_dst)."""
    L, BS = s.num_layers, s.block_size
    bpc = ct // BS
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, n, n)
    fill = Filled(seed, kvsynth.ROLE_NEW, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    chunks = [(kvx.kvx_chunk_path(str(tmp_path), "q", 0x2545F4914F6CDD1D * (i + 1) + seed), b,
               min(bpc, n - b)) for i, b in enumerate(range(0, n, bpc))]
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    try:
        ring.bind_offload_files(cache, 0, L, ct, chunks, io_depth=4)
        kvx.kvx_offload_to_staging(ring, _bt(bt_src))
        kvx.kvx_check()
    finally:
        ring.close()
    return chunks, cache, mirror, bt_dst


OVERLAP_CASES = [
    # (shape args, n, chunk_tokens, files preloaded first, ring slots, hip_copies, read delay us)
    ((4, 400, 16, 2, 64, 2), 150, 64, 0, 2, False, 0),      # every file read while restoring
    ((4, 400, 16, 2, 64, 2), 150, 64, 19, 2, False, 0),     # half staged
    ((4, 400, 16, 2, 64, 2), 150, 64, 38, 2, False, 0),     # all staged
    ((4, 400, 16, 2, 64, 2), 150, 64, 7, 2, True, 0),       # copies through the runtime
    ((4, 400, 16, 2, 64, 2), 100, 64, 5, 2, False, 3000),   # slow reads: pieces wait for files
    ((4, 400, 16, 2, 64, 2), 100, 64, 5, 1, False, 3000),   # one slot, slow reads
    ((3, 300, 5, 2, 16, 2), 70, 15, 7, 3, False, 1000),     # 320-byte slabs, 2 KiB files
    ((4, 400, 16, 2, 64, 2, 1), 90, 64, 9, 2, False, 1000),  # HND cache layout
    ((4, 400, 16, 2, 64, 2, 2), 90, 64, 3, 2, False, 1000),  # paged-attention cache layout
]


@pytest.mark.parametrize("case", OVERLAP_CASES, ids=[f"o{i}" for i in range(len(OVERLAP_CASES))])
def test_restore_overlapping_the_preload(tmp_path, case):
    shape_args, n, ct, n_pre, slots, hip_copies, delay = case
    s = oracle.Shape(*shape_args)
    L = s.num_layers
    chunks, cache, mirror, bt_dst = _offloaded_files(tmp_path, 700 + n + n_pre + slots, s, n, ct)
    paths = [c[0] for c in chunks]
    per_block = oracle.packed_bytes(s, 0, L, 1)
    slot = -(-(ct // s.block_size) * per_block // 4096) * 4096
    ring = kvx.StagingRing(DEV, slots, 64 << 10)
    pre = kvx.Preloader(len(chunks) + 2, slot, io_depth=4, reserve=2, pinned=True)
    try:
        ring.set_test_hooks(hip_copies=hip_copies)
        pre.hint(paths[:n_pre])
        pre.wait_idle()
        pre.set_test_hooks(delay_us=delay)
        ring.bind_preloaded(cache, 0, L, ct, pre, chunks)
        kvx.kvx_restore_from_staging(ring, _bt(bt_dst))
        torch.cuda.synchronize()
        kvx.kvx_check()
        st = pre.stats()
        assert st["held"] == 0, "the restore dropped its holds"
        assert st["hits_ready"] == n_pre and st["demand_reads"] == len(paths) - n_pre
        assert ring.stats()["dma"] == (0 if hip_copies else 1)
        pre.set_test_hooks(delay_us=0)
        kvx.kvx_restore_from_staging(ring, _bt(bt_dst))  # again: every image cached now
        torch.cuda.synchronize()
        kvx.kvx_check()
        assert pre.stats()["hits_ready"] == n_pre + len(paths)
    finally:
        ring.close()
        pre.close()
    for path, b0, nb in chunks:
        oracle.scatter(s, *mirror, 0, L, bt_dst[b0:b0 + nb], ct, np.fromfile(path, np.uint8))
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"


def test_bind_preloaded_errors(tmp_path):
    s = oracle.Shape(2, 300, 16, 2, 64, 2)
    n, ct = 64, 64
    chunks, cache, _, bt_dst = _offloaded_files(tmp_path, 801, s, n, ct)
    per_block = oracle.packed_bytes(s, 0, 2, 1)
    slot = 4 * per_block
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    try:
        plain = kvx.Preloader(4, slot, pinned=False)
        try:
            with pytest.raises(kvx.KvxError) as ei:  # a restore copies out of pinned slots only
                ring.bind_preloaded(cache, 0, 2, ct, plain, chunks)
            assert ei.value.status == kvx.KVX_EINVAL
        finally:
            plain.close()
        pre = kvx.Preloader(len(chunks) - 1, slot, io_depth=2, pinned=True)
        try:
            with pytest.raises(kvx.KvxError) as ei:  # one path, two chunk sizes
                ring.bind_preloaded(cache, 0, 2, ct, pre, [(chunks[0][0], 0, 4), (chunks[0][0], 4, 2)])
            assert ei.value.status == kvx.KVX_EINVAL
            ring.bind_preloaded(cache, 0, 2, ct, pre, chunks)
            with pytest.raises(kvx.KvxError) as ei:  # more files than the pool holds
                kvx.kvx_restore_from_staging(ring, _bt(bt_dst))
            assert ei.value.status == kvx.KVX_ENOMEM
            assert pre.stats()["held"] == 0
        finally:
            pre.close()
        pre = kvx.Preloader(len(chunks), slot, io_depth=2, pinned=True)
        try:
            bad = chunks[len(chunks) // 2][0]
            data = np.fromfile(bad, np.uint8)
            data[:-4096].tofile(bad)               # a short file in the middle
            ring.bind_preloaded(cache, 0, 2, ct, pre, chunks)
            with pytest.raises(kvx.KvxError) as ei:
                kvx.kvx_restore_from_staging(ring, _bt(bt_dst))
            assert ei.value.status == kvx.KVX_EIO
            torch.cuda.synchronize()
            kvx.kvx_check()
            assert pre.stats()["held"] == 0
            data.tofile(bad)                       # whole again: the same binding restores
            kvx.kvx_restore_from_staging(ring, _bt(bt_dst))
            torch.cuda.synchronize()
            kvx.kvx_check()
        finally:
            pre.close()
    finally:
        ring.close()


def test_abort_while_the_restore_waits_for_a_file(tmp_path):
    s = oracle.Shape(2, 300, 16, 2, 64, 2)
    n, ct = 64, 64
    chunks, cache, _, bt_dst = _offloaded_files(tmp_path, 803, s, n, ct)
    slot = 4 * oracle.packed_bytes(s, 0, 2, 1)
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    pre = kvx.Preloader(len(chunks), slot, io_depth=1, pinned=True)
    try:
        pre.set_test_hooks(delay_us=100000)        # 16 files: 1.6 s of reads
        ring.bind_preloaded(cache, 0, 2, ct, pre, chunks)
        timer = threading.Timer(0.25, ring.abort)
        timer.start()
        t0 = time.perf_counter()
        with pytest.raises(kvx.KvxError) as ei:
            kvx.kvx_restore_from_staging(ring, _bt(bt_dst))
        assert ei.value.status == kvx.KVX_ECLOSED
        assert time.perf_counter() - t0 < 1.0
        timer.join()
        torch.cuda.synchronize()
        kvx.kvx_check()
        assert pre.stats()["held"] == 0
        pre.set_test_hooks(delay_us=0)
        pre.wait_idle()
    finally:
        ring.close()
        pre.close()


def test_preloaded_restore_with_a_file_named_twice(tmp_path):
    # Two chunks restore the same file into different block ranges (identical
    # content restored twice): the file is held and read once, and both ranges
    # receive its image.
    s = oracle.Shape(2, 300, 16, 2, 64, 2)
    n, ct = 32, 64
    chunks, cache, mirror, bt_dst = _offloaded_files(tmp_path, 811, s, n, ct)
    twice = chunks + [(chunks[0][0], n, 4)]            # chunk 0's file again, for 4 more blocks
    extra = [b for b in range(s.num_blocks) if b not in set(bt_dst)][:4]
    bt = np.concatenate([bt_dst, np.asarray(extra, np.int32)])
    slot = 4 * oracle.packed_bytes(s, 0, 2, 1)
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    pre = kvx.Preloader(len(chunks) + 1, slot, io_depth=2, pinned=True)
    try:
        ring.bind_preloaded(cache, 0, 2, ct, pre, twice)
        kvx.kvx_restore_from_staging(ring, _bt(bt))
        torch.cuda.synchronize()
        kvx.kvx_check()
        st = pre.stats()
        assert st["demand_fetches"] == len(chunks) and st["bytes_read"] == sum(
            np.fromfile(p, np.uint8).size for p, _, _ in chunks)
        assert st["held"] == 0
    finally:
        ring.close()
        pre.close()
    for path, b0, nb in twice:
        oracle.scatter(s, *mirror, 0, 2, bt[b0:b0 + nb], ct, np.fromfile(path, np.uint8))
    for l in range(2):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"
