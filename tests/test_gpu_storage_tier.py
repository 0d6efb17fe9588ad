"""GPU parity of the storage tier (Secs. 6.3, 6.4): offload paged blocks to
hash-addressed chunk files through the staging ring (gather -> D2H -> file
writes by the io_uring reactor -> publication by hard link), then restore
them from the files (reads into slots -> H2D -> scatter), each bit-exact
against the oracle; plus the error paths (missing file) and an abort."""
import os
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


def _chunks(root, n, bpc, tag="m"):
    out = []
    for i, b in enumerate(range(0, n, bpc)):
        out.append((kvx.kvx_chunk_path(str(root), tag, 0x9E3779B97F4A7C15 * (i + 1)), b,
                    min(bpc, n - b)))
    return out


PA, HND = oracle.LAYOUT_PAGED_ATTN, oracle.LAYOUT_HND
CASES = [
    # (shape args, n, chunk_tokens, slots, slot_bytes, io_depth, hip_copies[, (l0, l1)])
    ((4, 400, 16, 2, 64, 2), 150, 64, 2, 256 << 10, 4, False),   # several chunks per slot
    ((4, 400, 16, 2, 64, 2), 150, 64, 3, 48 << 10, 2, False),    # chunks split by layers
    ((4, 400, 16, 2, 64, 2), 150, 64, 2, 256 << 10, 1, True),    # copies through the runtime
    ((3, 300, 5, 2, 16, 2), 70, 15, 2, 64 << 10, 8, False),      # 320-byte slabs: buffered I/O
    ((4, 400, 16, 2, 64, 2, PA), 150, 64, 2, 64 << 10, 4, False),  # paged-attention cache
    ((5, 300, 16, 1, 128, 2, HND), 90, 48, 3, 128 << 10, 2, False, (1, 4)),  # HND, layers 1..3
]


@pytest.mark.parametrize("case", CASES, ids=[f"c{i}" for i in range(len(CASES))])
def test_offload_to_files_then_restore_from_files(tmp_path, case):
    shape_args, n, ct, slots, slot_bytes, depth, hip_copies = case[:7]
    s = oracle.Shape(*shape_args)
    L, BS = s.num_layers, s.block_size
    l0, l1 = case[7] if len(case) > 7 else (0, L)
    seed = 300 + n + depth
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, n, n)
    fill = Filled(seed, kvsynth.ROLE_NEW, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    chunks = _chunks(tmp_path, n, ct // BS)
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    try:
        ring.set_test_hooks(hip_copies=hip_copies)
        ring.bind_offload_files(cache, l0, l1, ct, chunks, io_depth=depth)
        kvx.kvx_offload_to_staging(ring, _bt(bt_src))
        kvx.kvx_check()
        for path, b0, nb in chunks:  # every file holds its chunk's image, published
            exp = oracle.gather(s, *mirror, l0, l1, bt_src[b0:b0 + nb], ct)
            got = np.fromfile(path, dtype=np.uint8)
            assert np.array_equal(got, exp), f"chunk file {path} differs"
        assert not [f for d, _, fs in os.walk(tmp_path) for f in fs if ".tmp." in f]
        # restore the files into fresh blocks
        ring.bind_files(cache, l0, l1, ct, chunks, io_depth=depth)
        for _ in range(2):
            kvx.kvx_restore_from_staging(ring, _bt(bt_dst))
        torch.cuda.synchronize()
        kvx.kvx_check()
    finally:
        ring.close()
    for path, b0, nb in chunks:
        oracle.scatter(s, *mirror, l0, l1, bt_dst[b0:b0 + nb], ct, np.fromfile(path, np.uint8))
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"


def test_missing_file_fails_the_restore_with_eio(tmp_path):
    s = oracle.Shape(2, 100, 16, 2, 64, 2)
    n, ct = 32, 64
    (bt,) = seeded_ids(5, s.num_blocks, n)
    cache = device_cache(s, Filled(5, kvsynth.ROLE_DST), DEV)
    chunks = _chunks(tmp_path, n, ct // 16)
    img = kvsynth.host_bytes(oracle.packed_bytes(s, 0, 2, n), 5, 9)
    per_chunk = oracle.packed_bytes(s, 0, 2, 4)
    kvx.kvx_write_files([(p, img[i * per_chunk:(i + 1) * per_chunk], 0)
                         for i, (p, _, _) in enumerate(chunks[:-1])])  # the last one is missing
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    try:
        ring.bind_files(cache, 0, 2, ct, chunks, io_depth=4)
        with pytest.raises(kvx.KvxError) as ei:
            kvx.kvx_restore_from_staging(ring, _bt(bt))
        assert ei.value.status == kvx.KVX_EIO
        torch.cuda.synchronize()
        kvx.kvx_check()
        # once the file exists the same binding restores everything
        kvx.kvx_write_files([(chunks[-1][0], img[(len(chunks) - 1) * per_chunk:], 0)])
        kvx.kvx_restore_from_staging(ring, _bt(bt))
        torch.cuda.synchronize()
        kvx.kvx_check()
    finally:
        ring.close()
    mirror = host_mirror(s, Filled(5, kvsynth.ROLE_DST), range(s.num_blocks))
    oracle.scatter(s, *mirror, 0, 2, bt, ct, img)
    for l in range(2):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"


def test_abort_during_file_offload(tmp_path):
    s = oracle.Shape(2, 3000, 16, 2, 64, 2)
    n = 1200
    (bt,) = seeded_ids(13, s.num_blocks, n)
    cache = device_cache(s, Filled(13, kvsynth.ROLE_NEW), DEV)
    chunks = _chunks(tmp_path, n, 4)
    ring = kvx.StagingRing(DEV, 2, 64 << 10)
    try:
        ring.bind_offload_files(cache, 0, 2, 64, chunks, io_depth=1)
        t = threading.Thread(target=lambda: (time.sleep(0.02), ring.abort()))
        t.start()
        t0 = time.perf_counter()
        try:
            kvx.kvx_offload_to_staging(ring, _bt(bt))
        except kvx.KvxError as e:
            assert e.status == kvx.KVX_ECLOSED
        t.join()
        assert time.perf_counter() - t0 < 10.0
        torch.cuda.synchronize()
        kvx.kvx_check()
    finally:
        ring.close()
    # whatever was published is whole; nothing half-written is left
    per_chunk = oracle.packed_bytes(s, 0, 2, 4)
    for path, _, _ in chunks:
        if os.path.exists(path):
            assert os.path.getsize(path) == per_chunk
    assert not [f for d, _, fs in os.walk(tmp_path) for f in fs if ".tmp." in f]


def test_read_files_into_pinned_memory_with_several_transfers_per_file(tmp_path):
    """Direct reads into pinned memory fail (EFAULT) and are repeated on a
    buffered descriptor; with several transfers of one file in flight, the
    others (still on the old descriptor) must be repeated too, not fail."""
    rng = np.random.default_rng(77)
    files = []
    for i in range(6):
        data = rng.integers(0, 256, 4 << 20, dtype=np.uint8)
        p = tmp_path / f"r{i}.kvc"
        data.tofile(p)
        files.append((str(p), data))
    dst = kvx.PinnedBuffer(len(files) * (4 << 20))
    ops = []
    for i, (p, _) in enumerate(files):
        for q in range(4):  # four 1 MiB transfers per file, all in flight together
            off = q << 20
            ops.append((p, dst.array[i * (4 << 20) + off:i * (4 << 20) + off + (1 << 20)], off))
    kvx.kvx_read_files(ops, io_depth=16)
    for i, (_, data) in enumerate(files):
        assert np.array_equal(dst.array[i * (4 << 20):(i + 1) * (4 << 20)], data), f"file {i}"
    dst.free()
