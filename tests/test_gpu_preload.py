"""GPU parity of restores from preloaded chunk images (Sec. 6.5): chunk files
written by the ring's offload are read ahead into a pinned preloader pool;
the request's fetch claims the staged images and reads the others on demand;
the ring restores straight from the pool (fill_threads 0: host-to-device
copies out of the pinned slots), bit-exact against the oracle's scatter of
the file contents."""
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
