"""GPU parity of the staging ring on random configurations (derandomized
hypothesis draws, so every run checks the same cases): cache layout, block
size, heads, head dim, element size and layer range; a contiguous packed image
or a list of ragged chunks in separate host buffers; slot count, a slot size
from one layer of the largest chunk up to several chunks (so pieces are whole
chunks, several chunks or layer ranges); fill or drain threads, or none (the
copies then read or write pinned buffers directly); the DMA engines or the HIP
runtime for the host-link copies; the blocking call or begin / wait.

Each configuration runs its transfer twice in a row on one ring. A restore is
compared with the oracle's scatter of the whole image (every cache tensor
whole: the restored slabs and every other block); an offload compares every
host destination with the oracle's gather of its chunk."""
import numpy as np
import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import HealthCheck, example, given, settings, strategies as st  # noqa: E402

import kvsynth  # noqa: E402
import oracle  # noqa: E402
from kvtest_util import Filled, device_cache, host_mirror, to_host  # noqa: E402

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
NHD, HND, PA = oracle.LAYOUT_NHD, oracle.LAYOUT_HND, oracle.LAYOUT_PAGED_ATTN
IMAGE, CHUNKS, OFFLOAD = "image", "chunks", "offload"


@st.composite
def rings(draw):
    layout = draw(st.sampled_from([NHD, NHD, HND, PA]))
    elem = draw(st.sampled_from([2, 2, 1, 4]))
    BS = draw(st.sampled_from([1, 4, 16, 16, 32]))
    H = draw(st.integers(1, 8))
    D = draw(st.sampled_from([32, 64, 128]))
    while BS * H * D * elem > 16 * 1024:  # keep the cache small
        if H > 1:
            H //= 2
        else:
            BS //= 2
    L = draw(st.sampled_from([1, 2, 3, 5]))
    l0 = draw(st.integers(0, L - 1))
    l1 = draw(st.integers(l0 + 1, L))
    bpc = draw(st.sampled_from([1, 2, 3, 4, 16]))
    n_chunks = draw(st.integers(1, 24))
    mode = draw(st.sampled_from([IMAGE, CHUNKS, OFFLOAD]))
    slots = draw(st.integers(1, 6))
    slot_layers = draw(st.integers(1, 2 * (l1 - l0) + 1))  # slot size, in layers of a full chunk
    threads = draw(st.sampled_from([0, 1, 2, 5]))
    hip_copies = draw(st.booleans())
    use_async = draw(st.booleans())
    seed = draw(st.integers(0, 10**6))
    return (layout, elem, BS, H, D, L, l0, l1, bpc, n_chunks, mode, slots, slot_layers, threads,
            hip_copies, use_async, seed)


def _host(nbytes, pinned, fill=None):
    """A host buffer of nbytes: pinned (PinnedBuffer) or pageable (numpy)."""
    if pinned:
        b = kvx.PinnedBuffer(nbytes)
        b.array[:] = 0xEE if fill is None else fill
        return b
    return np.full(nbytes, 0xEE, np.uint8) if fill is None else fill.copy()


def _arr(b):
    return b.array if isinstance(b, kvx.PinnedBuffer) else b


@settings(max_examples=30, deadline=None, derandomize=True, database=None,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(rings())
@example((NHD, 2, 16, 8, 64, 5, 0, 5, 16, 9, IMAGE, 2, 1, 2, False, True, 1))    # layer pieces
@example((PA, 2, 16, 2, 128, 3, 1, 3, 4, 20, CHUNKS, 1, 5, 0, False, False, 2))  # one slot, pinned
@example((HND, 1, 32, 1, 128, 2, 0, 2, 3, 11, OFFLOAD, 3, 2, 0, True, True, 3))  # runtime D2H
@example((NHD, 4, 4, 3, 32, 3, 0, 3, 2, 24, OFFLOAD, 6, 7, 5, False, False, 4))  # many chunks a slot
@example((PA, 2, 16, 4, 64, 2, 0, 2, 16, 7, OFFLOAD, 2, 1, 2, False, True, 5))    # layer pieces, async
@example((NHD, 2, 16, 2, 128, 5, 2, 4, 4, 13, OFFLOAD, 1, 3, 1, True, False, 6))  # one slot, runtime
@example((HND, 2, 4, 8, 64, 3, 0, 3, 3, 15, CHUNKS, 3, 2, 2, False, True, 7))     # restore, async DMA
def test_random_ring_transfers_equal_oracle(case):
    (layout, elem, BS, H, D, L, l0, l1, bpc, n_chunks, mode, slots, slot_layers, threads,
     hip_copies, use_async, seed) = case
    ct = bpc * BS
    rng = np.random.default_rng(seed)
    sizes = [bpc] * n_chunks if mode == IMAGE else [int(rng.integers(1, bpc + 1))
                                                    for _ in range(n_chunks)]
    if mode == IMAGE:
        sizes[-1] = int(rng.integers(1, bpc + 1))  # a compact last chunk
    n = sum(sizes)
    NB = 2 * n + 7
    s = oracle.Shape(L, NB, BS, H, D, elem, layout)
    per_block = oracle.packed_bytes(s, l0, l1, 1)
    layer_bytes = bpc * 2 * s.slab_bytes  # one layer of a full chunk
    slot_bytes = -(-layer_bytes * slot_layers // 4096) * 4096
    print(f"case {case}: {n} blocks in {n_chunks} chunks, slot {slot_bytes} B", flush=True)
    bt = np.random.default_rng(seed + 1).permutation(NB)[:n].astype(np.int32)
    bt_off = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(int)
    pinned = threads == 0
    role = kvsynth.ROLE_NEW if mode == OFFLOAD else kvsynth.ROLE_DST
    fill = Filled(seed, role, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(NB))
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    bufs = []
    try:
        ring.set_test_hooks(hip_copies=hip_copies)
        if mode == IMAGE:
            img = kvsynth.host_bytes(n * per_block, seed, 0x51, mode=kvsynth.MODE_RAW)
            bufs = [_host(img.size, pinned, img)]
            ring.bind(cache, l0, l1, n, ct, bufs[0], fill_threads=threads)
        elif mode == CHUNKS:
            bufs = [_host(nb * per_block, pinned,
                          kvsynth.host_bytes(nb * per_block, seed, 0x52 + i, mode=kvsynth.MODE_RAW))
                    for i, nb in enumerate(sizes)]
            order = rng.permutation(n_chunks)  # chunks listed out of table order
            ring.bind_chunks(cache, l0, l1, ct,
                             [(bufs[c], int(bt_off[c]), sizes[c]) for c in order],
                             fill_threads=threads)
        else:
            bufs = [_host(nb * per_block, pinned) for nb in sizes]
            order = rng.permutation(n_chunks)
            ring.bind_offload(cache, l0, l1, ct,
                              [(bufs[c], int(bt_off[c]), sizes[c]) for c in order],
                              drain_threads=threads)
        table = torch.from_numpy(bt).to(DEV)
        torch.cuda.synchronize()
        for _ in range(2):  # slots and events carry over between calls
            if mode == OFFLOAD:
                if use_async:
                    kvx.kvx_offload_begin(ring, table)
                    kvx.kvx_offload_wait(ring)
                else:
                    kvx.kvx_offload_to_staging(ring, table)
            elif use_async:
                kvx.kvx_restore_begin(ring, table)
                kvx.kvx_restore_wait(ring)
            else:
                kvx.kvx_restore_from_staging(ring, table)
            torch.cuda.synchronize()
            kvx.kvx_check()
        assert ring.stats()["dma"] == (0 if hip_copies else 1)
    finally:
        ring.close()
    if mode == OFFLOAD:
        for c, nb in enumerate(sizes):
            exp = oracle.gather(s, *mirror, l0, l1, bt[bt_off[c]:bt_off[c] + nb], ct)
            assert np.array_equal(_arr(bufs[c]), exp), f"offloaded chunk {c} differs"
    else:
        if mode == IMAGE:
            oracle.restore(s, *mirror, l0, l1, bt, ct, _arr(bufs[0]))
        else:
            for c, nb in enumerate(sizes):
                oracle.scatter(s, *mirror, l0, l1, bt[bt_off[c]:bt_off[c] + nb], ct, _arr(bufs[c]))
        for l in range(L):
            assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
            assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"
    for b in bufs:
        if isinstance(b, kvx.PinnedBuffer):
            b.free()
    del cache
    torch.cuda.empty_cache()
