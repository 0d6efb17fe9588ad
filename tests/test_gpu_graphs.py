"""The copy kernels under HIP graph capture: a gather + scatter + chunk-list
gather step (sizes that take no scratch allocation: scatters below the
destination-ordering threshold), and a destination-ordered scatter through
kvx_scatter_blocks_noalloc (its order table in the library's fixed array),
each captured once and replayed several times with eager work and
synchronizations between replays, and every replay checked bit-exact against
the oracle of what it computes."""
import numpy as np
import pytest

import kvsynth
import oracle
from kvtest_util import Filled, device_cache, host_mirror, seeded_ids, to_host

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_captured_step_replays_bit_exact():
    s = oracle.Shape(3, 600, 16, 2, 64, 2)
    n, ct, L = 200, 64, 3
    seed = 71
    bt_src, bt_dst = seeded_ids(seed, s.num_blocks, n, n)
    fill = Filled(seed, kvsynth.ROLE_SRC, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    t_src = torch.from_numpy(bt_src.astype(np.int32)).to(DEV)
    t_dst = torch.from_numpy(bt_dst.astype(np.int32)).to(DEV)
    nbytes = oracle.packed_bytes(s, 0, L, n)
    packed = torch.zeros(nbytes, dtype=torch.uint8, device=DEV)
    packed2 = torch.zeros(nbytes, dtype=torch.uint8, device=DEV)
    per_block = oracle.packed_bytes(s, 0, L, 1)
    bpc = ct // 16
    refs = kvx.chunk_refs([(b * per_block, b, min(bpc, n - b)) for b in range(0, n, bpc)], DEV)
    n_refs = (n + bpc - 1) // bpc

    def step():
        kvx.kvx_gather_blocks(cache, 0, L, t_src, n, ct, packed)
        kvx.kvx_scatter_blocks(cache, 0, L, t_dst, n, ct, packed)
        kvx.kvx_gather_chunks(cache, 0, L, t_dst, n, refs, n_refs, ct, packed2)

    step()  # eager first: one-time setup stays out of the capture
    torch.cuda.synchronize()
    kvx.kvx_check()
    expect = oracle.gather(s, *mirror, 0, L, bt_src, ct)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        # eager work between replays: clear the outputs and the destinations
        packed.zero_()
        packed2.fill_(0x33)
        for l in range(L):
            cache.k[l].view(torch.uint8).view(s.num_blocks, -1)[t_dst.long()] = 0
            cache.v[l].view(torch.uint8).view(s.num_blocks, -1)[t_dst.long()] = 0
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        kvx.kvx_check()
        assert np.array_equal(to_host(packed), expect), f"replay {rep}: gather"
        assert np.array_equal(to_host(packed2), expect), f"replay {rep}: chunk-list gather"
        m = ([a.copy() for a in mirror[0]], [a.copy() for a in mirror[1]])
        oracle.scatter(s, *m, 0, L, bt_dst, ct, expect)
        for l in range(L):
            assert np.array_equal(to_host(cache.k[l]), m[0][l]), f"replay {rep}: K layer {l}"
            assert np.array_equal(to_host(cache.v[l]), m[1][l]), f"replay {rep}: V layer {l}"


def test_captured_noalloc_ordered_scatter_replays_bit_exact():
    """kvx_scatter_blocks_noalloc under graph capture: a scatter large enough to
    run in destination order (its order table in the library's fixed array,
    nothing allocated), captured once and replayed with a new packed image
    loaded into the same buffer before each replay; every replay against the
    oracle's scatter of that image."""
    import ctypes

    from paper_2609_11744_amd import _native

    s = oracle.Shape(2, 4000, 16, 8, 64, 2)  # 16 KiB slabs
    n, ct, L = 1500, 64, 2
    seed = 73
    assert kvx.kvx_copy_walk(kvx.shape_only_cache(2, 4000, 16, 8, 64, 2), 0, L, n, ct,
                             False)["ordered"] == 1
    (bt_dst,) = seeded_ids(seed, s.num_blocks, n)
    fill = Filled(seed, kvsynth.ROLE_DST, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    t_dst = torch.from_numpy(bt_dst.astype(np.int32)).to(DEV)
    nbytes = oracle.packed_bytes(s, 0, L, n)
    packed = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    lib = _native.lib()

    def step():
        st = lib.kvx_scatter_blocks_noalloc(ctypes.byref(cache.c_struct()), 0, L, t_dst.data_ptr(), n,
                                            ct, packed.data_ptr(),
                                            torch.cuda.current_stream().cuda_stream)
        assert st == kvx.KVX_OK

    packed.copy_(torch.from_numpy(kvsynth.host_bytes(nbytes, seed, 500, mode=kvsynth.MODE_RAW)))
    step()  # eager first: the scratch array's address is resolved outside the capture
    torch.cuda.synchronize()
    kvx.kvx_check()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        img = kvsynth.host_bytes(nbytes, seed, 501 + rep, mode=kvsynth.MODE_RAW)
        packed.copy_(torch.from_numpy(img))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        kvx.kvx_check()
        oracle.scatter(s, *mirror, 0, L, bt_dst, ct, img)
        for l in range(L):
            assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"replay {rep}: K layer {l}"
            assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"replay {rep}: V layer {l}"
