"""The scatter entry point that allocates nothing (kvx_scatter_blocks_noalloc),
called through the C ABI: two calls in a row, the second smaller, each
bit-exact against kvx_scatter_blocks on an identical cache (and against the
oracle), a call below the ordering threshold, and sizes beyond the fixed
scratch rejected on the host."""
import ctypes

import numpy as np
import pytest

import kvsynth
import oracle
from kvtest_util import Filled, device_cache, host_mirror, seeded_ids, to_host

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402
from paper_2609_11744_amd import _native  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _bt(ids):
    return torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(DEV)


def _call(fn, cache, L, bt, n, ct, src):
    return fn(ctypes.byref(cache.c_struct()), 0, L, bt.data_ptr(), n, ct, src.data_ptr(),
              torch.cuda.current_stream().cuda_stream)


def test_noalloc_scatter_matches_scatter_twice_smaller_second():
    lib = _native.lib()
    s = oracle.Shape(2, 7000, 16, 8, 64, 2)  # 16 KiB slabs: scatters of 1,024+ blocks ordered
    L, ct, seed = 2, 256, 91
    fill = Filled(seed, kvsynth.ROLE_DST, kvsynth.MODE_RAW)
    ref = device_cache(s, fill, DEV)
    new = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(s.num_blocks))
    first, second, third = seeded_ids(seed, s.num_blocks, 3000, 1500, 600)
    for i, ids in enumerate((first, second, third)):  # 3000, then 1500, then below 1024
        n = len(ids)
        img = kvsynth.host_bytes(oracle.packed_bytes(s, 0, L, n), seed, 1000 + i,
                                 mode=kvsynth.MODE_RAW)
        src = torch.from_numpy(img).to(DEV)
        bt = _bt(ids)
        assert _call(lib.kvx_scatter_blocks, ref, L, bt, n, ct, src) == kvx.KVX_OK
        assert _call(lib.kvx_scatter_blocks_noalloc, new, L, bt, n, ct, src) == kvx.KVX_OK
        torch.cuda.synchronize()
        kvx.kvx_check()
        oracle.scatter(s, *mirror, 0, L, ids, ct, img)
        for l in range(L):
            for a, b, m in ((new.k[l], ref.k[l], mirror[0][l]), (new.v[l], ref.v[l], mirror[1][l])):
                # compared as bytes: raw words include NaN patterns
                assert torch.equal(a.view(torch.int16), b.view(torch.int16)), \
                    f"call {i} (n={n}): layer {l} differs from kvx_scatter_blocks"
                assert np.array_equal(to_host(a), m), f"call {i} (n={n}): layer {l} differs from the oracle"


def test_noalloc_scatter_rejects_sizes_beyond_its_scratch():
    lib = _native.lib()
    s = oracle.Shape(1, 70000, 1, 1, 8, 2)  # 16-byte slabs: the pool holds more than the limit
    cache = kvx.PagedKVCache.allocate(1, s.num_blocks, 1, 1, 8, torch.bfloat16, DEV)
    n = kvx.KVX_NOALLOC_MAX_BLOCKS + 1
    bt = torch.zeros(n, dtype=torch.int32, device=DEV)
    src = torch.zeros(oracle.packed_bytes(s, 0, 1, n), dtype=torch.uint8, device=DEV)
    assert _call(lib.kvx_scatter_blocks_noalloc, cache, 1, bt, n, 1, src) == kvx.KVX_EINVAL
    torch.cuda.synchronize()
    kvx.kvx_check()
