"""GPU parity of the fused chunk-list kernels on random geometries
(derandomized hypothesis draws, so every run checks the same cases): cache
layout, block size, heads, head dim, element size, layer range and chunk size;
a batch of up to 48 chunks of 1 to bpc blocks each (ragged), whose block-table
slices are taken in a shuffled order and whose images sit in the packed buffer
in another shuffled order with 16-byte-multiple gaps.

The oracle's side of a chunk list is its plain definition: chunk c is the
oracle gather of its own blocks, as one chunk, at its packed offset. The
gathered buffer is compared whole (every image right, every gap byte still the
canary); after the scatter of that buffer into fresh blocks every cache tensor
is compared whole with the oracle's per-chunk scatters."""
import numpy as np
import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import HealthCheck, example, given, settings, strategies as st  # noqa: E402

import kvsynth  # noqa: E402
import oracle  # noqa: E402
from kvtest_util import Filled, device_cache, first_mismatch, host_mirror, to_host  # noqa: E402

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
NHD, HND, PA = oracle.LAYOUT_NHD, oracle.LAYOUT_HND, oracle.LAYOUT_PAGED_ATTN
CANARY = 0xA5


@st.composite
def batches(draw):
    layout = draw(st.sampled_from([NHD, NHD, HND, PA]))
    elem = draw(st.sampled_from([2, 2, 1, 4]))
    BS = draw(st.sampled_from([1, 4, 8, 16, 16, 32]))
    H = draw(st.integers(1, 8))
    D = draw(st.sampled_from([16, 32, 64, 128]))
    while BS * H * D * elem > 16 * 1024:  # keep the cache small
        if H > 1:
            H //= 2
        else:
            BS //= 2
    L = draw(st.sampled_from([1, 2, 3, 5, 8]))
    l0 = draw(st.integers(0, L - 1))
    l1 = draw(st.integers(l0 + 1, L))
    bpc = draw(st.sampled_from([1, 2, 3, 4, 16]))
    n_chunks = draw(st.integers(1, 48))
    seed = draw(st.integers(0, 10**6))
    return layout, elem, BS, H, D, L, l0, l1, bpc, n_chunks, seed


def _plan(seed, bpc, n_chunks, per_block):
    """Chunk sizes, their table slices (shuffled) and packed offsets
    (shuffled, with gaps): refs (packed_offset, bt_offset, n_blocks)."""
    rng = np.random.default_rng(seed)
    sizes = [int(rng.integers(1, bpc + 1)) for _ in range(n_chunks)]
    bt_off, at = [0] * n_chunks, 0
    for c in rng.permutation(n_chunks):
        bt_off[c] = at
        at += sizes[c]
    pk_off, off = [0] * n_chunks, 16 * int(rng.integers(0, 64))
    for c in rng.permutation(n_chunks):
        pk_off[c] = off
        off += sizes[c] * per_block + 16 * int(rng.integers(0, 5))
    refs = [(pk_off[c], bt_off[c], sizes[c]) for c in range(n_chunks)]
    return refs, at, off + 4096


@settings(max_examples=30, deadline=None, derandomize=True, database=None,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(batches())
@example((NHD, 2, 16, 8, 64, 8, 0, 8, 16, 40, 3))   # 16 KiB slabs, 256-token chunks
@example((PA, 2, 16, 4, 64, 3, 1, 3, 4, 48, 4))     # paged attention, two of three layers
@example((HND, 1, 32, 2, 128, 2, 0, 2, 3, 17, 5))   # byte elements, three-block chunks
@example((NHD, 4, 1, 1, 16, 1, 0, 1, 1, 1, 6))      # one 64-byte slab
def test_random_chunk_lists_bit_exact(case):
    layout, elem, BS, H, D, L, l0, l1, bpc, n_chunks, seed = case
    ct = bpc * BS
    s0 = oracle.Shape(L, 1, BS, H, D, elem, layout)
    per_block = oracle.packed_bytes(s0, l0, l1, 1)
    refs, n_ids, total = _plan(seed, bpc, n_chunks, per_block)
    NB = 2 * n_ids + 5
    s = oracle.Shape(L, NB, BS, H, D, elem, layout)
    print(f"case {case}: {n_ids} blocks in {n_chunks} chunks, packed {total} B", flush=True)
    perm = np.random.default_rng(seed + 1).permutation(NB).astype(np.int32)
    bt_src, bt_dst = perm[:n_ids].copy(), perm[n_ids:2 * n_ids].copy()
    fill = Filled(seed, kvsynth.ROLE_SRC, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, range(NB))
    dref = kvx.chunk_refs(refs, DEV)

    expect = np.full(total, CANARY, dtype=np.uint8)
    for off, b0, nb in refs:
        img = oracle.gather(s, *mirror, l0, l1, bt_src[b0:b0 + nb], ct)
        expect[off:off + img.size] = img
    packed = torch.full((total,), CANARY, dtype=torch.uint8, device=DEV)
    kvx.kvx_gather_chunks(cache, l0, l1, torch.from_numpy(bt_src).to(DEV), n_ids, dref, n_chunks,
                          ct, packed)
    torch.cuda.synchronize()
    kvx.kvx_check()
    bad = first_mismatch(to_host(packed), expect)
    assert bad is None, f"chunk-list gather differs at byte {bad}"

    kvx.kvx_scatter_chunks(cache, l0, l1, torch.from_numpy(bt_dst).to(DEV), n_ids, dref, n_chunks,
                           ct, packed)
    torch.cuda.synchronize()
    kvx.kvx_check()
    for off, b0, nb in refs:
        oracle.scatter(s, *mirror, l0, l1, bt_dst[b0:b0 + nb], ct,
                       expect[off:off + nb * per_block])
    for l in range(L):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"
    del cache, packed
    torch.cuda.empty_cache()
