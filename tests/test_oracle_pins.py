"""Pins for the CPU oracle, checked against what the paper and plain
mathematics fix rather than against the oracle itself.

* Size model: the paper's printed 3B figures (Sec. 2.1, Sec. 4.1, Sec. 6.4).
* Special cases that reduce to a memcpy or to numpy fancy indexing.
* Invariants: round trip, block relabelling, untouched bytes, chunk-size
  independence, layer-range decomposition.
* Brute force: the element-wise oracle (O1) equals the slab oracle (O2) on
  every tiny shape of a small grid.
"""
import itertools
import json
import os

import numpy as np
import pytest

import kvsynth
import oracle
from oracle import Shape

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _mirror(shape, seed, role=kvsynth.ROLE_SRC, mode=kvsynth.MODE_RAW):
    k, v = oracle.new_mirror(shape)
    for l in range(shape.num_layers):
        kvsynth.fill_host(k[l], seed, kvsynth.cache_stream(role, l, 0), mode=mode, threads=1)
        kvsynth.fill_host(v[l], seed, kvsynth.cache_stream(role, l, 1), mode=mode, threads=1)
    return k, v


def _slab(buf, shape, b):
    u = shape.slab_bytes
    return buf[b * u:(b + 1) * u]


def _copy(m):
    return [a.copy() for a in m[0]], [a.copy() for a in m[1]]


def _ids(rng, nb, n):
    return rng.permutation(nb)[:n].astype(np.int32)


# ---- size model -------------------------------------------------------------

def test_bytes_per_token_matches_paper_3b_figures():
    g = json.load(open(os.path.join(GOLDEN, "paper_sizes.json")))
    f = g["public_config_factors"]
    bpt = oracle.bytes_per_token(f["layers"], f["kv_heads"], f["head_dim"], g["dtype_bytes"])
    assert bpt == g["bytes_per_token"] == 112 * 1024
    assert bpt * g["tokens_80k"] == g["bytes_80k_gib"] * 2**30
    # "approximately 28 MiB" for one 256-token storage block (exact here)
    assert bpt * g["storage_block_tokens"] == g["storage_block_mib_approx"] * 2**20


def test_packed_size_is_exact_for_workload_shapes():
    # Llama-8B-shaped KV (32 layers, 8 KV heads, head dim 128, bf16): 128 KiB/token
    assert oracle.bytes_per_token(32, 8, 128, 2) == 131072
    s8 = Shape(32, 20000, 16, 8, 128, 2)
    # 5,000 blocks (80,000 tokens): "~10.5 GB"
    assert oracle.packed_bytes(s8, 0, 32, 5000) == 10_485_760_000
    assert oracle.packed_bytes(s8, 0, 32, 5000) == 80_000 * oracle.bytes_per_token(32, 8, 128, 2)
    # 70B-shaped: 80 layers -> 320 KiB/token
    assert oracle.bytes_per_token(80, 8, 128, 2) == 327680


# ---- special cases ----------------------------------------------------------

@pytest.mark.parametrize("elem_bytes", [1, 2, 4])
def test_identity_table_single_layer_is_memcpy(elem_bytes):
    s = Shape(3, 12, 4, 2, 8, elem_bytes)
    k, v = _mirror(s, 11)
    n, l = 7, 1
    out = oracle.gather(s, k, v, l, l + 1, np.arange(n), n * s.block_size)
    u = s.slab_bytes
    assert np.array_equal(out, np.concatenate([k[l][:n * u], v[l][:n * u]]))


def test_one_block_per_chunk_is_per_block_layer_interleave():
    s = Shape(3, 10, 2, 2, 4, 2)
    k, v = _mirror(s, 12)
    bt = np.array([7, 2, 9, 0], dtype=np.int32)
    out = oracle.gather(s, k, v, 0, 3, bt, s.block_size)
    parts = []
    for b in bt:
        for l in range(3):
            parts += [_slab(k[l], s, b), _slab(v[l], s, b)]
    assert np.array_equal(out, np.concatenate(parts))


def test_single_chunk_single_layer_is_fancy_indexing():
    s = Shape(2, 16, 4, 3, 8, 2)
    k, v = _mirror(s, 13)
    rng = np.random.default_rng(0)
    bt = _ids(rng, s.num_blocks, 5)
    out = oracle.gather(s, k, v, 1, 2, bt, 8 * s.block_size)  # chunk larger than the prefix
    kv = oracle.element_view(k[1], s)[bt].ravel()
    vv = oracle.element_view(v[1], s)[bt].ravel()
    assert np.array_equal(out.view(np.uint16), np.concatenate([kv, vv]))


def test_scatter_of_identity_image_is_memcpy():
    s = Shape(2, 9, 2, 1, 8, 2)
    k, v = oracle.new_mirror(s)
    n, l, u = 4, 0, s.slab_bytes
    img = kvsynth.host_bytes(oracle.packed_bytes(s, l, l + 1, n), 3, 77, mode=kvsynth.MODE_RAW)
    oracle.scatter(s, k, v, l, l + 1, np.arange(n), n * s.block_size, img)
    assert np.array_equal(k[l][:n * u], img[:n * u])
    assert np.array_equal(v[l][:n * u], img[n * u:])
    assert not k[l][n * u:].any() and not v[l][n * u:].any() and not k[1].any()


def test_nan_payloads_and_signed_zero_survive():
    s = Shape(1, 4, 1, 1, 8, 2)
    k, v = oracle.new_mirror(s)
    pats = np.array([0x7FC1, 0xFFFF, 0x8000, 0x0001, 0x7F80, 0xFF81, 0x0000, 0x807F], np.uint16)
    for b in range(4):
        oracle.element_view(k[0], s)[b, 0, 0, :] = np.roll(pats, b)
        oracle.element_view(v[0], s)[b, 0, 0, :] = np.roll(pats, -b)
    out = oracle.gather(s, k, v, 0, 1, [3, 1], 1)
    words = out.view(np.uint16)
    assert np.array_equal(words[:8], np.roll(pats, 3))
    assert np.array_equal(words[8:16], np.roll(pats, -3))
    assert np.array_equal(words[16:24], np.roll(pats, 1))


# ---- invariants -------------------------------------------------------------

SHAPES = [Shape(3, 40, 4, 2, 8, 2), Shape(2, 33, 16, 2, 64, 2), Shape(4, 25, 1, 1, 16, 4)]


@pytest.mark.parametrize("s", SHAPES)
@pytest.mark.parametrize("cpb", [1, 3, 4])
def test_round_trip(s, cpb):
    rng = np.random.default_rng(1)
    n = 11
    ids = rng.permutation(s.num_blocks).astype(np.int32)
    bt_src, bt_dst = ids[:n], ids[n:2 * n]
    src = _mirror(s, 21)
    dst = _mirror(s, 22, role=kvsynth.ROLE_DST)
    before = _copy(dst)
    l0, l1 = 0, s.num_layers
    ct = cpb * s.block_size
    img = oracle.gather(s, *src, l0, l1, bt_src, ct)
    oracle.scatter(s, *dst, l0, l1, bt_dst, ct, img)
    for side in range(2):
        for l in range(l0, l1):
            for j in range(n):
                assert np.array_equal(_slab(dst[side][l], s, bt_dst[j]),
                                      _slab(src[side][l], s, bt_src[j]))
            untouched = np.setdiff1d(np.arange(s.num_blocks), bt_dst)
            for b in untouched:
                assert np.array_equal(_slab(dst[side][l], s, b), _slab(before[side][l], s, b))
    assert np.array_equal(oracle.gather(s, *dst, l0, l1, bt_dst, ct), img)


def test_relabel_equivariance():
    s = Shape(2, 30, 4, 2, 8, 2)
    rng = np.random.default_rng(2)
    k, v = _mirror(s, 31)
    pi = rng.permutation(s.num_blocks)
    k2, v2 = oracle.new_mirror(s)
    for l in range(s.num_layers):
        for b in range(s.num_blocks):
            _slab(k2[l], s, pi[b])[:] = _slab(k[l], s, b)
            _slab(v2[l], s, pi[b])[:] = _slab(v[l], s, b)
    bt = _ids(rng, s.num_blocks, 13)
    for ct in (4, 8, 20, 64):
        a = oracle.gather(s, k, v, 0, 2, bt, ct)
        b = oracle.gather(s, k2, v2, 0, 2, pi[bt].astype(np.int32), ct)
        assert np.array_equal(a, b)


def test_permuting_table_permutes_single_block_chunks():
    s = Shape(2, 20, 4, 1, 8, 2)
    rng = np.random.default_rng(3)
    k, v = _mirror(s, 32)
    bt = _ids(rng, s.num_blocks, 9)
    sigma = rng.permutation(9)
    a = oracle.gather(s, k, v, 0, 2, bt, s.block_size)
    b = oracle.gather(s, k, v, 0, 2, bt[sigma], s.block_size)
    per = 2 * 2 * s.slab_bytes
    assert np.array_equal(b.reshape(9, per), a.reshape(9, per)[sigma])


def test_gather_writes_exactly_the_packed_range():
    s = Shape(2, 20, 4, 2, 8, 2)
    k, v = _mirror(s, 33)
    bt = [4, 9, 1, 16, 3]
    nbytes = oracle.packed_bytes(s, 0, 2, len(bt))
    buf = np.full(nbytes + 4096, 0xA5, dtype=np.uint8)
    oracle.gather(s, k, v, 0, 2, bt, 8, out=buf)
    assert (buf[nbytes:] == 0xA5).all()


def test_scatter_touches_only_named_layers_and_blocks():
    s = Shape(4, 16, 2, 1, 8, 2)
    dst = _mirror(s, 34, role=kvsynth.ROLE_DST)
    before = _copy(dst)
    bt = np.array([5, 11, 2], np.int32)
    img = kvsynth.host_bytes(oracle.packed_bytes(s, 1, 3, 3), 4, 99, mode=kvsynth.MODE_RAW)
    oracle.scatter(s, *dst, 1, 3, bt, 4, img)
    for side in range(2):
        for l in range(4):
            for b in range(16):
                same = np.array_equal(_slab(dst[side][l], s, b), _slab(before[side][l], s, b))
                assert same == (not (1 <= l < 3 and b in bt))


@pytest.mark.parametrize("t1,t2", [(4, 8), (4, 28), (8, 12), (16, 400)])
def test_chunk_size_independence(t1, t2):
    s = Shape(3, 40, 4, 2, 8, 2)
    rng = np.random.default_rng(4)
    src = _mirror(s, 41)
    ids = rng.permutation(s.num_blocks).astype(np.int32)
    bt_src, bt_dst = ids[:15], ids[15:30]
    out = []
    for t in (t1, t2):
        dst = _mirror(s, 42, role=kvsynth.ROLE_DST)
        oracle.scatter(s, *dst, 0, 3, bt_dst, t, oracle.gather(s, *src, 0, 3, bt_src, t))
        out.append(dst)
    for side in range(2):
        for l in range(3):
            assert np.array_equal(out[0][side][l], out[1][side][l])


@pytest.mark.parametrize("ct", [4, 12, 16])
def test_layer_range_decomposition(ct):
    s = Shape(5, 30, 4, 2, 8, 2)
    rng = np.random.default_rng(5)
    k, v = _mirror(s, 51)
    bt = _ids(rng, s.num_blocks, 10)
    l0, m, l1 = 1, 3, 5
    full = oracle.gather(s, k, v, l0, l1, bt, ct)
    a = oracle.gather(s, k, v, l0, m, bt, ct)
    b = oracle.gather(s, k, v, m, l1, bt, ct)
    bpc = ct // s.block_size
    pa = pb = pf = 0
    for c in range(0, len(bt), bpc):
        nc = min(bpc, len(bt) - c)
        sa, sb = nc * (m - l0) * 2 * s.slab_bytes, nc * (l1 - m) * 2 * s.slab_bytes
        assert np.array_equal(full[pf:pf + sa], a[pa:pa + sa])
        assert np.array_equal(full[pf + sa:pf + sa + sb], b[pb:pb + sb])
        pa, pb, pf = pa + sa, pb + sb, pf + sa + sb
    assert pf == full.size


# ---- errors and degenerate cases ---------------------------------------------

def test_bad_block_id_rejected_and_nothing_written():
    s = Shape(2, 8, 2, 1, 8, 2)
    k, v = oracle.new_mirror(s)
    img = np.ones(oracle.packed_bytes(s, 0, 2, 3), np.uint8)
    for bad in ([1, 8, 2], [1, -1, 2]):
        with pytest.raises(IndexError):
            oracle.scatter(s, k, v, 0, 2, bad, 2, img)
        assert not any(a.any() for a in k + v)


def test_chunk_tokens_must_group_whole_blocks():
    s = Shape(2, 8, 4, 1, 8, 2)
    k, v = oracle.new_mirror(s)
    for ct in (0, 2, 6, -4):
        with pytest.raises(ValueError):
            oracle.gather(s, k, v, 0, 2, [1, 2], ct)


def test_empty_prefix_and_empty_layer_range_are_noops():
    s = Shape(2, 8, 4, 1, 8, 2)
    k, v = _mirror(s, 61)
    assert oracle.gather(s, k, v, 0, 2, [], 4).size == 0
    assert oracle.gather(s, k, v, 1, 1, [3, 4], 4).size == 0
    before = _copy((k, v))
    oracle.scatter(s, k, v, 0, 0, [3, 4], 4, np.zeros(0, np.uint8))
    assert all(np.array_equal(a, b) for a, b in zip(k + v, before[0] + before[1]))


# ---- brute force: O1 == O2 on a grid of tiny shapes -------------------------

def _grid():
    for L, H, D, BS, e in itertools.product((1, 3), (1, 2), (4, 8), (1, 2, 4), (2, 4)):
        if D * e % 16 and BS * H * D * e % 16:
            pass
        yield Shape(L, 12, BS, H, D, e)


@pytest.mark.parametrize("s", list(_grid()), ids=lambda s: f"L{s.num_layers}H{s.kv_heads}"
                         f"D{s.head_dim}BS{s.block_size}e{s.elem_bytes}")
def test_elementwise_equals_slab_exhaustive(s):
    rng = np.random.default_rng(s.num_layers * 7 + s.block_size)
    src = _mirror(s, 71)
    ev = lambda m: [oracle.element_view(a, s) for a in m]  # noqa: E731
    for n in range(0, 6):
        bt = _ids(rng, s.num_blocks, n)
        for ct in range(s.block_size, (n + 1) * s.block_size + 1, s.block_size):
            for l0 in range(s.num_layers + 1):
                for l1 in range(l0, s.num_layers + 1):
                    o2 = oracle.gather(s, *src, l0, l1, bt, ct)
                    o1 = oracle.gather_elementwise(ev(src[0]), ev(src[1]), l0, l1, bt, ct)
                    assert np.array_equal(o2.view(o1.dtype), o1), (n, ct, l0, l1)
                    if n and l1 > l0:
                        d2 = _mirror(s, 72, role=kvsynth.ROLE_DST)
                        d1 = _copy(d2)
                        oracle.scatter(s, *d2, l0, l1, bt, ct, o2)
                        oracle.scatter_elementwise(ev(d1[0]), ev(d1[1]), l0, l1, bt, ct, o1)
                        for a, b in zip(d2[0] + d2[1], d1[0] + d1[1]):
                            assert np.array_equal(a, b)


def test_elementwise_equals_slab_tiny_config():
    """The tiny workload shape itself: 2 layers, 64 blocks of 16 tokens, 2 KV
    heads, head dim 64, 16-block prefix in one 256-token chunk."""
    s = Shape(2, 64, 16, 2, 64, 2)
    rng = np.random.default_rng(1)
    src = _mirror(s, 1, mode=kvsynth.MODE_NORMAL_BF16)
    ids = rng.permutation(64).astype(np.int32)
    ev = lambda m: [oracle.element_view(a, s) for a in m]  # noqa: E731
    o2 = oracle.gather(s, *src, 0, 2, ids[:16], 256)
    o1 = oracle.gather_elementwise(ev(src[0]), ev(src[1]), 0, 2, ids[:16], 256)
    assert np.array_equal(o2.view(np.uint16), o1)


# ---- cache layouts other than the default ------------------------------------

LAYOUTS = [oracle.LAYOUT_HND, oracle.LAYOUT_PAGED_ATTN]


def _as_default_layout(shape, m):
    """Copy a mirror of any layout into a default-layout mirror via numpy views."""
    s0 = oracle.Shape(shape.num_layers, shape.num_blocks, shape.block_size, shape.kv_heads,
                      shape.head_dim, shape.elem_bytes)
    k0, v0 = oracle.new_mirror(s0)
    for l in range(shape.num_layers):
        oracle.element_view(k0[l], s0)[...] = oracle.canonical_view(m[0][l], shape, 0)
        oracle.element_view(v0[l], s0)[...] = oracle.canonical_view(m[1][l], shape, 1)
    return s0, (k0, v0)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("e", [2, 4])
def test_layout_gather_equals_default_after_numpy_transpose(layout, e):
    s = Shape(3, 20, 4, 2, 16, e, layout)
    m = _mirror(s, 81)
    s0, m0 = _as_default_layout(s, m)
    bt = _ids(np.random.default_rng(8), s.num_blocks, 9)
    for ct in (4, 8, 16):
        assert np.array_equal(oracle.gather(s, *m, 0, 3, bt, ct), oracle.gather(s0, *m0, 0, 3, bt, ct))


@pytest.mark.parametrize("layout", LAYOUTS)
def test_layout_elementwise_equals_slab(layout):
    s = Shape(2, 12, 4, 2, 16, 2, layout)
    m = _mirror(s, 82)
    bt = _ids(np.random.default_rng(9), s.num_blocks, 5)
    o1 = oracle.gather_elementwise([oracle.canonical_view(a, s, 0) for a in m[0]],
                                   [oracle.canonical_view(a, s, 1) for a in m[1]], 0, 2, bt, 8)
    assert np.array_equal(oracle.gather(s, *m, 0, 2, bt, 8).view(np.uint16), o1)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_layout_round_trip_and_untouched(layout):
    s = Shape(2, 30, 4, 2, 16, 2, layout)
    src = _mirror(s, 83)
    dst = _mirror(s, 84, role=kvsynth.ROLE_DST)
    before = _copy(dst)
    ids = np.random.default_rng(10).permutation(s.num_blocks).astype(np.int32)
    img = oracle.gather(s, *src, 0, 2, ids[:11], 8)
    oracle.scatter(s, *dst, 0, 2, ids[11:22], 8, img)
    assert np.array_equal(oracle.gather(s, *dst, 0, 2, ids[11:22], 8), img)
    for side in range(2):
        for l in range(2):
            for b in np.setdiff1d(np.arange(s.num_blocks), ids[11:22]):
                assert np.array_equal(_slab(dst[side][l], s, b), _slab(before[side][l], s, b))


def test_layout_rejects_head_dim_not_a_whole_number_of_16_byte_groups():
    s = Shape(1, 4, 4, 1, 12, 2, oracle.LAYOUT_PAGED_ATTN)  # x = 8 does not divide 12
    k, v = oracle.new_mirror(s)
    with pytest.raises(ValueError):
        oracle.gather(s, k, v, 0, 1, [0], 4)
