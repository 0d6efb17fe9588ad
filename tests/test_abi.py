"""Host-side checks of the C ABI (no GPU): the library loads and exports every
function kvx.h declares, host validation rejects bad arguments before any
HIP call, and the staging-piece planner tiles the image so that scattering
the pieces one by one equals scattering the whole image (checked with the
oracle)."""
import ctypes
import os
import re

import numpy as np
import pytest

import kvsynth
import oracle
import paper_2609_11744_amd as kvx
from paper_2609_11744_amd import _native

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "kvx.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvx_[A-Za-z0-9_]+)\s*\(", text)))


def test_header_declares_the_three_path_calls():
    names = _declared_functions()
    for n in ("kvx_gather_blocks", "kvx_scatter_blocks", "kvx_restore_from_staging"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(_native.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert set(_declared_functions()) == set(_native.SIGNATURES)


def test_bytes_per_token_matches_oracle_and_paper():
    assert kvx.kvx_bytes_per_token(28, 8, 128, 2) == 114688
    assert kvx.kvx_bytes_per_token(0, 8, 128, 2) == -1
    for args in [(32, 8, 128, 2), (80, 8, 128, 2), (2, 2, 64, 2)]:
        assert kvx.kvx_bytes_per_token(*args) == oracle.bytes_per_token(*args)


def _fake_cache(L=4, NB=100, BS=16, H=8, D=128, e=2, base=0x10000000):
    tensor = NB * BS * H * D * e
    kp = (ctypes.c_void_p * L)(*[base + (2 * l) * tensor for l in range(L)])
    vp = (ctypes.c_void_p * L)(*[base + (2 * l + 1) * tensor for l in range(L)])
    c = _native.KvxCache(kp, vp, L, NB, BS, H, D, e)
    c._keep = (kp, vp)
    return c, base, tensor


def _gather(c, l0, l1, bt, n, ct, dst):
    return _native.lib().kvx_gather_blocks(ctypes.byref(c), l0, l1, bt, n, ct, dst, None)


@pytest.mark.parametrize("args", [
    dict(l0=-1), dict(l1=5), dict(l0=3, l1=2), dict(n=-1), dict(ct=0), dict(ct=24), dict(ct=-16),
    dict(bt=None), dict(dst=None), dict(dst=0x7000_0000_0008),
])
def test_validation_rejects_before_any_hip_call(args):
    c, base, tensor = _fake_cache()
    a = dict(l0=0, l1=4, bt=0x5000_0000_0000, n=10, ct=32, dst=0x7000_0000_0000)
    a.update(args)
    st = _gather(c, a["l0"], a["l1"], a["bt"], a["n"], a["ct"], a["dst"])
    assert st == kvx.KVX_EINVAL


def test_validation_rejects_dst_overlapping_cache():
    c, base, tensor = _fake_cache()
    assert _gather(c, 0, 4, 0x5000_0000_0000, 10, 32, base + tensor + 4096) == kvx.KVX_EINVAL


def test_validation_rejects_misaligned_cache_and_bad_shapes():
    c, base, tensor = _fake_cache(base=0x10000008)
    assert _gather(c, 0, 4, 0x5000_0000_0000, 1, 16, 0x7000_0000_0000) == kvx.KVX_EINVAL
    c, _, _ = _fake_cache(e=3)
    assert _gather(c, 0, 4, 0x5000_0000_0000, 1, 16, 0x7000_0000_0000) == kvx.KVX_EINVAL
    c, _, _ = _fake_cache(H=1, D=3, BS=1, e=2)  # 6-byte slab, not a multiple of 16
    assert _gather(c, 0, 4, 0x5000_0000_0000, 1, 1, 0x7000_0000_0000) == kvx.KVX_EINVAL
    c, _, _ = _fake_cache(L=200)
    assert _gather(c, 0, 200, 0x5000_0000_0000, 1, 16, 0x7000_0000_0000) == kvx.KVX_EINVAL


def test_noops_return_ok_without_touching_the_device():
    c, _, _ = _fake_cache()
    assert _gather(c, 0, 4, None, 0, 32, None) == kvx.KVX_OK
    assert _gather(c, 2, 2, 0x5000_0000_0000, 10, 32, 0x7000_0000_0000) == kvx.KVX_OK


def test_packed_bytes_matches_oracle():
    for L, NB, BS, H, D, e in [(32, 20000, 16, 8, 128, 2), (2, 64, 16, 2, 64, 2),
                               (80, 1000, 16, 8, 128, 2), (3, 7, 4, 1, 8, 4)]:
        c = kvx.shape_only_cache(L, NB, BS, H, D, e)
        s = oracle.Shape(L, NB, BS, H, D, e)
        for l0, l1, n in [(0, L, 5), (1, L, 0), (0, 1, 13)]:
            assert kvx.kvx_packed_bytes(c, l0, l1, n) == oracle.packed_bytes(s, l0, l1, n)


# ---- staging piece planner ---------------------------------------------------

PLAN_CASES = [
    # (layers, heads, dim, block_size, n_blocks, chunk_tokens, slot_bytes)
    (32, 8, 128, 16, 5000, 256, 64 << 20),    # 80k prefix, 4 x 64 MiB ring
    (32, 8, 128, 16, 2048, 16, 64 << 20),
    (32, 8, 128, 16, 2048, 1024, 64 << 20),   # chunk larger than a slot: layer split
    (80, 8, 128, 16, 1000, 256, 64 << 20),    # 70B chunk 80 MiB -> 64 + 16 layers
    (3, 1, 8, 4, 17, 12, 4096),
    (5, 2, 8, 2, 9, 6, 640),
]


@pytest.mark.parametrize("case", PLAN_CASES)
def test_plan_tiles_image_exactly_and_fits_slots(case):
    L, H, D, BS, n, ct, slot = case
    c = kvx.shape_only_cache(L, 4 * n + 8, BS, H, D, 2)
    pieces = kvx.kvx_plan_pieces(c, 0, L, n, ct, slot)
    total = kvx.kvx_packed_bytes(c, 0, L, n)
    at = 0
    for p in pieces:
        assert p["src_offset"] == at and 0 < p["bytes"] <= slot
        slab = BS * H * D * 2
        assert p["bytes"] == p["n_blocks"] * (p["l_end"] - p["l_begin"]) * 2 * slab
        at += p["bytes"]
    assert at == total


def test_plan_80k_prefix_has_157_pieces():
    c = kvx.shape_only_cache(32, 20000, 16, 8, 128, 2)
    pieces = kvx.kvx_plan_pieces(c, 0, 32, 5000, 256, 64 << 20)
    assert len(pieces) == 157
    assert pieces[-1]["bytes"] == 16 << 20 and pieces[-1]["n_blocks"] == 8


def test_plan_70b_chunk_splits_64_plus_16_layers():
    c = kvx.shape_only_cache(80, 2000, 16, 8, 128, 2)
    pieces = kvx.kvx_plan_pieces(c, 0, 80, 32, 256, 64 << 20)
    assert [(p["l_begin"], p["l_end"]) for p in pieces] == [(0, 64), (64, 80)] * 2


def test_plan_rejects_slot_smaller_than_one_layer():
    c = kvx.shape_only_cache(4, 100, 16, 8, 128, 2)
    with pytest.raises(kvx.KvxError):
        # one layer (K and V) of a 16-block chunk is 2 * 16 * 32 KiB = 1 MiB
        kvx.kvx_plan_pieces(c, 0, 4, 16, 256, (1 << 20) - 4096)


def _ramp_caps(sizes, slot, ramp):
    """Each piece's size limit under a ramp, from the pieces' own sizes: in
    ramp order (from the first piece, or from the last one backwards), the
    first at most slot / 8 and each next at most twice the piece before it,
    until a limit reaches the slot, and the slot from there on."""
    if ramp == kvx.KVX_RAMP_NONE:
        return [slot] * len(sizes)
    order = list(range(len(sizes)))
    if ramp == kvx.KVX_RAMP_LAST:
        order.reverse()
    caps = [slot] * len(sizes)
    prev = None
    for k in order:
        c = slot >> 3 if prev is None else max(slot >> 3, 2 * prev)
        if c >= slot:
            break
        caps[k] = c
        prev = sizes[k]
    return caps


@pytest.mark.parametrize("ramp", [kvx.KVX_RAMP_FIRST, kvx.KVX_RAMP_LAST])
@pytest.mark.parametrize("case", PLAN_CASES)
def test_ramped_plan_tiles_image_within_limits(case, ramp):
    """The ring's ramped plans: the pieces tile the image exactly once, each
    within its limit (or one layer of a chunk where a layer exceeds it), each
    carries its chunks in image order (one host copy per piece of a
    contiguous image), and the end ramp mirrors the first-piece ramp."""
    L, H, D, BS, n, ct, slot = case
    c = kvx.shape_only_cache(L, 4 * n + 8, BS, H, D, 2)
    slab = BS * H * D * 2
    pieces = kvx.kvx_plan_pieces(c, 0, L, n, ct, slot, ramp)
    caps = _ramp_caps([p["bytes"] for p in pieces], slot, ramp)
    bpc = ct // BS
    covered = []
    for p, cap in zip(pieces, caps):
        layer = min(bpc, n) * 2 * slab  # one layer of a full chunk
        assert 0 < p["bytes"] <= max(cap, layer if p["l_end"] - p["l_begin"] == 1 else 0), p
        assert p["bytes"] == p["n_blocks"] * (p["l_end"] - p["l_begin"]) * 2 * slab
        assert p["n_spans"] == 1
        covered.append((p["src_offset"], p["bytes"]))
    at = 0
    for off, b in sorted(covered):
        assert off == at
        at += b
    assert at == kvx.kvx_packed_bytes(c, 0, L, n)
    if n % bpc == 0:  # all chunks alike: the end ramp is the first ramp reversed
        other = kvx.kvx_plan_pieces(c, 0, L, n, ct, slot, 3 - ramp)
        assert [p["bytes"] for p in pieces] == [p["bytes"] for p in reversed(other)]


def test_ramped_80k_restore_plan():
    """The restore's first-piece ramp at 80k: the first 32 MiB chunk is cut
    into 8, 16 and 8 MiB layer ranges; after the 8 MiB tail the next chunk
    goes as two 16 MiB halves (at most twice the piece before), the next
    whole (32 MiB), and from there two-chunk pieces of a full slot."""
    c = kvx.shape_only_cache(32, 20000, 16, 8, 128, 2)
    pieces = kvx.kvx_plan_pieces(c, 0, 32, 5000, 256, 64 << 20, kvx.KVX_RAMP_FIRST)
    assert len(pieces) == 161
    assert [p["bytes"] >> 20 for p in pieces[:8]] == [8, 16, 8, 16, 16, 32, 64, 64]
    assert [(p["l_begin"], p["l_end"]) for p in pieces[:5]] == \
        [(0, 8), (8, 24), (24, 32), (0, 16), (16, 32)]
    # the end ramp starts from the compact 16 MiB last chunk: 8 + 8 MiB
    # layer halves, the 32 MiB chunk before it in 16 MiB halves, the one
    # before that alone
    end = kvx.kvx_plan_pieces(c, 0, 32, 5000, 256, 64 << 20, kvx.KVX_RAMP_LAST)
    assert [p["bytes"] >> 20 for p in end[-6:]] == [64, 32, 16, 16, 8, 8]
    assert [(p["l_begin"], p["l_end"]) for p in end[-2:]] == [(16, 32), (0, 16)]
    with pytest.raises(kvx.KvxError):
        kvx.kvx_plan_pieces(c, 0, 32, 5000, 256, 64 << 20, 3)


@pytest.mark.parametrize("ramp", [kvx.KVX_RAMP_NONE, kvx.KVX_RAMP_FIRST, kvx.KVX_RAMP_LAST])
@pytest.mark.parametrize("case", PLAN_CASES[4:] + [(4, 2, 8, 4, 23, 16, 2048), (6, 1, 8, 2, 13, 8, 256)])
def test_scattering_pieces_equals_scattering_image(case, ramp):
    """Every piece is a plain scatter of its bytes; together they reproduce the
    oracle's scatter of the whole image (restore transparency, on the CPU)."""
    L, H, D, BS, n, ct, slot = case
    NB = 3 * n + 5
    s = oracle.Shape(L, NB, BS, H, D, 2)
    c = kvx.shape_only_cache(L, NB, BS, H, D, 2)
    bt = np.random.default_rng(n).permutation(NB)[:n].astype(np.int32)
    img = kvsynth.host_bytes(oracle.packed_bytes(s, 0, L, n), 5, 123, mode=kvsynth.MODE_RAW)
    whole = oracle.new_mirror(s)
    oracle.scatter(s, *whole, 0, L, bt, ct, img)
    by_piece = oracle.new_mirror(s)
    for p in kvx.kvx_plan_pieces(c, 0, L, n, ct, slot, ramp):
        part = img[p["src_offset"]:p["src_offset"] + p["bytes"]]
        oracle.scatter(s, *by_piece, p["l_begin"], p["l_end"],
                       bt[p["bt_first"]:p["bt_first"] + p["n_blocks"]], p["chunk_tokens"], part)
    for a, b in zip(whole[0] + whole[1], by_piece[0] + by_piece[1]):
        assert np.array_equal(a, b)


def test_layout_validation_on_the_host():
    def call(layout, H=8, D=128, e=2, BS=16):
        c, _, _ = _fake_cache(H=H, D=D, e=e, BS=BS)
        c.layout = layout
        return _gather(c, 0, 4, 0x5000_0000_0000, 1, BS, 0x7000_0000_0000)
    assert call(3) == kvx.KVX_EINVAL                          # unknown layout
    assert call(kvx.KVX_LAYOUT_HND, BS=32) == kvx.KVX_EINVAL  # 64 KiB slab > 48 KiB LDS image
    assert call(kvx.KVX_LAYOUT_PAGED_ATTN, H=1, D=4, e=2) == kvx.KVX_EINVAL  # 8-byte rows
    assert call(kvx.KVX_LAYOUT_HND, H=1, D=12, e=2) == kvx.KVX_EINVAL       # 24-byte rows


def test_probe_rejects_bad_arguments_on_the_host():
    """kvx_probe_stream validates before it enqueues anything (the fake device
    addresses below are never dereferenced)."""
    import paper_2609_11744_amd as kvx
    from paper_2609_11744_amd import _native

    lib = _native.lib()
    unit = 4 << 10
    assert lib.kvx_probe_stream(None, None, unit, 0, None) == kvx.KVX_EINVAL  # read: no src
    assert lib.kvx_probe_stream(None, None, unit, 1, None) == kvx.KVX_EINVAL  # write: no dst
    assert lib.kvx_probe_stream(4096, 8192, unit + 16, 2, None) == kvx.KVX_EINVAL  # size
    assert lib.kvx_probe_stream(4096, 8192, unit, 3, None) == kvx.KVX_EINVAL  # mode
    assert lib.kvx_probe_stream(4100, 8192, unit, 2, None) == kvx.KVX_EINVAL  # alignment
    assert lib.kvx_probe_stream(4096, 8192, -unit, 2, None) == kvx.KVX_EINVAL


def test_layer_range_limit_on_the_host():
    """A call covers at most KVX_MAX_LAYERS (128) layers."""
    import paper_2609_11744_amd as kvx

    c = kvx.shape_only_cache(130, 100, 16, 8, 128, 2)
    assert kvx.KVX_MAX_LAYERS == 128
    assert kvx.kvx_packed_bytes(c, 1, 129, 10) == 128 * 2 * 10 * 16 * 8 * 128 * 2
    assert kvx.kvx_packed_bytes(c, 0, 129, 10) == -1
    assert kvx.kvx_packed_bytes(c, 0, 131, 10) == -1


# ---- the walk a copy takes (kvx_copy_walk: the launcher's choice, host only) ----------

HND_, PA_ = kvx.KVX_LAYOUT_HND, kvx.KVX_LAYOUT_PAGED_ATTN
# (layers, heads, layout, n_blocks, chunk_tokens, to_packed) -> (parts, ordered, linear,
# pair_slices, fronts); block size 16, head dim 128, 2-byte words, 20,000-block pool
WALKS = [
    ((32, 8, 0, 5000, 256, True), (8, 0, 0, 4, 1)),     # 80k gather: slices 4 apart (2 MiB)
    ((32, 8, 0, 5000, 256, False), (8, 1, 0, 4, 2)),    # 80k scatter: ordered, two fronts
    ((32, 8, 0, 2048, 16, False), (8, 0, 0, 0, 1)),     # one-block chunks: image order
    ((32, 8, 0, 2048, 16, True), (8, 0, 0, 0, 1)),      # D = 64 > 32: plain walk
    ((32, 8, 0, 2048, 64, False), (8, 1, 0, 16, 2)),    # 32 KiB x 4 blocks: fronts 16 apart
    ((32, 8, 0, 2048, 64, True), (8, 0, 0, 16, 1)),
    ((32, 8, 0, 2048, 128, False), (8, 1, 0, 8, 2)),
    ((32, 8, 0, 2048, 1024, False), (8, 1, 0, 1, 2)),
    ((32, 8, 0, 1023, 256, False), (8, 0, 0, 0, 1)),    # below 1,024 blocks: image order
    ((32, 1, 0, 5000, 256, True), (1, 0, 0, 32, 1)),    # tp = 8 shard: gather 32 apart
    ((32, 1, 0, 5000, 256, False), (1, 0, 1, 0, 1)),    # 4 KiB slabs: linear image order
    ((32, 2, 0, 5000, 256, False), (2, 0, 1, 0, 1)),    # 8 KiB slabs: linear image order
    ((32, 2, 0, 5000, 256, True), (2, 0, 0, 16, 1)),
    ((32, 4, 0, 5000, 256, False), (4, 1, 0, 8, 2)),    # 16 KiB slabs: fronts 8 apart
    ((32, 1, HND_, 5000, 256, False), (1, 0, 1, 0, 1)), # one-head HND = the default layout
    ((32, 2, HND_, 5000, 256, False), (2, 1, 0, 0, 1)), # two heads: ordered, D = 16 > 4
    ((32, 1, PA_, 5000, 256, False), (1, 0, 1, 0, 1)),  # one-head paged attention: linear
    ((32, 2, PA_, 5000, 256, False), (2, 1, 0, 0, 1)),  # two heads keep destination order
    ((32, 8, PA_, 5000, 256, True), (8, 0, 0, 4, 1)),
    ((80, 8, 0, 3000, 256, False), (8, 1, 0, 4, 2)),    # 70B shape: 160 slices
    ((80, 8, 0, 4000, 256, False), (8, 1, 0, 0, 1)),    # over 2^22 work items: one front
    ((10, 8, 0, 1100, 256, False), (8, 1, 0, 0, 1)),    # 20 slices: one front
    ((10, 8, 0, 1100, 256, True), (8, 0, 0, 0, 1)),     # 20 slices: not a multiple of 8
]


@pytest.mark.parametrize("case,want", WALKS, ids=[f"w{i}" for i in range(len(WALKS))])
def test_copy_walk_rules(case, want):
    L, H, layout, n, ct, to_packed = case
    c = kvx.shape_only_cache(L, 20000, 16, H, 128, 2, layout)
    w = kvx.kvx_copy_walk(c, 0, L, n, ct, to_packed)
    assert (w["parts"], w["ordered"], w["linear"], w["pair_slices"], w["fronts"]) == want
    assert w["work_items"] == n * L * 2 * w["parts"]


def test_copy_walk_empty_and_invalid():
    c = kvx.shape_only_cache(4, 100, 16, 2, 64, 2)
    assert kvx.kvx_copy_walk(c, 0, 4, 0, 16, True) == \
        {"work_items": 0, "parts": 0, "ordered": 0, "linear": 0, "pair_slices": 0, "fronts": 0}
    with pytest.raises(kvx.KvxError) as ei:
        kvx.kvx_copy_walk(c, 0, 4, 10, 24, False)  # not a multiple of the block size
    assert ei.value.status == kvx.KVX_EINVAL
    with pytest.raises(kvx.KvxError):
        kvx.kvx_copy_walk(c, 0, 5, 10, 16, False)  # layer range beyond the cache
    lib = _native.lib()
    w = _native.KvxWalk()
    assert lib.kvx_copy_walk(ctypes.byref(c), 0, 4, 10, 16, 2, ctypes.byref(w)) == kvx.KVX_EINVAL
    assert lib.kvx_copy_walk(ctypes.byref(c), 0, 4, 10, 16, 1, None) == kvx.KVX_EINVAL
    assert lib.kvx_copy_walk(None, 0, 4, 10, 16, 1, ctypes.byref(w)) == kvx.KVX_EINVAL


def test_calls_beyond_the_workgroup_range_are_invalid():
    """A call's workgroups (slabs x parts per slab) are counted in 31 bits: one
    more is rejected on the host as an invalid argument, not launched."""
    c = kvx.shape_only_cache(128, 16, 16, 64, 64, 2)  # 128 KiB slabs: 32 parts each
    n_ok = (2**31 - 1) // (256 * 32)                    # 128 layers x K|V = 256 slabs per block
    assert kvx.kvx_copy_walk(c, 0, 128, n_ok, 16, True)["work_items"] == n_ok * 256 * 32
    for fn in (lambda n: kvx.kvx_copy_walk(c, 0, 128, n, 16, True),
               lambda n: kvx.kvx_copy_walk(c, 0, 128, n, 16, False)):
        with pytest.raises(kvx.KvxError) as ei:
            fn(n_ok + 1)
        assert ei.value.status == kvx.KVX_EINVAL
    assert kvx.kvx_packed_bytes(c, 0, 128, n_ok + 1) == -1
