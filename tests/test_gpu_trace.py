"""The ring's transfer timeline (kvx_ring_set_trace / kvx_ring_trace_get), the
analogue of the profiler trace the paper shows for its connector (Sec. 4.1):
on a traced restore and offload, over both host-link paths (the DMA engines
driven directly, and the HIP runtime), every piece has its fill or drain
intervals (one per thread, bytes summing to the piece), one host-link copy and
one launch; each interval starts after what it depends on has ended (fills ->
host-to-device copy -> scatter; gather -> device-to-host copy -> drains; a
slot's next fill after its previous copy), and the results stay bit-exact
against the oracle."""
import collections

import numpy as np
import pytest

import kvsynth
import oracle
from kvtest_util import Filled, device_cache, host_mirror, seeded_ids, to_host

torch = pytest.importorskip("torch")
import paper_2609_11744_amd as kvx  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
# Device intervals sit on the host clock through a reference event (launches,
# runtime copies) or the HSA system clock (DMA copies): allow this much skew.
SKEW_NS = 200_000


def _bt(ids):
    return torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).to(DEV)


def _by(events):
    out = collections.defaultdict(lambda: collections.defaultdict(list))
    for e in events:
        out[e["kind"]][e["piece"]].append(e)
    return out


def _common(events, n_pieces):
    assert events == sorted(events, key=lambda e: e["t0_ns"])
    for e in events:
        assert e["t0_ns"] <= e["t1_ns"], e
    kinds = {e["kind"] for e in events}
    assert kinds <= set(kvx.TRACE_KINDS.values()), kinds
    assert max(e["piece"] for e in events) == n_pieces - 1


@pytest.mark.parametrize("hip_copies", [False, True], ids=["dma", "hip"])
def test_restore_timeline(hip_copies):
    s = oracle.Shape(4, 400, 16, 2, 64, 2)
    n, ct, slots, slot_bytes, threads = 150, 32, 3, 128 << 10, 3
    seed = 131
    (bt,) = seeded_ids(seed, s.num_blocks, n)
    cache = device_cache(s, Filled(seed, kvsynth.ROLE_DST), DEV)
    mirror = host_mirror(s, Filled(seed, kvsynth.ROLE_DST), range(s.num_blocks))
    image = kvsynth.host_bytes(oracle.packed_bytes(s, 0, 4, n), seed, kvsynth.image_stream(3),
                               mode=kvsynth.MODE_RAW)
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    try:
        ring.set_test_hooks(hip_copies=hip_copies)
        ring.bind(cache, 0, 4, n, ct, image, fill_threads=threads)
        ring.set_trace(True)
        kvx.kvx_restore_from_staging(ring, _bt(bt))
        torch.cuda.synchronize()
        kvx.kvx_check()
        P = ring.stats()["pieces"]
        ev = ring.trace()
        assert ring.trace() == ev  # reading it twice gives the same record
        ring.set_trace(False)
        kvx.kvx_restore_from_staging(ring, _bt(bt))
        torch.cuda.synchronize()
        assert ring.trace() == []  # an untraced transfer replaces the record
    finally:
        ring.close()
    oracle.restore(s, *mirror, 0, 4, bt, ct, image)
    for l in range(4):
        assert np.array_equal(to_host(cache.k[l]), mirror[0][l]), f"K layer {l}"
        assert np.array_equal(to_host(cache.v[l]), mirror[1][l]), f"V layer {l}"

    assert P > 3 * slots
    _common(ev, P)
    by = _by(ev)
    assert set(by) <= {"fill", "wait", "h2d", "scatter"}
    total = 0
    for i in range(P):
        fills, (copy,), (launch,) = by["fill"][i], by["h2d"][i], by["scatter"][i]
        assert sorted(f["lane"] for f in fills) == list(range(threads))
        assert sum(f["bytes"] for f in fills) == copy["bytes"] == launch["bytes"] > 0
        assert {f["slot"] for f in fills} == {copy["slot"]} == {launch["slot"]} == {i % slots}
        assert copy["t0_ns"] >= max(f["t1_ns"] for f in fills) - SKEW_NS
        assert launch["t0_ns"] >= copy["t1_ns"] - SKEW_NS
        if i >= slots:  # the slot is refilled once its previous copy has finished
            prev = by["h2d"][i - slots][0]
            assert min(f["t0_ns"] for f in fills) >= prev["t1_ns"] - SKEW_NS
        total += copy["bytes"]
    assert total == oracle.packed_bytes(s, 0, 4, n)
    print(f"\n{P} pieces, {len(ev)} intervals, span "
          f"{(ev[-1]['t1_ns'] - ev[0]['t0_ns']) / 1e6:.2f} ms", flush=True)
    chrome = kvx.trace_chrome(ev)
    assert sum(1 for e in chrome["traceEvents"] if e["ph"] == "X") == len(ev)


@pytest.mark.parametrize("hip_copies", [False, True], ids=["dma", "hip"])
def test_offload_timeline(hip_copies):
    L, ct, slots, slot_bytes, threads = 4, 32, 2, 96 << 10, 2
    s = oracle.Shape(L, 300, 16, 2, 64, 2)
    seed = 133
    (bt,) = seeded_ids(seed, s.num_blocks, 60)
    fill = Filled(seed, kvsynth.ROLE_NEW, kvsynth.MODE_RAW)
    cache = device_cache(s, fill, DEV)
    mirror = host_mirror(s, fill, bt)
    per_block = oracle.packed_bytes(s, 0, L, 1)
    sizes = [(a, min(2, 60 - a)) for a in range(0, 60, 2)]
    sinks = [np.full(nb * per_block, 0xEE, np.uint8) for _, nb in sizes]
    ring = kvx.StagingRing(DEV, slots, slot_bytes)
    try:
        ring.set_test_hooks(hip_copies=hip_copies)
        ring.bind_offload(cache, 0, L, ct, [(b, bt0, nb) for b, (bt0, nb) in zip(sinks, sizes)],
                          drain_threads=threads)
        ring.set_trace(True)
        kvx.kvx_offload_to_staging(ring, _bt(bt))
        torch.cuda.synchronize()
        kvx.kvx_check()
        P = ring.stats()["pieces"]
        ev = ring.trace()
    finally:
        ring.close()
    for b, (bt0, nb) in zip(sinks, sizes):
        assert np.array_equal(b, oracle.gather(s, *mirror, 0, L, bt[bt0:bt0 + nb], ct))
    _common(ev, P)
    by = _by(ev)
    assert set(by) <= {"drain", "wait", "d2h", "gather"}
    for i in range(P):
        (launch,), (copy,), drains = by["gather"][i], by["d2h"][i], by["drain"][i]
        assert sorted(d["lane"] for d in drains) == list(range(threads))
        assert sum(d["bytes"] for d in drains) == copy["bytes"] == launch["bytes"] > 0
        assert copy["t0_ns"] >= launch["t1_ns"] - SKEW_NS
        assert min(d["t0_ns"] for d in drains) >= copy["t1_ns"] - SKEW_NS
