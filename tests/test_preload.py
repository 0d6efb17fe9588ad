"""The storage-tier preloader (Sec. 6.5) on the host: chunk files read ahead
into a bounded pool of slots, demand fetches that claim staged images or read
what is missing first, the reserve that speculative reads leave free, one read
per file however often it is hinted or fetched, least-recently-used eviction
for demand, and the error paths. Pools here are plain host memory (no GPU);
every case runs on io_uring and on the synchronous fallback
(KVX_IO_NO_URING=1)."""
import threading
import time

import numpy as np
import pytest

import paper_2609_11744_amd as kvx

SLOT = 48 << 20


@pytest.fixture(params=["uring", "sync"])
def engine(request, monkeypatch):
    if request.param == "sync":
        monkeypatch.setenv("KVX_IO_NO_URING", "1")
    else:
        monkeypatch.delenv("KVX_IO_NO_URING", raising=False)
    return request.param


def _files(tmp_path, sizes, seed=0):
    rng = np.random.default_rng(seed)
    out = []
    for i, n in enumerate(sizes):
        data = rng.integers(0, 256, n, dtype=np.uint8)
        p = tmp_path / f"c{i:03d}.kvc"
        data.tofile(p)
        out.append((str(p), data))
    return out


def _pre(**kw):
    args = dict(n_slots=4, slot_bytes=SLOT, io_depth=4, reserve=0, pinned=False)
    args.update(kw)
    return kvx.Preloader(**args)


def test_hint_then_fetch_returns_staged_images(tmp_path, engine):
    files = _files(tmp_path, [40 << 20, 4096, 12345])  # 2 pieces, one page, a ragged size
    p = _pre()
    try:
        p.hint([f for f, _ in files])
        p.wait_idle()
        st = p.stats()
        assert st["spec_reads"] == 3 and st["staged"] == 3
        imgs = p.fetch([f for f, _ in files])
        for img, (_, data) in zip(imgs, files):
            assert np.array_equal(img, data)
        st = p.stats()
        assert st["hits_ready"] == 3 and st["demand_reads"] == 0 and st["held"] == 3
        assert st["bytes_read"] == sum(d.size for _, d in files)
        p.release([f for f, _ in files])
        assert p.stats()["held"] == 0
    finally:
        p.close()


def test_fetch_without_hint_reads_on_demand(tmp_path, engine):
    files = _files(tmp_path, [SLOT, 3 << 20, 100], seed=1)  # a file of exactly one slot
    p = _pre(io_depth=2)
    try:
        imgs = p.fetch([f for f, _ in files])
        for img, (_, data) in zip(imgs, files):
            assert np.array_equal(img, data)
        st = p.stats()
        assert st["demand_reads"] == 3 and st["spec_reads"] == 0 and st["hits_ready"] == 0
        p.release([f for f, _ in files])
    finally:
        p.close()


def test_each_file_is_read_once(tmp_path, engine):
    files = _files(tmp_path, [6 << 20, 2 << 20], seed=2)
    paths = [f for f, _ in files]
    p = _pre()
    try:
        p.hint(paths + paths)           # the second hint of each is a duplicate
        imgs = p.fetch(paths + [paths[0]])  # joins or claims; a path twice in one fetch
        assert np.array_equal(imgs[0], files[0][1]) and np.array_equal(imgs[2], files[0][1])
        p.hint(paths)                   # already staged
        p.wait_idle()
        st = p.stats()
        assert st["spec_deduped"] == 4
        assert st["bytes_read"] == sum(d.size for _, d in files)
        assert st["spec_reads"] + st["demand_reads"] == 2
        assert st["held"] == 2
        p.release(paths)
        assert p.stats()["held"] == 0
    finally:
        p.close()


def test_reserve_limits_speculation_but_not_demand(tmp_path, engine):
    files = _files(tmp_path, [1 << 20] * 3, seed=3)
    a, b, c = (f for f, _ in files)
    p = _pre(n_slots=3, reserve=2)  # one slot for speculation
    try:
        p.hint([a, b, c])
        p.wait_idle()
        st = p.stats()
        assert st["spec_reads"] == 1 and st["staged"] == 1  # a only: b, c wait for the reserve
        (img,) = p.fetch([c])           # a queued hint becomes demand and runs past the reserve
        assert np.array_equal(img, files[2][1])
        p.wait_idle()
        st = p.stats()
        assert st["demand_reads"] == 1 and st["spec_reads"] == 1 and st["staged"] == 2
        p.release([c])
    finally:
        p.close()


def test_demand_evicts_least_recently_used_staged_file(tmp_path, engine):
    files = _files(tmp_path, [1 << 20] * 3, seed=4)
    a, b, c = (f for f, _ in files)
    p = _pre(n_slots=2)
    try:
        p.hint([a])
        p.wait_idle()
        p.hint([b])
        p.wait_idle()
        (img_c,) = p.fetch([c])         # pool full of unheld files: a (older) goes
        assert np.array_equal(img_c, files[2][1])
        st = p.stats()
        assert st["evictions"] == 1 and st["staged"] == 2
        (img_a,) = p.fetch([a])         # a is read again, evicting b (c is held)
        assert np.array_equal(img_a, files[0][1]) and np.array_equal(img_c, files[2][1])
        assert p.stats()["evictions"] == 2
        p.release([a, c])
    finally:
        p.close()


def test_speculation_reuses_cached_slots_never_unclaimed_preloads(tmp_path, engine):
    files = _files(tmp_path, [1 << 20] * 5, seed=10)
    a, b, c, d, e = (f for f, _ in files)
    p = _pre(n_slots=2)
    try:
        for f in (a, b):                # fetched and released: cached images fill the pool
            p.fetch([f])
            p.release([f])
        p.hint([c])                     # takes the least recently used cached slot (a)
        p.wait_idle()
        st = p.stats()
        assert st["spec_reads"] == 1 and st["evictions"] == 1 and st["staged"] == 2
        p.hint([d])                     # takes b's
        p.wait_idle()
        assert p.stats()["spec_reads"] == 2
        p.hint([e])                     # only unclaimed preloads left: e waits
        p.wait_idle()
        st = p.stats()
        assert st["spec_reads"] == 2 and st["staged"] == 2 and st["evictions"] == 2
        imgs = p.fetch([c, d])
        assert np.array_equal(imgs[0], files[2][1]) and np.array_equal(imgs[1], files[3][1])
        assert p.stats()["hits_ready"] == 2
        p.release([c, d])               # now cached: e may take one of them
        p.wait_idle()
        assert p.stats()["spec_reads"] == 3
    finally:
        p.close()


def test_fetch_beyond_the_pool_is_refused(tmp_path, engine):
    files = _files(tmp_path, [1 << 20] * 3, seed=5)
    a, b, c = (f for f, _ in files)
    p = _pre(n_slots=2)
    try:
        p.fetch([a, b])
        with pytest.raises(kvx.KvxError) as ei:
            p.fetch([c])
        assert ei.value.status == kvx.KVX_ENOMEM
        assert p.stats()["held"] == 2
        p.release([a])
        (img,) = p.fetch([c])
        assert np.array_equal(img, files[2][1])
        p.release([b, c])
    finally:
        p.close()


def test_missing_empty_and_oversized_files_fail_the_fetch(tmp_path, engine):
    (good, data), = _files(tmp_path, [1 << 20], seed=6)
    empty = tmp_path / "empty.kvc"
    empty.write_bytes(b"")
    big = tmp_path / "big.kvc"
    np.zeros(SLOT + 4096, np.uint8).tofile(big)
    p = _pre()
    try:
        for bad in (str(tmp_path / "missing.kvc"), str(empty), str(big)):
            with pytest.raises(kvx.KvxError) as ei:
                p.fetch([good, bad])
            assert ei.value.status == kvx.KVX_EIO
            assert p.stats()["held"] == 0   # nothing is held after a failed fetch
        (img,) = p.fetch([good])          # the good file stays usable
        assert np.array_equal(img, data)
        p.release([good])
        p.hint([str(tmp_path / "missing.kvc")])  # a failed hint is harmless
        p.wait_idle()
    finally:
        p.close()


def test_release_of_an_unheld_file_is_rejected(tmp_path, engine):
    (a, _), = _files(tmp_path, [4096], seed=7)
    p = _pre()
    try:
        with pytest.raises(kvx.KvxError) as ei:
            p.release([a])
        assert ei.value.status == kvx.KVX_EINVAL
        p.fetch([a])
        p.release([a])
        with pytest.raises(kvx.KvxError):
            p.release([a])
    finally:
        p.close()


def test_concurrent_fetches_share_reads(tmp_path, engine):
    files = _files(tmp_path, [3 << 20] * 6, seed=8)
    paths = [f for f, _ in files]
    p = _pre(n_slots=6, io_depth=3)
    errors = []

    def worker(sel):
        try:
            imgs = p.fetch([paths[i] for i in sel])
            for img, i in zip(imgs, sel):
                assert np.array_equal(img, files[i][1])
        except Exception as e:  # noqa: BLE001
            errors.append(e)

    try:
        p.hint(paths[3:])
        th = [threading.Thread(target=worker, args=(sel,)) for sel in ([0, 1, 2, 3], [2, 3, 4, 5])]
        for t in th:
            t.start()
        for t in th:
            t.join()
        assert not errors, errors
        st = p.stats()
        assert st["bytes_read"] == sum(d.size for _, d in files)  # one read per file
        assert st["held"] == 6
        p.release([paths[i] for i in (0, 1, 2, 3)])
        p.release([paths[i] for i in (2, 3, 4, 5)])
        assert p.stats()["held"] == 0
    finally:
        p.close()


def test_hint_queue_is_bounded(tmp_path, engine):
    files = _files(tmp_path, [4096] * 5, seed=9)
    p = _pre(n_slots=2, reserve=1)
    try:
        p.hint([f for f, _ in files])
        st = p.stats()
        assert st["hints"] + st["spec_dropped"] == 5 and st["spec_dropped"] >= 3 - 1
        p.wait_idle()
    finally:
        p.close()


def test_invalid_arguments(tmp_path):
    for kw in (dict(n_slots=0), dict(slot_bytes=1000), dict(io_depth=0), dict(reserve=4),
               dict(io_depth=300)):
        with pytest.raises(kvx.KvxError):
            _pre(**kw)
    p = _pre()
    try:
        with pytest.raises(kvx.KvxError):
            p.hint([""])
        with pytest.raises(kvx.KvxError):
            p.fetch([""])
    finally:
        p.close()


def test_demand_preempts_a_speculative_read_holding_the_last_slot(tmp_path, engine):
    # One slot, taken by a speculative read with pieces still to issue: the
    # demand file takes it over once the pieces in flight have landed, and the
    # speculative file is read again after the demand image is released.
    files = _files(tmp_path, [128 << 20, 1 << 20], seed=11)  # 4 pieces, 1 piece
    (a, data_a), (b, data_b) = files
    p = _pre(n_slots=1, slot_bytes=128 << 20, io_depth=1)
    got = {}
    try:
        p.set_test_hooks(delay_us=50000)  # each piece takes >= 50 ms
        p.hint([a])
        time.sleep(0.06)                  # a's read has started; pieces remain
        th = threading.Thread(target=lambda: got.setdefault("b", p.fetch([b])))
        th.start()
        th.join(timeout=30)
        assert "b" in got, "the demand fetch never got the slot"
        assert np.array_equal(got["b"][0], data_b)
        st = p.stats()
        assert st["spec_preempted"] == 1 and st["demand_reads"] == 1
        assert st["spec_reads"] == 0 and st["evictions"] == 0
        p.set_test_hooks(delay_us=0)
        p.release([b])                    # b is cached now: a takes its slot
        p.wait_idle()
        st = p.stats()
        assert st["spec_reads"] == 1 and st["evictions"] == 1 and st["staged"] == 1
        (img_a,) = p.fetch([a])
        assert np.array_equal(img_a, data_a) and p.stats()["hits_ready"] == 1
        p.release([a])
    finally:
        p.close()


def test_demand_waits_for_a_speculative_read_about_to_stage(tmp_path, engine):
    # Every piece of the speculative file is already issued: it is staged,
    # then evicted for the demand file, and nothing is preempted.
    files = _files(tmp_path, [2 << 20, 1 << 20], seed=12)  # one piece each
    (a, _), (b, data_b) = files
    p = _pre(n_slots=1, io_depth=2)
    try:
        p.set_test_hooks(delay_us=50000)
        p.hint([a])
        time.sleep(0.02)                  # a's only piece is in flight
        (img_b,) = p.fetch([b])
        assert np.array_equal(img_b, data_b)
        st = p.stats()
        assert st["spec_preempted"] == 0 and st["spec_reads"] == 1 and st["evictions"] == 1
        p.release([b])
    finally:
        p.close()
