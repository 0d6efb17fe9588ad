"""Storage tier on the host (Secs. 6.3, 6.4): hash-addressed chunk paths, the
io_uring engine's reads and writes (and its blocking fallback), publication
by hard link (first writer wins, no temporary left behind, readers see whole
files or none), and its error paths. The GPU ring's file-backed restore and
offload are in test_gpu_storage_tier.py."""
import os
import threading

import numpy as np
import pytest

import paper_2609_11744_amd as kvx


@pytest.fixture(params=["uring", "blocking"])
def engine(request, monkeypatch):
    if request.param == "blocking":
        monkeypatch.setenv("KVX_IO_NO_URING", "1")
    else:
        monkeypatch.delenv("KVX_IO_NO_URING", raising=False)
    return request.param


def _leftovers(root):
    return [os.path.join(d, f) for d, _, fs in os.walk(root) for f in fs if ".tmp." in f]


def test_chunk_path_layout():
    p = kvx.kvx_chunk_path("/data/kv", "llama-8b", 0x0123456789ABCDEF)
    assert p == "/data/kv/llama-8b/01/23/0123456789abcdef.kvc"
    assert kvx.kvx_chunk_path("r", "t", 0) == "r/t/00/00/0000000000000000.kvc"
    assert kvx.kvx_chunk_path("r", "t", -1).endswith("/ff/ff/ffffffffffffffff.kvc")
    for root, tag in (("", "t"), ("r", ""), ("r", "a/b")):
        with pytest.raises(kvx.KvxError):
            kvx.kvx_chunk_path(root, tag, 1)


@pytest.mark.parametrize("depth", [1, 4, 32])
def test_write_then_read_round_trip(tmp_path, engine, depth):
    rng = np.random.default_rng(depth)
    files = {}
    ops = []
    for i, size in enumerate([4096, 3 * 4096, 1 << 20, 12345, 5000]):  # aligned and not
        data = rng.integers(0, 256, size, dtype=np.uint8)
        path = kvx.kvx_chunk_path(str(tmp_path), "m", 0x1000 * (i + 1))
        files[path] = data
        # several ops per file, out of order, tiling it exactly
        cuts = sorted(set([0, size] + [int(c) for c in rng.integers(1, size, 3)]))
        parts = [(a, b) for a, b in zip(cuts, cuts[1:])]
        rng.shuffle(parts)
        ops += [(path, data[a:b], a) for a, b in parts]
    kvx.kvx_write_files(ops, io_depth=depth)
    assert not _leftovers(tmp_path)
    for path, data in files.items():
        assert open(path, "rb").read() == data.tobytes()
    got = {p: np.zeros(d.size, np.uint8) for p, d in files.items()}
    reads = []
    for p, d in files.items():  # read back in two halves each
        h = d.size // 2
        reads += [(p, got[p][:h], 0), (p, got[p][h:], h)]
    kvx.kvx_read_files(reads, io_depth=depth)
    for p, d in files.items():
        assert np.array_equal(got[p], d)


def test_first_writer_wins(tmp_path, engine):
    path = str(tmp_path / "a" / "b" / "chunk.kvc")
    first = np.full(8192, 1, np.uint8)
    kvx.kvx_write_files([(path, first, 0)])
    kvx.kvx_write_files([(path, np.full(8192, 2, np.uint8), 0)])  # succeeds, keeps the first
    assert open(path, "rb").read() == first.tobytes()
    assert not _leftovers(tmp_path)


def test_concurrent_writers_publish_one_whole_file(tmp_path, engine):
    path = str(tmp_path / "c.kvc")
    size = 1 << 20
    datas = [np.full(size, v, np.uint8) for v in (3, 4, 5, 6)]
    errs = []

    def write(d):
        try:
            kvx.kvx_write_files([(path, d[:size // 2], 0), (path, d[size // 2:], size // 2)],
                                io_depth=2)
        except Exception as e:  # noqa: BLE001
            errs.append(e)

    ts = [threading.Thread(target=write, args=(d,)) for d in datas]
    [t.start() for t in ts]
    [t.join() for t in ts]
    assert not errs
    got = np.frombuffer(open(path, "rb").read(), np.uint8)
    assert got.size == size and len(set(got.tolist())) == 1 and int(got[0]) in (3, 4, 5, 6)
    assert not _leftovers(tmp_path)


def test_errors(tmp_path, engine):
    buf = np.zeros(4096, np.uint8)
    with pytest.raises(kvx.KvxError) as ei:  # missing file
        kvx.kvx_read_files([(str(tmp_path / "none.kvc"), buf, 0)])
    assert ei.value.status == kvx.KVX_EIO
    short = str(tmp_path / "short.kvc")
    kvx.kvx_write_files([(short, np.ones(1000, np.uint8), 0)])
    with pytest.raises(kvx.KvxError) as ei:  # read past the end of the file
        kvx.kvx_read_files([(short, buf, 0)])
    assert ei.value.status == kvx.KVX_EIO
    gap = str(tmp_path / "gap.kvc")
    with pytest.raises(kvx.KvxError) as ei:  # writes that do not tile the file
        kvx.kvx_write_files([(gap, np.ones(100, np.uint8), 0), (gap, np.ones(100, np.uint8), 200)])
    assert ei.value.status == kvx.KVX_EINVAL
    assert not os.path.exists(gap) and not _leftovers(tmp_path)
    with pytest.raises(kvx.KvxError):
        kvx.kvx_read_files([(short, buf, 0)], io_depth=0)
    kvx.kvx_read_files([])  # nothing to do
