"""libkvx.so called from C alone (tests/c_abi/kvx_c_caller.c, built by
__graft_entry__.build()): a gather, a scatter into other blocks and a staged
restore through a ring, on a stream of the program's own, then the error
paths. Its outputs are compared with the oracle byte for byte: the gathered
image, and the whole cache after the scatter and the restore (every block:
the scattered and restored slabs, and every other block unchanged)."""
import os
import re
import subprocess

import numpy as np
import pytest

import kvsynth
import oracle

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "tests", "c_abi", "kvx_c_caller")
L, NB, BS, H, D, E = 3, 96, 16, 2, 64, 2  # the program's cache shape


@pytest.mark.parametrize("n,ct", [(24, 64), (17, 48), (5, 256)])
def test_c_caller_equals_oracle(tmp_path, n, ct):
    assert os.path.exists(BIN), "tests/c_abi/kvx_c_caller is not built (run __graft_entry__.build())"
    s = oracle.Shape(L, NB, BS, H, D, E)
    seed, mode, base = 91 + n, kvsynth.MODE_RAW, 0x5C000
    ids = np.random.default_rng(seed).permutation(NB).astype(np.int32)
    bt_src, bt_dst, bt_rst = ids[:n], ids[n:2 * n], ids[2 * n:3 * n]
    for name, bt in (("bt_src.bin", bt_src), ("bt_dst.bin", bt_dst), ("bt_rst.bin", bt_rst)):
        bt.tofile(tmp_path / name)
    nbytes = oracle.packed_bytes(s, 0, L, n)
    image = kvsynth.host_bytes(nbytes, seed, kvsynth.image_stream(3), mode=mode)
    image.tofile(tmp_path / "image.bin")
    print(f"c caller: n={n} chunk_tokens={ct} seed={seed}", flush=True)
    r = subprocess.run([BIN, str(tmp_path), str(seed), str(mode), str(base), str(n), str(ct)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, f"kvx_c_caller failed:\n{r.stdout}\n{r.stderr}"
    assert "c caller: ok" in r.stdout
    m = re.search(r"packed_bytes=(\d+) chunk_stride=(\d+)", r.stdout)
    assert int(m.group(1)) == nbytes
    assert int(m.group(2)) == L * 2 * ct * H * D * E  # a full chunk (Sec. 2.1 size model)

    k, v = oracle.new_mirror(s)
    for l in range(L):
        kvsynth.fill_host(k[l].reshape(-1).view(np.uint8), seed, base + 2 * l, mode=mode)
        kvsynth.fill_host(v[l].reshape(-1).view(np.uint8), seed, base + 2 * l + 1, mode=mode)
    expect = oracle.gather(s, k, v, 0, L, bt_src, ct)
    got = np.fromfile(tmp_path / "gathered.bin", dtype=np.uint8)
    assert np.array_equal(got, expect), "gathered image differs from the oracle"
    oracle.scatter(s, k, v, 0, L, bt_dst, ct, expect)
    oracle.restore(s, k, v, 0, L, bt_rst, ct, image)
    after = np.fromfile(tmp_path / "cache_after.bin", dtype=np.uint8)
    want = np.concatenate([a.reshape(-1).view(np.uint8) for a in k + v])
    assert after.size == want.size
    bad = np.flatnonzero(after != want)
    assert bad.size == 0, f"cache differs from the oracle at {bad.size} bytes, first {bad[:4]}"
