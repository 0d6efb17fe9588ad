"""The seeded input generator: its table is N(0,1) quantiles to bf16, its
streams are position-addressed (a sub-range fill equals the slice of a whole
fill), and thread count does not change the bytes."""
import numpy as np
import pytest
from scipy.stats import norm

import kvsynth


def _bf16_to_f32(u16):
    return (u16.astype(np.uint32) << 16).view(np.float32)


def test_table_is_normal_quantiles_rounded_to_bf16():
    tab = kvsynth.normal_table()
    x = _bf16_to_f32(tab).astype(np.float64)
    q = norm.ppf((np.arange(65536) + 0.5) / 65536)
    # bf16 keeps 8 significant bits: relative rounding error <= 2^-8
    assert np.all(np.abs(x - q) <= np.abs(q) * 2.0**-8 + 1e-30)
    assert np.all(np.diff(x) >= 0)
    assert np.array_equal(tab[:32768] ^ 0x8000, tab[65535:32767:-1])


def test_normal_mode_moments():
    a = kvsynth.host_bytes(1 << 22, 7, 1234)
    x = _bf16_to_f32(a.view(np.uint16)).astype(np.float64)
    assert abs(x.mean()) < 0.01 and abs(x.std() - 1) < 0.01


@pytest.mark.parametrize("mode", [kvsynth.MODE_NORMAL_BF16, kvsynth.MODE_RAW])
def test_position_addressed_and_thread_invariant(mode):
    whole = kvsynth.host_bytes(1 << 23, 5, 42, mode=mode, threads=1)
    par = kvsynth.host_bytes(1 << 23, 5, 42, mode=mode, threads=8)
    assert np.array_equal(whole, par)
    for off, n in ((0, 8), (4096, 32768), (8 * 12345, 8 * 999), ((1 << 23) - 64, 64)):
        part = kvsynth.host_bytes(n, 5, 42, byte_offset=off, mode=mode)
        assert np.array_equal(part, whole[off:off + n])


def test_streams_and_seeds_differ():
    a = kvsynth.host_bytes(4096, 1, kvsynth.cache_stream(kvsynth.ROLE_SRC, 0, 0))
    b = kvsynth.host_bytes(4096, 1, kvsynth.cache_stream(kvsynth.ROLE_SRC, 0, 1))
    c = kvsynth.host_bytes(4096, 2, kvsynth.cache_stream(kvsynth.ROLE_SRC, 0, 0))
    assert not np.array_equal(a, b) and not np.array_equal(a, c)


def test_rejects_unaligned():
    with pytest.raises(ValueError):
        kvsynth.fill_host(np.zeros(12, np.uint8), 1, 1)
    with pytest.raises(ValueError):
        kvsynth.fill_host(np.zeros(16, np.uint8), 1, 1, byte_offset=4)


def test_fill_ranges_matches_whole_fill():
    whole = kvsynth.host_bytes(1 << 20, 9, 77, mode=kvsynth.MODE_RAW)
    buf = np.zeros(1 << 20, np.uint8)
    offs = [0, 4096 * 3, 4096 * 17, (1 << 20) - 4096]
    kvsynth.fill_ranges(buf, offs, 4096, 9, 77, mode=kvsynth.MODE_RAW, threads=3)
    for o in offs:
        assert np.array_equal(buf[o:o + 4096], whole[o:o + 4096])
    mask = np.ones(1 << 20, bool)
    for o in offs:
        mask[o:o + 4096] = False
    assert not buf[mask].any()
