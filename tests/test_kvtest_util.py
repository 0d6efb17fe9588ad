"""The GPU tests' full-tensor expectation (kvtest_util.oracle_layer_after_scatters)
against the oracle's scatter of whole chunks, on the CPU: restricting each
chunk image to one layer and scattering it there gives, layer by layer, the
same tensors as scattering the whole chunks into a full mirror."""
import numpy as np
import pytest

import kvsynth
import oracle
from kvtest_util import Filled, generator_tensor, oracle_layer_after_scatters


@pytest.mark.parametrize("l0,l1", [(0, 3), (1, 3)])
def test_layer_restricted_scatter_equals_whole_chunk_scatter(l0, l1):
    s = oracle.Shape(3, 50, 4, 2, 8, 2)
    fill = Filled(9, kvsynth.ROLE_NEW)
    rng = np.random.default_rng(l0)
    ids = rng.permutation(s.num_blocks).astype(np.int32)
    chunks, at = [], 0
    for nb in (4, 1, 3, 4, 2):  # chunks of 16 tokens = 4 blocks, some partial
        img = rng.integers(0, 256, size=(l1 - l0) * 2 * nb * s.slab_bytes, dtype=np.uint8)
        chunks.append((img, ids[at:at + nb], l0))
        at += nb
    k = [generator_tensor(s, fill, l, 0) for l in range(s.num_layers)]
    v = [generator_tensor(s, fill, l, 1) for l in range(s.num_layers)]
    for img, bt, _ in chunks:
        oracle.scatter(s, k, v, l0, l1, bt, 16, img)
    for l in range(s.num_layers):
        if l < l0 or l >= l1:
            continue
        ek, ev = oracle_layer_after_scatters(s, fill, l, chunks, 16)
        assert np.array_equal(ek, k[l]) and np.array_equal(ev, v[l]), l
