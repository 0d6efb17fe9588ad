"""Step planner on the host: the prefix-hash chain and chunk dedupe of the
library, checked against the oracle's exact-key definitions and against the
paper's worked prefix-tree example (Sec. 2.1)."""
import json
import os

import numpy as np
import pytest

import kvsynth.prefix_tree as pt
import oracle.prefix as op
import paper_2609_11744_amd as kvx
from paper_2609_11744_amd import step

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "prefix_hash_example.json")


def _replay(ex, keys_of):
    cached, out = set(), []
    for req in ex["requests"]:
        keys = keys_of(req["tokens"], ex["block_size"])
        n = 0
        for k in keys:
            if k not in cached:
                break
            n += 1
        cached.update(keys)
        out.append((n, len(req["tokens"]) - n * ex["block_size"], len(cached)))
    return out


def test_oracle_reproduces_paper_example():
    ex = json.load(open(GOLDEN))
    got = _replay(ex, op.block_keys)
    want = [(r["reused_blocks"], r["computed_tokens"], r["cached_full_blocks_after"])
            for r in ex["requests"]]
    assert got == want
    # and the oracle's own lookup helper agrees
    cached = set(op.block_keys(ex["requests"][0]["tokens"], 2))
    assert op.matched_blocks(ex["requests"][1]["tokens"], 2, cached) == 2


def test_library_hash_chain_reproduces_paper_example():
    ex = json.load(open(GOLDEN))
    got = _replay(ex, lambda t, bs: [int(h) for h in kvx.kvx_block_hashes(np.array(t), bs)])
    want = [(r["reused_blocks"], r["computed_tokens"], r["cached_full_blocks_after"])
            for r in ex["requests"]]
    assert got == want


def test_partial_block_gets_no_hash():
    assert kvx.kvx_block_hashes(np.arange(7), 2).size == 3
    assert kvx.kvx_block_hashes(np.arange(1), 2).size == 0
    assert kvx.kvx_block_hashes(np.arange(0), 2).size == 0


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_hash_equality_is_prefix_equality(seed):
    """Across a batch of prompts with shared prefixes, two blocks hash equal
    exactly when their token prefixes are equal (no collisions, no misses)."""
    reqs = pt.make_requests(seed, n=12, lo=64, hi=1024, chunk_tokens=64)
    exact, hashed = [], []
    for r in reqs:
        exact += op.block_keys(r.tokens, 16)
        hashed += [int(h) for h in kvx.kvx_block_hashes(r.tokens, 16)]
    assert len(exact) == len(hashed)
    first_exact = op.dedupe(exact)
    first_hash = op.dedupe(hashed)
    assert first_exact == first_hash


@pytest.mark.parametrize("seed", [4, 5])
def test_library_dedupe_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    keys = rng.integers(0, 50, size=400).astype(np.uint64)
    assert list(kvx.kvx_dedupe_keys(keys)) == op.dedupe([int(k) for k in keys])
    assert kvx.kvx_dedupe_keys(np.zeros(0, np.uint64)).size == 0


@pytest.mark.parametrize("seed", [5, 6])
def test_step_plan_restores_each_missing_chunk_once(seed):
    reqs = pt.make_requests(seed, n=24, lo=256, hi=4096)
    plan = step.plan_step(reqs, block_size=16, chunk_tokens=256)
    # oracle: exact chunk keys, dedupe, residency
    exact_chunks = []
    for r in reqs:
        for (key, nb), res in zip(op.chunk_keys(r.tokens, 16, 256), r.resident):
            exact_chunks.append((key, nb, bool(res)))
    first = op.dedupe([c[0] for c in exact_chunks])
    missing_unique = [i for i, c in enumerate(exact_chunks) if first[i] == i and not c[2]]
    resident_unique = [i for i, c in enumerate(exact_chunks) if first[i] == i and c[2]]
    assert len(plan.restore) == len(missing_unique)
    assert sum(c.n_blocks for c in plan.restore) == sum(exact_chunks[i][1] for i in missing_unique)
    assert plan.resident_hits == len(resident_unique)
    # the restore list is keyed consistently: the same chunk (by exact key) is
    # restored once and every request chunk that needs it points at it
    exact_of_restore = [exact_chunks[i][0] for i in missing_unique]
    assert len(set(exact_of_restore)) == len(exact_of_restore)
    # each request's table references a restored chunk or a resident one
    assert len(plan.request_chunks) == sum(len(op.chunk_keys(r.tokens, 16, 256)) for r in reqs)
    # new blocks: one offload chunk list covering every request's new blocks
    assert sum(c.n_blocks for c in plan.offload) == sum(r.new_blocks for r in reqs)


def test_residency_is_consistent_across_sharing_requests():
    reqs = pt.make_requests(7, n=40, lo=256, hi=8192)
    seen = {}
    for r in reqs:
        for (key, nb), res in zip(op.chunk_keys(r.tokens, 16, 256), r.resident):
            assert seen.setdefault(key, bool(res)) == bool(res)
