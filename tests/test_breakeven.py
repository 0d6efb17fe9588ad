"""Break-even gate (Secs. 4.1, 5.2, 6.6): the oracle pinned by closed forms and
special cases, then the library (kvx_curve calls) against the oracle, and the
step planner's gate against the oracle's reading of it."""
import math
import random

import numpy as np
import pytest

import oracle.breakeven as ob
from paper_2609_11744_amd import breakeven as be

# ---- oracle pins ----------------------------------------------------------------


def lin(c, a):
    """A straight line through two knots (exactly linear everywhere)."""
    return [1000.0, 9000.0], [c + a * 1000.0, c + a * 9000.0]


def test_oracle_curve_interpolates_and_extrapolates():
    t, s = [1000.0, 2000.0, 8000.0], [0.5, 0.75, 3.0]
    assert ob.curve(t, s, 2000.0) == 0.75
    assert ob.curve(t, s, 1500.0) == 0.625                 # midpoint
    assert ob.curve(t, s, 5000.0) == 0.75 + 2.25 * 0.5      # second segment
    assert ob.curve(t, s, 0.0) == 0.5 - 0.25                # first segment continued
    assert ob.curve(t, s, 10000.0) == 3.0 + 2.25 / 6 * 2    # last segment continued
    lt, ls = lin(0.03, 2e-5)
    for x in (0.0, 512.0, 40000.0, 123456.0):
        assert math.isclose(ob.curve(lt, ls, x), 0.03 + 2e-5 * x, rel_tol=1e-12)


# cold f = c0 + a x, hit g = c1 + b x with a > b. Loading P of D pays iff
# c1 + b P < a P, i.e. P > c1 / (a - b), whatever D is; a full hit of x
# tokens beats recompute iff x > (c1 - c0) / (a - b).
LINES = [
    # (c0, a, c1, b, granularity)
    (0.02, 2.0e-5, 0.05, 0.5e-5, 256),
    (0.10, 1.0e-4, 0.30, 0.3e-4, 16),
    (0.01, 3.0e-5, 0.02, 2.9e-5, 64),
]


def _grid_above(v, gran):
    return (math.floor(v / gran) + 1) * gran


@pytest.mark.parametrize("c0,a,c1,b,gran", LINES)
def test_oracle_linear_closed_forms(c0, a, c1, b, gran):
    f = lambda x: ob.curve(*lin(c0, a), x)  # noqa: E731
    g = lambda x: ob.curve(*lin(c1, b), x)  # noqa: E731
    p_star = _grid_above(c1 / (a - b), gran)
    x_star = _grid_above((c1 - c0) / (a - b), gran)
    for D in (p_star, p_star + 3 * gran, 50 * gran, 80000):
        want = p_star if p_star <= D else None
        assert ob.break_even_prefix(f, g, D, gran) == want
    assert ob.break_even_prefix(f, g, p_star - 1, gran) is None
    assert ob.break_even_tokens(f, g, 200000, gran) == x_star
    assert p_star != x_star  # the two points are different quantities
    k = 1.5e-5  # copy time k x
    cp = lambda x: ob.curve(*lin(0.0, k), x)  # noqa: E731
    for D in (1024, 8192, 81920):
        assert math.isclose(ob.max_io(f, g, cp, D), (c0 - c1) + (a - b + k) * D, rel_tol=1e-12)


# The paper's 3B model moves 114,688 B of KV per token (Sec. 2.1); at a
# restore rate R (GB/s) a fully cached x-token prompt takes c1 + (b + beta/R) x
# with beta = 114,688 B/token over R * 1e9 B/s. The threshold is then the first
# grid size above (c1 - c0) / (a - b - beta / (R * 1e9)).
RATES = [(0.02, 2.0e-5, 0.05, 0.5e-5, 16, 55.0), (0.10, 1.0e-4, 0.30, 0.3e-4, 64, 5.2)]


@pytest.mark.parametrize("c0,a,c1,b,gran,rate", RATES)
def test_oracle_hit_from_rate_closed_forms(c0, a, c1, b, gran, rate):
    beta = 114688
    f = lambda x: ob.curve(*lin(c0, a), x)  # noqa: E731
    g0 = lambda x: ob.curve(*lin(c1, b), x)  # noqa: E731
    g = ob.hit_from_rate(g0, beta, rate)
    assert math.isclose(g(81920), c1 + b * 81920 + 81920 * beta / (rate * 1e9), rel_tol=1e-12)
    x_star = _grid_above((c1 - c0) / (a - b - beta / (rate * 1e9)), gran)
    assert ob.break_even_tokens(f, g, 200000, gran) == x_star
    assert x_star != _grid_above((c1 - c0) / (a - b), gran)  # the transfer term matters
    # required bandwidth: the document's bytes over max_io, copy = k x
    k = 1.5e-6
    copy = lambda x: k * x  # noqa: E731
    for D in (1024, 8192, 81920):
        budget = c0 + a * D - (c1 + b * D + D * beta / (rate * 1e9) - k * D)
        want = D * beta / budget / 1e9 if budget > 0 else math.inf
        got = ob.required_GBps(f, g, copy, D, beta)
        assert got == want or math.isclose(got, want, rel_tol=1e-9)
    assert ob.required_GBps(f, lambda x: f(x) + 1.0, lambda x: 0.0, 1000, beta) == math.inf


@pytest.mark.parametrize("c0,a,c1,b,gran,rate", RATES)
def test_library_rate_calls_match_oracle(c0, a, c1, b, gran, rate):
    beta = 114688
    cold, base = be.Curve(*lin(c0, a)), be.Curve(*lin(c1, b))
    f = lambda x: ob.curve(*lin(c0, a), x)  # noqa: E731
    g = ob.hit_from_rate(lambda x: ob.curve(*lin(c1, b), x), beta, rate)
    hit = be.hit_curve_from_restore(base, beta, rate)
    for x in (1000.0, 5000.0, 9000.0, 81920.0):
        assert math.isclose(hit(x), g(x), rel_tol=1e-12)
    assert be.tier_threshold(cold, base, beta, rate, 200000, gran) == \
        ob.break_even_tokens(f, g, 200000, gran)
    copy = be.Curve([1000.0, 9000.0], [1.5e-3, 13.5e-3])
    for D in (1024, 8192, 81920):
        want = ob.required_GBps(f, g, lambda x: 1.5e-6 * x, D, beta)
        assert math.isclose(be.required_GBps(cold, hit, copy, D, beta), want, rel_tol=1e-9)
    with pytest.raises(be.KvxError):
        be.hit_curve_from_restore(base, beta, 0.0)
    with pytest.raises(be.KvxError):
        be.tier_threshold(cold, base, 0, rate, 200000, gran)


def test_oracle_special_cases():
    f = lambda x: ob.curve(*lin(0.05, 2e-5), x)  # noqa: E731
    # a hit that costs as much as recomputing never pays (fixed cost counted twice)
    assert ob.break_even_prefix(f, f, 100000, 16) is None
    assert ob.break_even_tokens(f, f, 100000, 16) is None
    # a free, instant hit pays for the first grid prefix
    zero = lambda x: 0.0  # noqa: E731
    assert ob.break_even_prefix(f, zero, 4096, 256) == 256
    assert ob.break_even_tokens(f, zero, 4096, 256) == 256
    # the threshold needs the hit to stay ahead up to the end: a hit that
    # is faster only in the middle of the range has no threshold
    mid_t, mid_s = [0.0, 1000.0, 2000.0, 3000.0], [1.0, 0.0, 0.0, 100.0]
    g = lambda x: ob.curve(mid_t, mid_s, x)  # noqa: E731
    assert ob.break_even_tokens(f, g, 3000, 100) is None
    assert ob.plan_gate([0, 3, 16], 16, 64) == [True, False, True]


def test_oracle_exact_tie_does_not_pay():
    """With no fixed cost and a hit exactly as dear as recompute, g(P) + f(D-P)
    equals f(D) (exact in binary: integer tokens, a power-of-two slope): the
    inequality is strict, so no prefix pays and there is no threshold."""
    t, s = [0.0, 65536.0], [0.0, 1.0]
    f = lambda x: ob.curve(t, s, x)  # noqa: E731
    assert f(81920) + 0.0 == 1.25
    assert ob.break_even_prefix(f, f, 81920, 256) is None
    assert ob.break_even_tokens(f, f, 81920, 256) is None


def test_oracle_brute_force_frontier_is_minimal():
    rng = random.Random(5)
    for _ in range(20):
        ft = sorted(rng.sample(range(1, 100000), 6))
        fs = sorted(rng.uniform(0.01, 5.0) for _ in ft)
        gs = [rng.uniform(0.01, 2.0) for _ in ft]
        f = lambda x: ob.curve(ft, fs, x)  # noqa: E731
        g = lambda x: ob.curve(ft, gs, x)  # noqa: E731
        D = rng.randrange(1, 60000)
        p = ob.break_even_prefix(f, g, D, 128)
        pays = [P for P in range(128, D + 1, 128) if g(P) + f(D - P) < f(D)]
        assert p == (pays[0] if pays else None)


# ---- library against the oracle -------------------------------------------------


def _random_curves(rng, n_knots=6):
    ft = sorted(rng.sample(range(1, 120000), n_knots))
    fs = sorted(rng.uniform(0.01, 6.0) for _ in ft)
    gt = sorted(rng.sample(range(1, 120000), n_knots))
    gs = sorted(rng.uniform(0.01, 3.0) for _ in gt)
    return (ft, fs), (gt, gs)


@pytest.mark.parametrize("seed", [1, 2, 3, 4])
def test_library_curves_match_oracle(seed):
    rng = random.Random(seed)
    (ft, fs), (gt, gs) = _random_curves(rng)
    F, G = be.Curve(ft, fs), be.Curve(gt, gs)
    f = lambda x: ob.curve(ft, fs, x)  # noqa: E731
    g = lambda x: ob.curve(gt, gs, x)  # noqa: E731
    for x in [0, 1, ft[0], ft[-1], 200000] + [rng.uniform(-1000, 150000) for _ in range(50)]:
        assert math.isclose(F(x), f(x), rel_tol=1e-12, abs_tol=1e-12)
    for _ in range(200):
        D = rng.randrange(0, 100000)
        P = rng.randrange(0, D + 1)
        margin = f(D) - (g(P) + f(D - P))
        if abs(margin) > 1e-9:  # both sides decide in float64; skip ties within rounding
            assert be.load_beats_recompute(F, G, D, P) == (margin > 0)
    for D in (0, 100, 4096, 32768, 81920):
        for gran in (16, 256):
            grid = range(gran, D + 1, gran)
            if all(abs(f(D) - g(P) - f(D - P)) > 1e-9 for P in grid):
                assert be.break_even_prefix(F, G, D, gran) == ob.break_even_prefix(f, g, D, gran)
    for gran in (16, 256, 1000):
        if all(abs(f(y) - g(y)) > 1e-9 for y in range(gran, 100001, gran)):
            assert be.break_even_tokens(F, G, 100000, gran) == ob.break_even_tokens(f, g, 100000, gran)
    C = be.Curve([0, 100000], [0.0, 1.8])
    for D in (1024, 8192, 81920):
        assert math.isclose(be.max_io(F, G, C, D),
                            ob.max_io(f, g, lambda x: ob.curve([0, 100000], [0.0, 1.8], x), D),
                            rel_tol=1e-12, abs_tol=1e-12)


@pytest.mark.parametrize("c0,a,c1,b,gran", LINES)
def test_library_linear_closed_forms(c0, a, c1, b, gran):
    F, G = be.Curve(*lin(c0, a)), be.Curve(*lin(c1, b))
    p_star = _grid_above(c1 / (a - b), gran)
    assert be.break_even_prefix(F, G, 80000, gran) == p_star
    assert be.break_even_prefix(F, G, p_star - 1, gran) is None
    assert be.break_even_tokens(F, G, 200000, gran) == _grid_above((c1 - c0) / (a - b), gran)
    t, s = [0.0, 65536.0], [0.0, 1.0]
    assert be.break_even_prefix(be.Curve(t, s), be.Curve(t, s), 81920, 256) is None


def test_hit_curve_from_restore_adds_the_transfer():
    """Hit TTFT = non-transfer part + bytes / measured rate; with the
    Llama-3.2-3B size of Sec. 2.1 (114,688 B/token) at 55 GB/s an 80k-token
    prefix adds 81920 * 114688 / 55e9 s."""
    base = be.Curve([1024, 81920], [0.05, 0.20])
    hit = be.hit_curve_from_restore(base, 114688, 55.0)
    assert math.isclose(hit(81920), 0.20 + 81920 * 114688 / 55e9, rel_tol=1e-12)
    assert math.isclose(hit(40000), base(40000) + 40000 * 114688 / 55e9, rel_tol=1e-12)
    # a required bandwidth is the document's bytes over max_io
    cold = be.Curve([1024, 81920], [0.1, 3.0])
    copy = be.Curve([1024, 81920], [1024 * 114688 / 55e9, 81920 * 114688 / 55e9])
    budget = cold(81920) - (hit(81920) - copy(81920))
    assert math.isclose(be.required_GBps(cold, hit, copy, 81920, 114688),
                        81920 * 114688 / budget / 1e9, rel_tol=1e-12)


def test_library_rejects_bad_curves():
    good = be.Curve([1, 2], [1.0, 2.0])
    for bad in (be.Curve([1], [1.0]), be.Curve([2, 1], [1.0, 2.0]), be.Curve([1, 1], [1.0, 2.0]),
                be.Curve([1, 2], [1.0, float("nan")]), be.Curve([], [])):
        with pytest.raises(be.KvxError):
            bad(1.0)
        with pytest.raises(be.KvxError):
            be.break_even_prefix(good, bad, 100, 16)
    with pytest.raises(be.KvxError):
        be.load_beats_recompute(good, good, 10, 11)  # prefix longer than the document
    with pytest.raises(be.KvxError):
        be.break_even_tokens(good, good, 100, 0)


# ---- the gate in the step planner --------------------------------------------------


def _oracle_plan(reqs, gate_tokens):
    import oracle.prefix as op

    chunks = []  # (request, key, n_blocks, resident)
    for ri, r in enumerate(reqs):
        for (key, nb), res in zip(op.chunk_keys(r.tokens, 16, 256), r.resident):
            chunks.append((ri, key, nb, bool(res)))
    first = op.dedupe([c[1] for c in chunks])
    load = [0] * len(reqs)
    for i, (ri, key, nb, res) in enumerate(chunks):
        if not chunks[first[i]][3]:
            load[ri] += nb
    loads = ob.plan_gate(load, 16, gate_tokens)
    restored = []  # exact keys, in order of the first loading request that needs them
    for i, (ri, key, nb, res) in enumerate(chunks):
        if not chunks[first[i]][3] and loads[ri] and key not in restored:
            restored.append(key)
    recompute = sum(nb for i, (ri, key, nb, res) in enumerate(chunks)
                    if not chunks[first[i]][3] and key not in restored)
    declined = [ri for ri in range(len(reqs)) if not loads[ri]]
    return restored, recompute, declined, load


@pytest.mark.parametrize("seed", [5, 9])
def test_step_plan_gate_matches_oracle(seed):
    import kvsynth.prefix_tree as pt
    import oracle.prefix as op
    from paper_2609_11744_amd import step

    reqs = pt.make_requests(seed, n=24, lo=256, hi=8192)
    _, _, _, load = _oracle_plan(reqs, 0)
    loads = sorted(lb * 16 for lb in load if lb)
    for gate in (0, loads[len(loads) // 2], loads[-1] + 1):
        restored, recompute, declined, _ = _oracle_plan(reqs, gate)
        plan = step.plan_step(reqs, 16, 256, gate_tokens=gate)
        assert plan.declined == declined
        assert plan.recompute_blocks == recompute
        # the restore list holds the same chunks in the same order (by exact key)
        exact = {}
        for r in reqs:
            for (key, nb), h in zip(op.chunk_keys(r.tokens, 16, 256),
                                    _chunk_hashes(r.tokens)):
                exact[h] = key
        assert [exact[c.key] for c in plan.restore] == restored
        if gate == 0:
            assert not plan.declined and plan.recompute_blocks == 0
        if gate > loads[-1]:
            assert not plan.restore


def _chunk_hashes(tokens):
    import paper_2609_11744_amd as kvx

    h = kvx.kvx_block_hashes(np.asarray(tokens), 16)
    return [int(h[min(k + 16, h.size) - 1]) for k in range(0, h.size, 16)]
