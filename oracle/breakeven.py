"""Oracle for the break-even gate: when loading a cached prefix beats
recomputing it.

TEST INFRASTRUCTURE ONLY.

Written from the definitions, in float64:
  * Sec. 4.1 (Pareto capture): cold TTFT f(x) and cache-hit TTFT g(x) are
    measured at a sweep of document sizes x and interpolated in between.
    Reading: linear between measured sizes; outside the measured range the
    first / last segment's line continued.
  * Sec. 4.1: caching a prefix of P tokens of a D-token document pays when
    g(P) + f(D - P) < f(D) (strict).
  * Sec. 5.2: the break-even frontier is, per document size, the smallest
    reusable prefix for which that holds. Reading: prefixes are searched on a
    grid of whole multiples of a granularity (a chunk), none if no grid
    prefix pays.
  * Sec. 5.2: max_io(D) = f(D) - (g(D) - t_copy(D)); D's KV bytes over
    max_io(D) is the bandwidth a path needs to match recomputation.
  * Sec. 6.6: the gate keeps one break-even prefix length per source tier
    and recomputes any reusable prefix shorter than it. Reading: the
    threshold is the smallest grid size from which on (up to the largest
    size considered) a fully cached prompt loads faster than it recomputes,
    g(x) < f(x); none if the largest size does not.
  * Step planning under the gate: a request loads its missing chunks when
    their tokens reach the threshold; otherwise it declines, and a chunk is
    restored when at least one request that needs it loads.
  * Secs. 5.2, 6.6: a tier's hit time is its non-transfer part plus the KV
    bytes moved at the tier's restore rate; the bandwidth a path must
    sustain is a document's KV bytes over max_io.

Pinned against closed forms on linear curves (the two break-even points
have different closed forms), special cases, and brute force.
"""
from __future__ import annotations

import math


def curve(tokens, seconds, x):
    """Piecewise-linear curve through (tokens[i], seconds[i]), extended by
    its end segments."""
    n = len(tokens)
    assert n >= 2 and len(seconds) == n
    assert all(tokens[i] < tokens[i + 1] for i in range(n - 1))
    i = 0
    while i < n - 2 and x > tokens[i + 1]:
        i += 1
    x0, x1, y0, y1 = tokens[i], tokens[i + 1], seconds[i], seconds[i + 1]
    slope = (y1 - y0) / (x1 - x0)
    return y0 + slope * (x - x0)


def load_pays(f, g, D, P):
    """f, g: callables (token count -> seconds)."""
    return g(P) + f(D - P) < f(D)


def break_even_prefix(f, g, D, granularity):
    for P in range(granularity, D + 1, granularity):
        if load_pays(f, g, D, P):
            return P
    return None


def break_even_tokens(f, g, max_tokens, granularity):
    grid = list(range(granularity, max_tokens + 1, granularity))
    for x in grid:
        if all(g(y) < f(y) for y in grid if y >= x):
            return x
    return None


def max_io(f, g, copy, D):
    return f(D) - (g(D) - copy(D))


def plan_gate(load_blocks_per_request, block_size, gate_tokens):
    """Per request: True = loads its missing chunks, False = declines. A
    request with nothing to load counts as loading (nothing to decide)."""
    return [lb == 0 or lb * block_size >= gate_tokens for lb in load_blocks_per_request]


def hit_from_rate(non_transfer, bytes_per_token, restore_GBps):
    """Hit time of a tier restoring at restore_GBps (1e9 bytes per second):
    the non-transfer part plus the prompt's KV bytes at that rate."""
    return lambda x: non_transfer(x) + x * bytes_per_token / (restore_GBps * 1e9)


def required_GBps(f, g, copy, D, bytes_per_token):
    """D's KV bytes over max_io(D), in GB/s; infinite without a budget."""
    budget = max_io(f, g, copy, D)
    return D * bytes_per_token / budget / 1e9 if budget > 0 else math.inf
