"""Break-even gate: load a cached prefix only where that beats recomputing it
(Secs. 4.1, 5.2, 6.6), on calibrated timing curves. Marshalling over the
kvx_curve calls of libkvx.so; the arithmetic is in the library.

A curve is a pair of sequences (tokens, seconds) from an offline calibration
sweep: the serving engine's cold TTFT at a set of document sizes, its
cache-hit TTFT, or its measured KV copy time. hit_curve_from_restore builds
the hit curve of the pinned-host tier from its non-transfer part and the
restore rate measured here.
"""
from __future__ import annotations

import ctypes

from . import KvxError, _native
from . import _ok


class Curve:
    """Piecewise-linear timing curve (kvx_curve); keeps its arrays alive."""

    def __init__(self, tokens, seconds):
        tokens, seconds = [float(t) for t in tokens], [float(s) for s in seconds]
        if len(tokens) != len(seconds):
            raise ValueError("tokens and seconds differ in length")
        n = len(tokens)
        self.tokens, self.seconds = tokens, seconds
        self._t = (ctypes.c_double * max(n, 1))(*tokens)
        self._s = (ctypes.c_double * max(n, 1))(*seconds)
        self.c = _native.KvxCurve(self._t, self._s, n)

    def __call__(self, tokens) -> float:
        out = ctypes.c_double()
        _ok(_native.lib().kvx_curve_eval(ctypes.byref(self.c), float(tokens), ctypes.byref(out)),
            "kvx_curve_eval")
        return out.value


def hit_curve_from_restore(non_transfer: Curve, bytes_per_token: int, restore_GBps: float) -> Curve:
    """Hit TTFT = its non-transfer part + the KV bytes at the measured restore
    rate (kvx_hit_curve_from_rate), on the same knots."""
    n = len(non_transfer.tokens)
    out = (ctypes.c_double * max(n, 1))()
    _ok(_native.lib().kvx_hit_curve_from_rate(ctypes.byref(non_transfer.c), bytes_per_token,
                                              float(restore_GBps), out),
        "kvx_hit_curve_from_rate")
    return Curve(non_transfer.tokens, list(out[:n]))


def tier_threshold(cold: Curve, non_transfer: Curve, bytes_per_token: int, restore_GBps: float,
                   max_tokens: int, granularity: int):
    """The gate threshold of a tier restoring at restore_GBps (kvx_tier_threshold);
    None if loading never pays up to max_tokens."""
    out = ctypes.c_int64()
    _ok(_native.lib().kvx_tier_threshold(ctypes.byref(cold.c), ctypes.byref(non_transfer.c),
                                         bytes_per_token, float(restore_GBps), max_tokens,
                                         granularity, ctypes.byref(out)), "kvx_tier_threshold")
    return None if out.value < 0 else out.value


def load_beats_recompute(cold: Curve, hit: Curve, doc_tokens: int, prefix_tokens: int) -> bool:
    out = ctypes.c_int32()
    _ok(_native.lib().kvx_load_beats_recompute(ctypes.byref(cold.c), ctypes.byref(hit.c),
                                               doc_tokens, prefix_tokens, ctypes.byref(out)),
        "kvx_load_beats_recompute")
    return bool(out.value)


def break_even_prefix(cold: Curve, hit: Curve, doc_tokens: int, granularity: int):
    """Smallest prefix (a multiple of granularity) worth loading; None if none."""
    out = ctypes.c_int64()
    _ok(_native.lib().kvx_break_even_prefix(ctypes.byref(cold.c), ctypes.byref(hit.c), doc_tokens,
                                            granularity, ctypes.byref(out)),
        "kvx_break_even_prefix")
    return None if out.value < 0 else out.value


def break_even_tokens(cold: Curve, hit: Curve, max_tokens: int, granularity: int):
    """The gate threshold of a tier; None if loading never pays up to max_tokens."""
    out = ctypes.c_int64()
    _ok(_native.lib().kvx_break_even_tokens(ctypes.byref(cold.c), ctypes.byref(hit.c), max_tokens,
                                            granularity, ctypes.byref(out)),
        "kvx_break_even_tokens")
    return None if out.value < 0 else out.value


def max_io(cold: Curve, hit: Curve, copy: Curve, doc_tokens: int) -> float:
    out = ctypes.c_double()
    _ok(_native.lib().kvx_max_io(ctypes.byref(cold.c), ctypes.byref(hit.c), ctypes.byref(copy.c),
                                 doc_tokens, ctypes.byref(out)), "kvx_max_io")
    return out.value


def required_GBps(cold: Curve, hit: Curve, copy: Curve, doc_tokens: int,
                  bytes_per_token: int) -> float:
    """Bandwidth a cache path must sustain for a fully cached document to match
    recomputing it (kvx_required_GBps, Sec. 5.2)."""
    out = ctypes.c_double()
    _ok(_native.lib().kvx_required_GBps(ctypes.byref(cold.c), ctypes.byref(hit.c),
                                        ctypes.byref(copy.c), doc_tokens, bytes_per_token,
                                        ctypes.byref(out)), "kvx_required_GBps")
    return out.value


__all__ = ["Curve", "hit_curve_from_restore", "load_beats_recompute", "break_even_prefix",
           "break_even_tokens", "max_io", "required_GBps", "tier_threshold", "KvxError"]
