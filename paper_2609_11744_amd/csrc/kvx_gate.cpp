// Break-even gate (host code): decides from calibrated timing curves whether
// loading a cached prefix beats recomputing it.
//
// Sec. 4.1 (Pareto capture) measures, over a sweep of document sizes, the
// cold TTFT f (full prefill) and the cache-hit TTFT g, and interpolates
// between the measured sizes. Loading a cached prefix of P tokens of a
// D-token document pays when g(P) + f(D - P) < f(D). Sec. 5.2 turns the same
// curves into a transfer budget max_io(D) = f(D) - (g(D) - t_copy(D)).
// Sec. 6.6 runs the calibration offline and keeps one break-even prefix
// length per source tier; at lookup a reusable prefix below it is recomputed.
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "kvx.h"

namespace {

bool valid(const kvx_curve* c) {
  if (!c || c->n < 2 || !c->tokens || !c->seconds) return false;
  for (int32_t i = 0; i < c->n; ++i) {
    if (!std::isfinite(c->tokens[i]) || !std::isfinite(c->seconds[i])) return false;
    if (i > 0 && !(c->tokens[i] > c->tokens[i - 1])) return false;
  }
  return true;
}

// Piecewise-linear through the points; beyond either end, the end segment's
// line continued.
double eval(const kvx_curve* c, double x) {
  int32_t i = 1;
  while (i < c->n - 1 && x > c->tokens[i]) ++i;  // segment [i - 1, i]
  const double x0 = c->tokens[i - 1], x1 = c->tokens[i];
  const double y0 = c->seconds[i - 1], y1 = c->seconds[i];
  return y0 + (y1 - y0) * ((x - x0) / (x1 - x0));
}

bool beats(const kvx_curve* cold, const kvx_curve* hit, int64_t d, int64_t p) {
  return eval(hit, (double)p) + eval(cold, (double)(d - p)) < eval(cold, (double)d);
}

}  // namespace

extern "C" {

kvx_status kvx_curve_eval(const kvx_curve* c, double tokens, double* out) {
  if (!valid(c) || !out || !std::isfinite(tokens)) return KVX_EINVAL;
  *out = eval(c, tokens);
  return KVX_OK;
}

kvx_status kvx_load_beats_recompute(const kvx_curve* cold, const kvx_curve* hit,
                                    int64_t doc_tokens, int64_t prefix_tokens, int32_t* out) {
  if (!valid(cold) || !valid(hit) || !out || doc_tokens < 0 || prefix_tokens < 0 ||
      prefix_tokens > doc_tokens)
    return KVX_EINVAL;
  *out = beats(cold, hit, doc_tokens, prefix_tokens) ? 1 : 0;
  return KVX_OK;
}

kvx_status kvx_break_even_prefix(const kvx_curve* cold, const kvx_curve* hit, int64_t doc_tokens,
                                 int32_t granularity, int64_t* out) {
  if (!valid(cold) || !valid(hit) || !out || doc_tokens < 0 || granularity <= 0)
    return KVX_EINVAL;
  *out = -1;
  for (int64_t p = granularity; p <= doc_tokens; p += granularity)
    if (beats(cold, hit, doc_tokens, p)) {
      *out = p;
      break;
    }
  return KVX_OK;
}

kvx_status kvx_break_even_tokens(const kvx_curve* cold, const kvx_curve* hit, int64_t max_tokens,
                                 int32_t granularity, int64_t* out) {
  if (!valid(cold) || !valid(hit) || !out || max_tokens < 0 || granularity <= 0)
    return KVX_EINVAL;
  // Walk down from the largest grid size while a full hit stays faster.
  int64_t x = (max_tokens / granularity) * granularity, last = -1;
  for (; x >= granularity; x -= granularity) {
    if (!(eval(hit, (double)x) < eval(cold, (double)x))) break;
    last = x;
  }
  *out = last;
  return KVX_OK;
}

kvx_status kvx_max_io(const kvx_curve* cold, const kvx_curve* hit, const kvx_curve* copy,
                      int64_t doc_tokens, double* out_seconds) {
  if (!valid(cold) || !valid(hit) || !valid(copy) || !out_seconds || doc_tokens < 0)
    return KVX_EINVAL;
  const double d = (double)doc_tokens;
  *out_seconds = eval(cold, d) - (eval(hit, d) - eval(copy, d));
  return KVX_OK;
}

kvx_status kvx_hit_curve_from_rate(const kvx_curve* non_transfer, int64_t bytes_per_token,
                                   double restore_GBps, double* out_seconds) {
  if (!valid(non_transfer) || !out_seconds || bytes_per_token <= 0 ||
      !std::isfinite(restore_GBps) || !(restore_GBps > 0))
    return KVX_EINVAL;
  const double rate = restore_GBps * 1e9;  // bytes per second
  for (int32_t i = 0; i < non_transfer->n; ++i)
    out_seconds[i] =
        non_transfer->seconds[i] + non_transfer->tokens[i] * (double)bytes_per_token / rate;
  return KVX_OK;
}

kvx_status kvx_required_GBps(const kvx_curve* cold, const kvx_curve* hit, const kvx_curve* copy,
                             int64_t doc_tokens, int64_t bytes_per_token, double* out_GBps) {
  if (!out_GBps || bytes_per_token <= 0) return KVX_EINVAL;
  double budget = 0;
  const kvx_status st = kvx_max_io(cold, hit, copy, doc_tokens, &budget);
  if (st != KVX_OK) return st;
  *out_GBps = budget > 0 ? (double)doc_tokens * (double)bytes_per_token / budget / 1e9
                         : std::numeric_limits<double>::infinity();
  return KVX_OK;
}

kvx_status kvx_tier_threshold(const kvx_curve* cold, const kvx_curve* non_transfer,
                              int64_t bytes_per_token, double restore_GBps, int64_t max_tokens,
                              int32_t granularity, int64_t* out) {
  if (!valid(non_transfer)) return KVX_EINVAL;
  std::vector<double> sec((size_t)non_transfer->n);
  const kvx_status st =
      kvx_hit_curve_from_rate(non_transfer, bytes_per_token, restore_GBps, sec.data());
  if (st != KVX_OK) return st;
  const kvx_curve hit{non_transfer->tokens, sec.data(), non_transfer->n};
  return kvx_break_even_tokens(cold, &hit, max_tokens, granularity, out);
}

}  // extern "C"
