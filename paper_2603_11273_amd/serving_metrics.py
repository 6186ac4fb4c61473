"""Serving metrics of a finished run (host logic; Section 4.1's evaluation
metrics and the burst appendix's per-token ones).

For every request: time to first token (TTFT = first token - arrival),
end-to-end latency (E2EL = last token - arrival), time per output token
(TPOT = (last - first) / (tokens - 1), requests with two tokens or more) and
the inter-token latencies (gaps between consecutive emissions of one
request).  Percentiles are nearest-rank: the smallest value with at least p
percent of the values at or below it, exact on the integer microsecond
times.  Throughput counts requests and tokens over the span from the first
arrival to the end of the run.
"""
from __future__ import annotations

import numpy as np


def nearest_rank(values, p: int):
    """Nearest-rank percentile of a non-empty sequence (integer p in 1..100)."""
    v = np.sort(np.asarray(values))
    k = max(1, -(-len(v) * p // 100))
    return v[k - 1]


def latency_metrics(arrival_us, first_us, finish_us, n_tokens, token_us, t_end_us):
    """arrival_us, first_us, finish_us, n_tokens: per request (same order);
    token_us: the emission times of every request's tokens, request after
    request (n_tokens[i] entries each).  Returns the paper's metrics in
    microseconds (TPOT as a mean, the rest as P50 / P90) plus throughput."""
    arrival = np.asarray(arrival_us, np.int64)
    first = np.asarray(first_us, np.int64)
    finish = np.asarray(finish_us, np.int64)
    ntok = np.asarray(n_tokens, np.int64)
    tok = np.asarray(token_us, np.int64)
    if len(arrival) == 0:
        raise ValueError("no requests")
    if ntok.sum() != len(tok):
        raise ValueError("token_us must hold n_tokens entries per request")
    ttft = first - arrival
    e2el = finish - arrival
    multi = ntok > 1
    tpot = (finish[multi] - first[multi]) / (ntok[multi] - 1)
    # gaps between consecutive tokens of the same request: drop the gap that
    # crosses from one request's last token to the next request's first
    gaps = np.diff(tok)
    starts = np.cumsum(ntok)[:-1]              # index of each later request's first token
    keep = np.ones(len(gaps), bool)
    keep[starts[starts <= len(gaps)] - 1] = False
    itl = gaps[keep]
    span = int(t_end_us) - int(arrival.min())
    n_all = int(ntok.sum())
    return {
        "ttft_p50_us": int(nearest_rank(ttft, 50)),
        "ttft_p90_us": int(nearest_rank(ttft, 90)),
        "e2el_p50_us": int(nearest_rank(e2el, 50)),
        "e2el_p90_us": int(nearest_rank(e2el, 90)),
        "tpot_mean_us": float(tpot.mean()) if len(tpot) else 0.0,
        "itl_p50_us": int(nearest_rank(itl, 50)) if len(itl) else 0,
        "itl_p90_us": int(nearest_rank(itl, 90)) if len(itl) else 0,
        "req_per_s": len(arrival) / (span * 1e-6) if span else 0.0,
        "tok_per_s": n_all / (span * 1e-6) if span else 0.0,
    }
