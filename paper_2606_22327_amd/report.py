"""Host-side aggregates of a finished run (the paper's reporting, Section 4.1).

All inputs are the exact integers the GPU produced; every floating-point
number below is derived on the host in a fixed order, so two runs with
identical integers report identical figures.

  mean latency        sum(finish - a) / n, from an exact int64 sum
  p95 / p99 latency   nearest rank: the value at position ceil(q n) - 1 of the
                      sorted latencies, pooled over all instances
  per-token latency   (finish - a) / o per request, mean and nearest-rank p95/p99
  throughput          generated tokens per simulated step: sum(o) / sum(makespan)
"""

from typing import Dict

import numpy as np


def nearest_rank(sorted_vals: np.ndarray, q: float) -> float:
    n = len(sorted_vals)
    if n == 0:
        return 0.0
    k = int(np.ceil(q * n)) - 1
    return float(sorted_vals[min(max(k, 0), n - 1)])


def summarize(arrival, output, finish, stats) -> Dict[str, float]:
    """Aggregate one policy slot: per-request arrays (int32 [N]) and the
    per-instance statistics (structured array from ``Simulator.stats``)."""
    a = np.asarray(arrival, dtype=np.int64)
    o = np.asarray(output, dtype=np.int64)
    f = np.asarray(finish, dtype=np.int64)
    done = f >= 0
    lat = (f - a)[done]
    lat_sorted = np.sort(lat)
    per_tok = lat / o[done]
    per_tok_sorted = np.sort(per_tok)
    n = int(done.sum())
    sum_lat = int(lat.sum())
    assert sum_lat == int(np.asarray(stats["sum_latency"], dtype=np.int64).sum())
    makespans = int(np.asarray(stats["makespan"], dtype=np.int64).sum())
    return {
        "requests_finished": n,
        "mean_latency": sum_lat / n if n else 0.0,
        "p95_latency": nearest_rank(lat_sorted, 0.95),
        "p99_latency": nearest_rank(lat_sorted, 0.99),
        "mean_per_token_latency": float(per_tok.sum() / n) if n else 0.0,
        "p95_per_token_latency": nearest_rank(per_tok_sorted, 0.95),
        "p99_per_token_latency": nearest_rank(per_tok_sorted, 0.99),
        "tokens_per_step": int(o[done].sum()) / makespans if makespans else 0.0,
        "request_steps": int(np.asarray(stats["request_steps"], dtype=np.int64).sum()),
        "preemptions": int(np.asarray(stats["preemptions"], dtype=np.int64).sum()),
        "peak_mem_max": int(np.asarray(stats["peak_mem"], dtype=np.int64).max()) if len(stats) else 0,
    }
