"""Host aggregates computed from exact integers (CPU only)."""

import numpy as np

import oracle
from paper_2606_22327_amd import report
from paper_2606_22327_amd import svfsim as S
from paper_2606_22327_amd import workloads as W


def _stats_from_oracle(r):
    st = np.zeros(len(r["stats"]), dtype=S.STATS_DTYPE)
    for c, f in enumerate(oracle.STAT_FIELDS):
        if f in st.dtype.names:
            st[f] = r["stats"][:, c]
    return st


def test_nearest_rank():
    v = np.arange(1, 101)
    assert report.nearest_rank(v, 0.99) == 99
    assert report.nearest_rank(v, 0.95) == 95
    assert report.nearest_rank(np.array([7]), 0.99) == 7
    assert report.nearest_rank(np.array([]), 0.5) == 0.0


def test_summary_matches_definitions():
    b = W.config(2, instances=4, n=200)
    r = oracle.run(b, "svf")
    rep = report.summarize(b.arrival, b.output, r["finish"], _stats_from_oracle(r))
    lat = (r["finish"].astype(np.int64) - b.arrival)
    assert rep["requests_finished"] == b.num_requests
    assert rep["mean_latency"] == lat.sum() / len(lat)
    assert rep["p99_latency"] == np.sort(lat)[int(np.ceil(0.99 * len(lat))) - 1]
    assert abs(rep["mean_per_token_latency"] - np.mean(lat / b.output)) < 1e-12
    assert rep["request_steps"] == int(b.output.astype(np.int64).sum())
    # SVF beats FCFS on mean latency on this overloaded workload
    rf = oracle.run(b, "fcfs")
    repf = report.summarize(b.arrival, b.output, rf["finish"], _stats_from_oracle(rf))
    assert rep["mean_latency"] < repf["mean_latency"]
