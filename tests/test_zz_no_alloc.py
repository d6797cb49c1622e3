"""The no-allocation entry point (svf_run_noalloc) against the handle-based
entry points (svf_create + svf_run + svf_read + svf_stats) on the same
batches: every per-request output and every per-instance statistic must be
identical.  Calls come in a row on one GPU, the later ones smaller than the
ones before, so that each must clear what the previous call left in the
shared scratch."""

import numpy as np
import pytest

from paper_2606_22327_amd import svfsim as S
from paper_2606_22327_amd import workloads as W

pytestmark = pytest.mark.gpu

FIELDS = ("start", "finish", "preempt", "admit_seq")


def handle_outputs(b, pols):
    out = {}
    with S.Simulator.from_batch(b, pols) as sim:
        sim.run()
        for slot, pol in enumerate(pols):
            d = sim.read(slot)
            d["stats"] = sim.stats(slot)
            out[pol] = d
    return out


def noalloc_outputs(b, pols):
    import torch

    P, N, I = len(pols), b.num_requests, b.num_instances
    outs = {f: torch.full((max(P * N, 1),), -7, dtype=torch.int32, device="cuda") for f in FIELDS}
    stats = torch.zeros(max(P * I, 1) * S.STATS_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    S.run_noalloc(b.offsets, b.arrival, b.prompt, b.output, b.M, pols, outs["start"],
                  outs["finish"], outs["preempt"], outs["admit_seq"], stats,
                  plan_len=b.plan_len, long_bit=b.long_bit, O0=b.O0, O1=b.O1,
                  max_steps=b.max_steps)
    torch.cuda.synchronize()
    host = {f: outs[f].cpu().numpy() for f in FIELDS}
    st = np.frombuffer(stats.cpu().numpy().tobytes(), dtype=S.STATS_DTYPE)
    res = {}
    for p, pol in enumerate(pols):
        d = {f: host[f][p * N:(p + 1) * N] for f in FIELDS}
        d["stats"] = st[p * I:(p + 1) * I]
        res[pol] = d
    return res


def assert_same(b, pols, label):
    want = handle_outputs(b, pols)
    got = noalloc_outputs(b, pols)
    for pol in pols:
        for f in FIELDS:
            assert np.array_equal(got[pol][f], want[pol][f]), (label, pol, f)
        for f in S.STATS_DTYPE.names:
            assert np.array_equal(got[pol]["stats"][f], want[pol]["stats"][f]), (label, pol, f)
    return want


def test_noalloc_equals_the_handle_entry_points_on_calls_in_a_row():
    # 0: the large-queue shape (event path with the ring profile in LDS)
    b5 = W.config(5, instances=2, n=6000, burst=1500)
    print(f"[noalloc] call 0: config 5 reduced, {b5.num_requests} requests", flush=True)
    assert_same(b5, b5.policies, "cfg5")
    # 1: the 1-bit workload (per-step path with evictions, and the event path)
    b3 = W.config(3, instances=24, n=600)
    print(f"[noalloc] call 1: config 3 reduced, {b3.num_requests} requests x "
          f"{len(b3.policies)} policies", flush=True)
    w = assert_same(b3, b3.policies, "cfg3")
    assert int(w["svf1bit"]["stats"]["preemptions"].sum()) > 0
    # 2: smaller, the burst workload
    b1 = W.config(1, instances=40)
    print(f"[noalloc] call 2: config 1 reduced, {b1.num_requests} requests", flush=True)
    assert_same(b1, ("svf", "sjf", "fcfs"), "cfg1")
    # 3: smaller again, ragged instances with predicted lengths and next-step admission
    r = W.random_small(31, instances=9, n_max=40, s_max=10, o_max=20, M=50, gap_mean=0.6,
                       plan_noise=True)
    r.max_steps = W.default_max_steps(r)
    print(f"[noalloc] call 3: random ragged, {r.num_requests} requests", flush=True)
    assert_same(r, ("svf", "svf+cur", "fcfs"), "random")


def test_noalloc_rejects_a_batch_beyond_its_scratch():
    import torch

    b = W.config(2, instances=2048, n=1000)
    dummy = torch.empty(1, dtype=torch.int32, device="cuda")
    big = torch.empty(3 * b.num_requests, dtype=torch.int32, device="cuda")
    stats = torch.empty(3 * b.num_instances * S.STATS_DTYPE.itemsize, dtype=torch.uint8,
                        device="cuda")
    with pytest.raises(S.SvfError) as ei:
        S.run_noalloc(b.offsets, b.arrival, b.prompt, b.output, b.M, b.policies, big, big, big,
                      big, stats, max_steps=b.max_steps)
    assert ei.value.code == -1 and "scratch" in str(ei.value)
    del dummy
