"""Exhaustive GPU parity at full size.

Configs 2, 3 and 4 in the launch configuration the benchmark times: every
instance of every policy is compared with the CPU oracle element by element
(start, finish, preemption count, admission order) and in every per-instance
statistic.  Each configuration runs once on the GPU (cached for the module);
the comparison is split into tests over blocks of instances so that each test
ends within a minute and reports its progress.
"""

import os
import time

import numpy as np
import pytest

import oracle
from paper_2606_22327_amd import svfsim as S
from paper_2606_22327_amd import workloads as W

pytestmark = pytest.mark.gpu

FIELDS = ("start", "finish", "preempt", "admit_seq")
THREADS = min(16, os.cpu_count() or 1)
# instances per test: the oracle needs about 12 s per 1024 instances of the
# heavy-traffic workload on 16 threads
BLOCKS = {2: 1024, 3: 1024, 4: 2048}
INSTANCES = {2: 4096, 3: 4096, 4: 16384}

_cache = {}


def say(msg):
    print(f"[full-parity] {msg}", flush=True)


def gpu_outputs(cfg):
    if cfg not in _cache:
        _cache.clear()
        b = W.config(cfg)
        assert b.num_instances == INSTANCES[cfg]
        say(f"config {cfg}: {b.num_instances} instances x {len(b.policies)} policies on the GPU")
        with S.Simulator.from_batch(b) as sim:
            sim.run()
            out = {}
            for slot, pol in enumerate(b.policies):
                d = sim.read(slot)
                d["stats"] = sim.stats(slot)
                out[pol] = d
        _cache[cfg] = (b, out)
    return _cache[cfg]


@pytest.mark.parametrize("cfg,lo", [(c, lo) for c in (2, 3, 4)
                                    for lo in range(0, INSTANCES[c], BLOCKS[c])])
def test_every_instance_equals_the_oracle(cfg, lo):
    batch, g = gpu_outputs(cfg)
    ids = list(range(lo, min(lo + BLOCKS[cfg], batch.num_instances)))
    sub = batch.subset(ids)
    a0, a1 = int(batch.offsets[ids[0]]), int(batch.offsets[ids[-1] + 1])
    for pol in batch.policies:
        t0 = time.time()
        r = oracle.run(sub, pol, threads=THREADS)
        for f in FIELDS:
            gv, ov = g[pol][f][a0:a1], r[f]
            if not np.array_equal(gv, ov):
                k = int(np.nonzero(gv != ov)[0][0])
                i = int(np.searchsorted(batch.offsets, a0 + k, side="right") - 1)
                raise AssertionError(f"cfg{cfg} {pol} instance {i} field {f}: gpu {int(gv[k])} "
                                     f"oracle {int(ov[k])}")
        for c, f in enumerate(oracle.STAT_FIELDS):
            if f not in g[pol]["stats"].dtype.names:
                continue
            gv = g[pol]["stats"][f][ids].astype(np.int64)
            ov = r["stats"][:, c].astype(np.int64)
            assert np.array_equal(gv, ov), f"cfg{cfg} {pol} stat {f} in instances {ids[0]}..{ids[-1]}"
        say(f"cfg{cfg} {pol}: instances {ids[0]}..{ids[-1]} equal ({time.time() - t0:.1f}s)")


def test_config2_next_step_admission_every_instance():
    """The current-capacity rule (admission on the next step's memory, with
    evictions when the running set outgrows M) under SVF, SJF and FCFS on all
    4,096 instances of config 2, element by element against the oracle."""
    pols = ("svf+cur", "sjf+cur", "fcfs+cur")
    b = W.config(2, policies=pols)
    say(f"config 2 with next-step admission: {b.num_instances} instances x {len(pols)} policies")
    with S.Simulator.from_batch(b) as sim:
        sim.run()
        g = {}
        for slot, pol in enumerate(pols):
            d = sim.read(slot)
            d["stats"] = sim.stats(slot)
            g[pol] = d
    for pol in pols:
        t0 = time.time()
        r = oracle.run(b, pol, threads=THREADS)
        for f in FIELDS:
            if not np.array_equal(g[pol][f], r[f]):
                k = int(np.nonzero(g[pol][f] != r[f])[0][0])
                i = int(np.searchsorted(b.offsets, k, side="right") - 1)
                raise AssertionError(f"{pol} instance {i} field {f}: gpu {int(g[pol][f][k])} "
                                     f"oracle {int(r[f][k])}")
        for c, f in enumerate(oracle.STAT_FIELDS):
            if f in g[pol]["stats"].dtype.names:
                assert np.array_equal(g[pol]["stats"][f].astype(np.int64), r["stats"][:, c]), (pol, f)
        assert int(g[pol]["stats"]["preemptions"].sum()) > 0
        say(f"{pol}: every instance equal ({time.time() - t0:.1f}s)")
