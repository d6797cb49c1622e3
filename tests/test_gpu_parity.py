"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Every integer output is compared element by element (start, finish,
preemption count, admission order) together with the per-instance
statistics.  Small cases run the oracle on every instance; the full-size
configurations, in the launch configuration the benchmark times, are compared
on sampled instances (each instance is independent and regenerated from its
own seed) and checked on all instances through properties that hold at any
size; the large-queue configuration is compared on every instance through
digests of the oracle's outputs (tests/golden/oracle_digests.json), and
tests/test_gpu_full_parity.py compares every instance of the others.
"""

import hashlib
import json
import os
import sys
import time

import numpy as np
import pytest

import oracle
from oracle import validate
from paper_2606_22327_amd import svfsim as S
from paper_2606_22327_amd import workloads as W

import hand_cases

pytestmark = pytest.mark.gpu

FIELDS = ("start", "finish", "preempt", "admit_seq")
SFIELDS = ("makespan", "status", "sum_latency", "request_steps", "peak_mem", "preemptions",
           "t_end")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
THREADS = min(16, os.cpu_count() or 1)


def say(msg):
    print(f"[gpu-parity] {msg}", file=sys.stderr, flush=True)


def gpu_run(batch, policies=None, device_inputs=False, chunks=None):
    """Run on the GPU; ``chunks``: list of svf_step sizes instead of one run."""
    pols = tuple(policies or batch.policies)
    sim = S.Simulator.from_batch(batch, pols, device_inputs=device_inputs)
    try:
        if chunks is None:
            sim.run()
        else:
            for c in chunks:
                sim.step(c)
        out = {}
        for slot, pol in enumerate(pols):
            d = sim.read(slot)
            d["stats"] = sim.stats(slot)
            out[pol] = d
    finally:
        sim.close()
    return out


def compare(batch, g, pol, ids=None, t_stop=2 ** 62, max_steps=None, label=""):
    """Oracle on the listed instances (all by default) vs the GPU outputs."""
    ids = list(range(batch.num_instances)) if ids is None else list(ids)
    sub = batch.subset(ids) if len(ids) != batch.num_instances else batch
    r = oracle.run(sub, pol, threads=THREADS, t_stop=t_stop, max_steps=max_steps)
    for j, i in enumerate(ids):
        glo, ghi = int(batch.offsets[i]), int(batch.offsets[i + 1])
        olo, ohi = int(sub.offsets[j]), int(sub.offsets[j + 1])
        for f in FIELDS:
            a = g[f][glo:ghi]
            b = r[f][olo:ohi]
            if not np.array_equal(a, b):
                k = int(np.nonzero(a != b)[0][0])
                raise AssertionError(f"{label} {pol} instance {i} field {f}: first mismatch at "
                                     f"request {k}: gpu {int(a[k])} oracle {int(b[k])}")
        for c, f in enumerate(oracle.STAT_FIELDS):
            if f not in SFIELDS:
                continue
            gv = int(g["stats"][f][i])
            ov = int(r["stats"][j, c])
            assert gv == ov, f"{label} {pol} instance {i} stat {f}: gpu {gv} oracle {ov}"


def properties(batch, g, pol, ids=None):
    """Checks that hold at any size for known-length runs: V1, V2 and the
    statistics recomputed from the schedule."""
    ids = range(batch.num_instances) if ids is None else ids
    for i in ids:
        lo, hi = int(batch.offsets[i]), int(batch.offsets[i + 1])
        a = batch.arrival[lo:hi].astype(np.int64)
        s = batch.prompt[lo:hi].astype(np.int64)
        o = batch.output[lo:hi].astype(np.int64)
        k = g["start"][lo:hi].astype(np.int64)
        f = g["finish"][lo:hi].astype(np.int64)
        st = g["stats"][i]
        assert int(st["status"]) == 0
        assert (k >= a).all() and (f == k + o).all()
        prof = validate.true_profile(s, o, k, int(f.max()) + 1 if hi > lo else 1)
        assert int(prof.max()) <= batch.M
        assert int(st["peak_mem"]) == int(prof.max())
        assert int(st["makespan"]) == (int(f.max()) if hi > lo else 0)
        assert int(st["sum_latency"]) == int((f - a).sum())
        assert int(st["request_steps"]) == int(o.sum())
        assert int(st["preemptions"]) == 0
        seq = g["admit_seq"][lo:hi].astype(np.int64)
        assert np.array_equal(np.sort(seq), np.arange(hi - lo))
        assert (np.diff(k[np.argsort(seq, kind="stable")]) >= 0).all()


# ------------------------------------------------------------ small, full oracle

def test_config1_full():
    b = W.config(1)
    say("config 1: 256 x 50, fcfs/sjf/svf")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, label="cfg1")


def test_config2_subset():
    b = W.config(2, instances=64)
    say("config 2: 64 x 1000")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, label="cfg2")


def test_config3_subset_with_onebit_and_preemption():
    b = W.config(3, instances=64)
    say("config 3: 64 x 1000, 1-bit with preemption")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, label="cfg3")
    assert int(g["svf1bit"]["stats"]["preemptions"].sum()) > 0


def test_config4_subset():
    b = W.config(4, instances=16)
    say("config 4: 16 x 5000")
    g = gpu_run(b)
    compare(b, g["svf"], "svf", label="cfg4")


def test_config5_reduced_bursts():
    b = W.config(5, instances=3, n=6000, burst=1500)
    say("config 5 reduced: 3 x 6000 in bursts of 1500 (sort with merge passes: no)")
    g = gpu_run(b)
    compare(b, g["svf"], "svf", label="cfg5r")


@pytest.mark.parametrize("seed", range(6))
def test_random_ragged(seed):
    say(f"random ragged batches seed {seed}")
    for kw in (dict(), dict(bits=True), dict(plan_noise=True)):
        b = W.random_small(seed, instances=40, n_max=60, s_max=12, o_max=20, M=60,
                           gap_mean=[0.0, 0.3, 1.0][seed % 3], **kw)
        g = gpu_run(b)
        for pol in b.policies:
            compare(b, g[pol], pol, label=f"rand{seed}{kw}")


@pytest.mark.parametrize("seed", range(4))
def test_current_capacity_rule_random(seed):
    """Next-step admission (Alg. 1's Process 2 read literally) with evictions of
    requests whose lengths are known, next to the forward-looking rule."""
    say(f"current-capacity admission, random ragged batches seed {seed}")
    for kw, pols in ((dict(), ("svf+cur", "sjf+cur", "fcfs+cur", "svf")),
                     (dict(bits=True), ("svf1bit+cur", "svf+cur", "svf1bit")),
                     (dict(plan_noise=True), ("svf+cur", "sjf+cur", "sjf"))):
        b = W.random_small(100 + seed, instances=40, n_max=60, s_max=12, o_max=20, M=60,
                           gap_mean=[0.0, 0.3, 1.0, 0.1][seed], **kw)
        b.policies = pols
        b.max_steps = W.default_max_steps(b)
        g = gpu_run(b)
        for pol in pols:
            compare(b, g[pol], pol, label=f"cur{seed}{kw}")
        chunked = gpu_run(b, chunks=[1] * 50 + [9, 4, 10 ** 9])
        for pol in pols:
            for f in FIELDS:
                assert np.array_equal(g[pol][f], chunked[pol][f]), (pol, f)
            assert np.array_equal(g[pol]["stats"], chunked[pol]["stats"]), pol


def test_current_capacity_rule_config2_and_config4():
    pols = ("svf", "svf+cur", "sjf+cur", "fcfs+cur")
    b = W.config(2, instances=32, policies=pols)
    say("current-capacity admission: config 2, 32 x 1000")
    g = gpu_run(b)
    for pol in pols:
        compare(b, g[pol], pol, label="cur-cfg2")
    assert sum(int(g[p]["stats"]["preemptions"].sum()) for p in pols[1:]) > 0
    b4 = W.config(4, instances=4, policies=("svf", "svf+cur"))
    say("current-capacity admission: config 4, 4 x 5000")
    g4 = gpu_run(b4)
    for pol in b4.policies:
        compare(b4, g4[pol], pol, label="cur-cfg4")
    assert int(g4["svf"]["stats"]["preemptions"].sum()) == 0


def test_predictor_in_the_loop_config2_and_config4():
    """Plans from a noisy length predictor (o * LogNormal(0, sigma)): requests
    outrun their plans, get evicted and restart; plans that never undershoot
    never evict."""
    b = W.with_predictor(W.config(2, instances=32, policies=("svf", "sjf", "fcfs", "svf+cur")),
                         0.5)
    say("predicted lengths: config 2, 32 x 1000, sigma 0.5")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, label="pred-cfg2")
    assert int(g["svf"]["stats"]["preemptions"].sum()) > 0
    b.plan_len = np.maximum(b.plan_len, b.output).astype(np.int32)
    b.policies = ("svf", "sjf", "fcfs")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, label="pred-over-cfg2")
        assert int(g[pol]["stats"]["preemptions"].sum()) == 0
    b4 = W.with_predictor(W.config(4, instances=4), 0.5)
    say("predicted lengths: config 4, 4 x 5000, sigma 0.5")
    g4 = gpu_run(b4)
    compare(b4, g4["svf"], "svf", label="pred-cfg4")


def test_ragged_sizes_with_merge_passes():
    """Instances of very different sizes in one batch: 0, 1, a partial chunk,
    and several chunks of the 8192-element LDS sort joined by merge passes."""
    sizes = [0, 1, 70, 9000, 20000, 3]
    parts = []
    rng = np.random.default_rng(42)
    for n in sizes:
        a = np.floor(np.cumsum(rng.exponential(0.7, n))).astype(np.int64)
        parts.append({"arrival": a, "prompt": rng.integers(1, 200, n),
                      "output": rng.integers(1, 300, n)})
    b = W.assemble("ragged", parts, 4096, ("svf", "sjf", "fcfs"))
    say("ragged sizes with merge passes")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, label="ragged")


def test_fused_sort_shapes_boundary_and_wide_keys():
    """Instances sorted by the one-workgroup radix sort in each of its
    workgroup shapes (largest instance 200, 1000, 2000, 4000, 5000, exactly
    5120, 6144 and 8192 requests, and one past the first two), the first size
    past the largest (8193, sorted in chunks and merged),
    and SVF keys just below 2^32 (eight radix passes) next to tiny ones."""
    rng = np.random.default_rng(2606)

    def part(n, s_hi, o_hi, gap):
        a = np.floor(np.cumsum(rng.exponential(gap, n))).astype(np.int64)
        return {"arrival": a, "prompt": rng.integers(1, s_hi + 1, n),
                "output": rng.integers(1, o_hi + 1, n)}

    for top in (200, 1000, 2000, 4000, 5000, 5120, 5121, 6144, 6145, 8192, 8193):
        sizes = [top, 0, 1, max(1, top // 3), 7]
        parts = [part(n, 300, 400, 0.3) for n in sizes]
        b = W.assemble(f"shape{top}", parts, 4096, ("svf", "sjf", "fcfs"))
        say(f"fused sort shape, largest instance {top}")
        g = gpu_run(b)
        for pol in b.policies:
            compare(b, g[pol], pol, label=f"shape{top}")
    # s * o + o(o+1)/2 up to 53000 * 53000 + 53000 * 53001 / 2 < 2^32
    wide = []
    for n in (300, 40):
        p = part(n, 10, 10, 2.0)
        k = rng.random(n) < 0.3
        p["prompt"] = np.where(k, rng.integers(45000, 53001, n), p["prompt"])
        p["output"] = np.where(k, rng.integers(45000, 53001, n), p["output"])
        wide.append(p)
    b = W.assemble("widekeys", wide, 140000, ("svf",))
    key = b.prompt.astype(np.int64) * b.output + (b.output.astype(np.int64) ** 2 + b.output) // 2
    assert int(key.max()).bit_length() == 32
    say("keys just below 2^32")
    g = gpu_run(b)
    compare(b, g["svf"], "svf", label="widekeys")


def test_stepped_many_concurrent_tiny_prompts():
    """The per-step path with more than a thousand requests running at once
    (tiny prompts), next-step admission and evictions, against the oracle."""
    rng = np.random.default_rng(77)
    parts = []
    for n in (1500, 300, 2):
        a = np.floor(np.cumsum(rng.exponential(0.05, n))).astype(np.int64)
        parts.append({"arrival": a, "prompt": rng.integers(1, 3, n),
                      "output": rng.integers(1, 40, n)})
    b = W.assemble("tinyprompts", parts, 3000, ("svf+cur", "sjf+cur"))
    say("stepped: 1500 tiny prompts, M = 3000, next-step admission")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, label="tinyprompts")


def max_concurrent(b, res):
    """Largest number of requests of one instance running at the same step
    (started at k, running at the steps k+1 .. finish)."""
    best = 0
    for i in range(b.num_instances):
        lo, hi = b.offsets[i], b.offsets[i + 1]
        st = res["start"][lo:hi].astype(np.int64)
        fi = res["finish"][lo:hi].astype(np.int64)
        ok = st >= 0
        if not ok.any():
            continue
        ev = np.concatenate([st[ok] + 1, fi[ok] + 1])
        dv = np.concatenate([np.ones(ok.sum(), np.int64), -np.ones(ok.sum(), np.int64)])
        order = np.lexsort((dv, ev))  # at equal steps the ends (-1) go first
        best = max(best, int(np.cumsum(dv[order]).max()))
    return best


def test_ring_in_global_memory():
    """The ring profile kept in global memory instead of LDS (where the ring
    and bitmap pass 64 KB and the list does not fit either), forced on both
    paths; then a long tail without forcing (one request 20,000 steps long per
    instance: a ring of 32,768 slots, too large for LDS, so the host takes the
    finish-ordered list)."""
    env = {"SVFSIM_RING": "global", "SVFSIM_PROFILE": "ring", "SVFSIM_STEP_PROFILE": "ring"}
    old = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    try:
        b = W.config(2, instances=12, n=400)
        say("ring in global memory: config 2 reduced")
        g = gpu_run(b)
        for pol in b.policies:
            compare(b, g[pol], pol, label="gring-cfg2")
        b3 = W.config(3, instances=8)
        say("ring in global memory: config 3 reduced (1-bit, evictions)")
        g3 = gpu_run(b3, chunks=[500, 1, 2000, 10 ** 9])
        for pol in b3.policies:
            compare(b3, g3[pol], pol, label="gring-cfg3")
        assert int(g3["svf1bit"]["stats"]["preemptions"].sum()) > 0
        r = W.random_small(9, instances=40, n_max=60, s_max=12, o_max=20, M=60, gap_mean=0.3,
                           plan_noise=True)
        gr = gpu_run(r)
        for pol in r.policies:
            compare(r, gr[pol], pol, label="gring-random")
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    rng = np.random.default_rng(5)
    parts = []
    for i in range(6):
        n = 300
        a = np.sort(rng.integers(0, 2000, n))
        o = rng.integers(1, 400, n)
        o[rng.integers(0, n)] = 20000
        parts.append({"arrival": a, "prompt": rng.integers(1, 200, n), "output": o})
    bl = W.assemble("longtail", parts, 40000, ("svf", "sjf", "fcfs"))
    say("one request 20000 steps long per instance")
    gl = gpu_run(bl)
    for pol in bl.policies:
        compare(bl, gl[pol], pol, label="longtail")


@pytest.mark.parametrize("profile", ["ring", "list", "list-lds7", "list-lds64"])
def test_event_path_both_profiles(profile):
    """The event path keeps the future memory profile either as the ring of
    G = D + tau or as the finish-ordered list (the host picks by LDS and
    occupancy).  Each forced on the same batches, against the oracle: burst
    and online instances, ragged sizes, a step-by-step run with partial reads.
    The list-ldsN cases give the list in LDS room for only N entries, so
    segments stop when it is full and the continuation launch (room for the
    host's bound) finishes them, also inside step-by-step runs."""
    os.environ["SVFSIM_PROFILE"] = profile.split("-")[0]
    cap = int(profile.split("lds")[1]) if "lds" in profile else None
    if cap:
        os.environ["SVFSIM_LIST_LDS_CAP"] = str(cap)
    try:
        most = 0
        b = W.config(2, instances=12, n=400)
        say(f"profile {profile}: config 2 reduced")
        g = gpu_run(b)
        for pol in b.policies:
            compare(b, g[pol], pol, label=f"{profile}-cfg2")
            most = max(most, max_concurrent(b, g[pol]))
        b1 = W.config(1, instances=64)
        g1 = gpu_run(b1)
        for pol in b1.policies:
            compare(b1, g1[pol], pol, label=f"{profile}-cfg1")
        b4 = W.config(4, instances=6, n=1500)
        g4 = gpu_run(b4, chunks=[97, 1, 1000, 5, 4000, 1 << 20])
        compare(b4, g4["svf"], "svf", label=f"{profile}-cfg4-chunked")
        most = max(most, max_concurrent(b4, g4["svf"]))
        r = W.random_small(5, instances=40, n_max=120, s_max=30, o_max=90, M=300, gap_mean=0.8)
        gr = gpu_run(r, ("svf", "sjf", "fcfs"))
        for pol in ("svf", "sjf", "fcfs"):
            compare(r, gr[pol], pol, label=f"{profile}-random")
        if cap:
            assert most > cap, "no segment outgrew the LDS list: the continuation went untested"
    finally:
        del os.environ["SVFSIM_PROFILE"]
        os.environ.pop("SVFSIM_LIST_LDS_CAP", None)


@pytest.mark.parametrize("profile", ["ring", "list", "list-lds7", "list-lds64"])
def test_stepped_path_both_profiles(profile):
    """The per-step path (1-bit SVF, predicted lengths, next-step admission)
    keeps the planned profile either in the ring or in the finish-ordered
    list (early completions and evictions remove entries from its middle).
    Each forced on the same batches, against the oracle, also step by step.
    The list-ldsN cases give the list in LDS room for only N entries, so
    segments stop inside the admission phase of a step and the continuation
    launch resumes them there."""
    os.environ["SVFSIM_STEP_PROFILE"] = profile.split("-")[0]
    cap = int(profile.split("lds")[1]) if "lds" in profile else None
    if cap:
        os.environ["SVFSIM_STEP_LDS_CAP"] = str(cap)
    try:
        b3 = W.config(3, instances=24, n=600)
        say(f"step profile {profile}: config 3 reduced")
        g3 = gpu_run(b3)
        for pol in b3.policies:
            compare(b3, g3[pol], pol, label=f"{profile}-cfg3")
        assert int(g3["svf1bit"]["stats"]["preemptions"].sum()) > 0
        b4 = W.with_predictor(W.config(4, instances=3, n=2000, policies=("svf", "svf+cur")), 0.5)
        say(f"step profile {profile}: config 4 reduced, predicted lengths, chunked")
        g4 = gpu_run(b4, chunks=[53, 1, 700, 3, 2500, 1 << 20])
        for pol in b4.policies:
            compare(b4, g4[pol], pol, label=f"{profile}-pred-cfg4")
        for seed in range(3):
            r = W.random_small(300 + seed, instances=40, n_max=80, s_max=12, o_max=30, M=70,
                               gap_mean=[0.0, 0.3, 1.0][seed], bits=seed == 0,
                               plan_noise=seed != 0)
            r.policies = ("svf", "svf+cur", "sjf+cur") if seed else ("svf1bit", "svf1bit+cur")
            r.max_steps = W.default_max_steps(r)
            gr = gpu_run(r)
            for pol in r.policies:
                compare(r, gr[pol], pol, label=f"{profile}-random{seed}")
        if cap:
            assert max_concurrent(b3, g3["svf1bit"]) > cap, "no list outgrew the LDS room"
    finally:
        del os.environ["SVFSIM_STEP_PROFILE"]
        os.environ.pop("SVFSIM_STEP_LDS_CAP", None)


@pytest.mark.parametrize("profile", ["ring", "list"])
def test_eviction_hand_worked_cases(profile):
    """The hand-worked eviction instances (tests/golden/eviction_cases.txt)
    through the C ABI, compared with the values derived by hand (not with the
    oracle): each case replicated over 300 instances of one launch, run to the
    end or stopped by svf_step before the case's stop step, with the per-step
    path's planned profile forced to the ring or to the finish-ordered list."""
    os.environ["SVFSIM_STEP_PROFILE"] = profile
    try:
        for case in hand_cases.load():
            one = case["batch"]
            reps = 300
            b = W.assemble(case["name"], [one.instance(0)] * reps, one.M, one.policies,
                           O0=one.O0, O1=one.O1)
            say(f"hand case {case['name']} ({case['policy']}), profile {profile}")
            chunks = None if case["t_stop"] is None else [case["t_stop"]]
            g = gpu_run(b, chunks=chunks)[case["policy"]]
            n = int(one.offsets[1])
            for f, want in case["expected"].items():
                got = g[f].reshape(reps, n)
                assert (got == want[None, :]).all(), (case["name"], f, got[0].tolist())
            for f in SFIELDS:
                got = g["stats"][f].astype(np.int64)
                assert (got == case["stats"][f]).all(), (case["name"], f, int(got[0]))
    finally:
        del os.environ["SVFSIM_STEP_PROFILE"]


def test_degenerate_cases():
    say("degenerate cases")
    # all instances empty
    e = W.assemble("empty", [{"arrival": [], "prompt": [], "output": []}] * 5, 10, ("svf",))
    g = gpu_run(e)
    assert g["svf"]["stats"]["t_end"].tolist() == [0] * 5
    # one request; exact fit s + o = M; equal keys; unbounded memory
    parts = [
        {"arrival": np.array([3]), "prompt": np.array([7]), "output": np.array([9])},
        {"arrival": np.zeros(20), "prompt": np.full(20, 4), "output": np.full(20, 12)},
        {"arrival": np.arange(30) // 3, "prompt": np.full(30, 1), "output": np.full(30, 1)},
    ]
    b = W.assemble("deg", parts, 16, ("svf", "sjf", "fcfs"))
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, label="deg")
    big = W.config(2, instances=4, n=300)
    b2 = W.assemble("big", [big.instance(i) for i in range(4)], 2 ** 29 // 4,
                    ("svf", "sjf", "fcfs"))
    g = gpu_run(b2)
    for pol in b2.policies:
        compare(b2, g[pol], pol, label="unbounded")
        assert np.array_equal(g[pol]["start"], b2.arrival)


def _parts_near_largest_budget(seed, instances, M, plans):
    """Four requests at t = 0 whose prompts nearly fill M (slack of 0..63
    tokens, so that a few steps of growth overflow it) and three smaller later
    arrivals; lengths 1..12, plans 1..4 when asked for."""
    rng = np.random.Generator(np.random.PCG64(seed))
    parts = []
    for _ in range(instances):
        base = (M - int(rng.integers(0, 64))) // 4
        s = np.concatenate([base + rng.integers(-3, 4, 4), rng.integers(2 ** 18, 2 ** 26, 3)])
        a = np.concatenate([np.zeros(4, np.int64), np.sort(rng.integers(0, 20, 3))])
        o = rng.integers(1, 13, 7)
        d = {"arrival": a, "prompt": s, "output": o, "long_bit": (o > 4).astype(np.int8)}
        if plans:
            d["plan_len"] = rng.integers(1, 5, 7)
        parts.append(d)
    return parts


@pytest.mark.parametrize("profile", ["ring", "list"])
def test_largest_memory_budget(profile):
    """M = 2^30 - 1, the largest budget the library accepts, with prompts of
    up to 2^28 tokens: every memory total, planned sum and release step sits
    near the top of the int32 range.  Known lengths, 1-bit plans, noisy plans
    and next-step admission (evictions included), each profile forced."""
    M = 2 ** 30 - 1
    os.environ["SVFSIM_PROFILE"] = profile
    os.environ["SVFSIM_STEP_PROFILE"] = profile
    try:
        for plans, pols in ((False, ("svf", "sjf", "fcfs", "svf1bit", "svf+cur", "fcfs+cur",
                                     "svf1bit+cur")),
                            (True, ("svf", "sjf", "svf+cur"))):
            b = W.assemble("budget", _parts_near_largest_budget(11, 48, M, plans), M, pols,
                           O0=2, O1=8)
            say(f"largest budget, {profile}, plans={plans}")
            g = gpu_run(b)
            evicted = 0
            for pol in pols:
                compare(b, g[pol], pol, label=f"budget-{profile}")
                assert int(g[pol]["stats"]["peak_mem"].max()) > M - 64
                evicted += int(g[pol]["preempt"].sum())
            assert evicted > 0, "no eviction near the budget"
    finally:
        del os.environ["SVFSIM_PROFILE"]
        del os.environ["SVFSIM_STEP_PROFILE"]


def test_step_by_step_equals_run_and_partial_states():
    b = W.random_small(11, instances=24, n_max=50, s_max=10, o_max=16, M=40, gap_mean=0.5,
                       bits=True)
    say("svf_step chunks vs one run, and vs the oracle stopped at the same step")
    full = gpu_run(b)
    T = max(int(full[p]["stats"]["t_end"].max()) for p in b.policies)
    ones = min(T, 3000)
    one = gpu_run(b, chunks=[1] * ones + [T])
    for pol in b.policies:
        for f in FIELDS:
            assert np.array_equal(full[pol][f], one[pol][f]), (pol, f)
        assert np.array_equal(full[pol]["stats"], one[pol]["stats"]), pol
    for stop in (0, 1, 5, 17, 60, 333):
        g = gpu_run(b, chunks=[stop] if stop else [0])
        for pol in b.policies:
            compare(b, g[pol], pol, t_stop=stop, label=f"t_stop={stop}")
    g = gpu_run(b, chunks=[7, 3, 11, 10 ** 9])
    for pol in b.policies:
        compare(b, g[pol], pol, label="chunks")
    # known lengths only: the event-driven path across many small launches
    b2 = W.config(2, instances=16, n=300)
    full = gpu_run(b2)
    T = max(int(full[p]["stats"]["t_end"].max()) for p in b2.policies)
    parts = gpu_run(b2, chunks=[1] * 200 + [13] * 50 + [T])
    for pol in b2.policies:
        for f in FIELDS:
            assert np.array_equal(full[pol][f], parts[pol][f]), (pol, f)
        assert np.array_equal(full[pol]["stats"], parts[pol]["stats"]), pol
        for stop in (150, 777):
            g = gpu_run(b2, chunks=[stop])
            compare(b2, g[pol], pol, t_stop=stop, label=f"known t_stop={stop}")


def test_step_budget_exhaustion():
    b = W.config(2, instances=8, n=400)
    b.max_steps = 150
    say("max_steps exhaustion")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, max_steps=150, label="exhausted")
        assert (g[pol]["stats"]["status"] == 1).all()
    b3 = W.config(3, instances=8, n=400)
    b3.max_steps = 200
    g = gpu_run(b3)
    for pol in b3.policies:
        compare(b3, g[pol], pol, max_steps=200, label="exhausted3")


def test_device_inputs_and_determinism():
    import torch
    b = W.config(3, instances=32)
    say("device inputs + determinism")
    g1 = gpu_run(b)
    g2 = gpu_run(b, device_inputs=True)
    for pol in b.policies:
        for f in FIELDS:
            assert np.array_equal(g1[pol][f], g2[pol][f])
        assert np.array_equal(g1[pol]["stats"], g2[pol]["stats"])
    sim = S.Simulator.from_batch(b)
    sim.run()
    a = sim.read(0)
    sim.reset()
    sim.run()
    c = sim.read(0)
    n = sim.num_requests
    dev = [torch.empty(n, dtype=torch.int32, device="cuda") for _ in range(4)]
    sim.read_device(0, *dev)
    torch.cuda.synchronize()
    sim.close()
    for f in FIELDS:
        assert np.array_equal(a[f], c[f])
    for f, t in zip(FIELDS, dev):
        assert np.array_equal(a[f], t.cpu().numpy())


# ------------------------------------------------ full sizes, sampled

def _sample(n_inst, k, seed):
    rng = np.random.default_rng(seed)
    ids = sorted(set([0, n_inst - 1] + rng.choice(n_inst, size=k, replace=False).tolist()))
    return ids


@pytest.mark.parametrize("kw", [dict(bits=True), dict(plan_noise=True)], ids=["onebit", "noisy"])
def test_stepped_jumps_across_launch_limits(kw):
    """The per-step path jumps from one step at which something can happen to
    the next (arrivals ranked above the blocked head, completions, planned
    lengths running out, the first overflow of M, the head's release step);
    a launch's step limit cuts a jump short.  Runs in irregular step chunks
    equal one run to completion, and the oracle, in every output and
    statistic (request-steps and peak memory included)."""
    b = W.random_small(404, instances=60, n_max=80, s_max=16, o_max=40, M=90,
                       gap_mean=0.7, **kw)
    b.policies = ("svf1bit", "svf", "sjf+cur") if kw.get("bits") else ("svf", "sjf", "fcfs+cur")
    b.max_steps = W.default_max_steps(b)
    say(f"stepped jumps {kw}: one run")
    whole = gpu_run(b)
    say(f"stepped jumps {kw}: chunks")
    chunks = [1, 2, 3, 5, 8, 13, 21, 34, 55, 89] * 4 + [10 ** 9]
    parts = gpu_run(b, chunks=chunks)
    for pol in b.policies:
        for f in FIELDS:
            assert np.array_equal(whole[pol][f], parts[pol][f]), (pol, f)
        assert np.array_equal(whole[pol]["stats"], parts[pol]["stats"]), pol
        compare(b, whole[pol], pol, label=f"jumps{kw}")


def test_concurrent_launches_equal_one_stream(monkeypatch):
    """A batch with event-driven and per-step segments runs its two launches on
    two streams; on one stream (SVFSIM_CONCURRENT=0) every output is the same,
    and both equal the oracle on sampled instances."""
    b = W.config(3, instances=64, n=500)
    say("concurrent launches vs one stream")
    two = gpu_run(b)
    monkeypatch.setenv("SVFSIM_CONCURRENT", "0")
    one = gpu_run(b)
    for pol in b.policies:
        for f in FIELDS:
            assert np.array_equal(two[pol][f], one[pol][f]), (pol, f)
        assert np.array_equal(two[pol]["stats"], one[pol]["stats"]), pol
        compare(b, two[pol], pol, ids=_sample(b.num_instances, 8, 11), label="concurrent")


def test_many_tiny_instances():
    """100,000 instances of one to eight requests under four policies: 400,000
    single-wave segments, far more workgroups than wave slots, on both paths
    (1-bit plans take the per-step one)."""
    b = W.random_small(21, instances=100000, n_max=8, s_max=6, o_max=10, M=24, gap_mean=0.5,
                       bits=True)
    pols = ("svf", "sjf", "fcfs", "svf1bit")
    say(f"many tiny instances: {b.num_instances} instances, {b.num_requests} requests")
    g = gpu_run(b, pols)
    for pol in pols:
        compare(b, g[pol], pol, label="tiny")


def test_two_handles_on_two_streams_at_once():
    """Two handles, each on a stream of its own (default priority), launched
    back to back without synchronising: each owns its buffers, so both give
    what one handle alone gives (config 3: event-driven and per-step
    segments, issue priorities on)."""
    import torch
    b = W.config(3, instances=48, n=600)
    alone = gpu_run(b)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    h1 = S.Simulator.from_batch(b, stream=s1.cuda_stream)
    h2 = S.Simulator.from_batch(b, stream=s2.cuda_stream)
    try:
        say("two handles on two streams")
        h1.run()
        h2.run()
        for h in (h1, h2):
            for slot, pol in enumerate(b.policies):
                d = h.read(slot)
                for f in FIELDS:
                    assert np.array_equal(d[f], alone[pol][f]), (pol, f)
                assert np.array_equal(h.stats(slot), alone[pol]["stats"]), pol
    finally:
        h1.close()
        h2.close()


def test_issue_priorities_do_not_change_results(monkeypatch):
    """More segments than the GPU holds at once (several rounds of resident
    workgroups), on the event and the per-step path: outputs with the waves'
    issue priorities set by their progress equal those with one priority for
    all, and the oracle's."""
    b = W.random_small(77, instances=12000, n_max=30, s_max=12, o_max=20, M=60,
                       gap_mean=0.3, bits=True)
    b.policies = ("svf", "svf1bit", "sjf+cur")
    b.max_steps = W.default_max_steps(b)
    say("issue priorities: 12000 x <= 30 requests, 3 policies, priorities on")
    on = gpu_run(b)
    monkeypatch.setenv("SVFSIM_ISSUE_PRIO", "0")
    say("issue priorities off")
    off = gpu_run(b)
    for pol in b.policies:
        for f in FIELDS:
            assert np.array_equal(on[pol][f], off[pol][f]), (pol, f)
        assert np.array_equal(on[pol]["stats"], off[pol]["stats"]), pol
        compare(b, on[pol], pol, label="prio")


def test_full_config2_sampled():
    b = W.config(2)
    say("full config 2: 4096 x 1000 x 3 policies")
    t0 = time.time()
    g = gpu_run(b)
    say(f"  gpu done in {time.time() - t0:.1f}s; comparing samples")
    for pol in b.policies:
        compare(b, g[pol], pol, ids=_sample(b.num_instances, 30, 2), label="cfg2full")
        assert (g[pol]["stats"]["status"] == 0).all()
        assert (g[pol]["stats"]["preemptions"] == 0).all()
        properties(b, g[pol], pol, ids=_sample(b.num_instances, 200, 7))


def test_full_config3_sampled():
    b = W.config(3)
    say("full config 3: 4096 x 1000 x 4 policies")
    g = gpu_run(b)
    for pol in b.policies:
        compare(b, g[pol], pol, ids=_sample(b.num_instances, 30, 3), label="cfg3full")
        assert (g[pol]["stats"]["status"] == 0).all()


def test_full_config4_sampled():
    b = W.config(4)
    say("full config 4: 16384 x 5000")
    t0 = time.time()
    g = gpu_run(b)
    say(f"  gpu done in {time.time() - t0:.1f}s; comparing samples")
    compare(b, g["svf"], "svf", ids=_sample(b.num_instances, 20, 4), label="cfg4full")
    assert (g["svf"]["stats"]["status"] == 0).all()
    properties(b, g["svf"], "svf", ids=_sample(b.num_instances, 60, 5))


def test_full_config5_against_stored_oracle_digests():
    path = os.path.join(GOLDEN, "oracle_digests.json")
    data = json.load(open(path))["cfg5/svf"]
    b = W.config(5)
    assert sorted(map(int, data["instances"])) == list(range(b.num_instances)), \
        "the stored digests do not cover every instance"
    say("full config 5: 64 x 200000")
    g = gpu_run(b)["svf"]
    # with known lengths neither run can reach its step budget (the budgets of
    # the sample and the full batch differ), so the outputs do not depend on it
    assert (g["stats"]["status"] == 0).all()
    for i_str, ent in data["instances"].items():
        i = int(i_str)
        lo, hi = int(b.offsets[i]), int(b.offsets[i + 1])
        h = hashlib.sha256()
        for f in FIELDS:
            h.update(np.ascontiguousarray(g[f][lo:hi], dtype=np.int32).tobytes())
        assert h.hexdigest() == ent["sha256_start_finish_preempt_admit"], f"instance {i}"
        for f in SFIELDS:
            assert int(g["stats"][f][i]) == ent["stats"][f], (i, f)
    properties(b, g, "svf")


def test_full_config4_predictor_sampled():
    """The full heavy-traffic workload planned with predicted lengths (sigma
    0.5), in one launch: every instance against the oracle through the
    digests of its outputs stored per block of 1,024 instances
    (tests/golden/oracle_digests.json), sampled instances directly, and every
    instance through properties that hold with preemption."""
    b = W.with_predictor(W.config(4), 0.5)
    say(f"full config 4 with predicted lengths: {b.num_instances} instances")
    t0 = time.time()
    g = gpu_run(b)
    say(f"gpu done in {time.time() - t0:.1f}s")
    st = g["svf"]["stats"]
    assert (st["status"] == 0).all()
    assert (g["svf"]["finish"] == g["svf"]["start"] + b.output).all()
    assert (g["svf"]["start"] >= b.arrival).all()
    assert (st["peak_mem"] <= b.M).all()
    assert int(st["preemptions"].sum()) == int(g["svf"]["preempt"].sum()) > 0
    ids = [0, 1, 4095, 8191, 12000, b.num_instances - 1]
    compare(b, g["svf"], "svf", ids=ids, label="pred-full-cfg4")
    check_block_digests(b, g["svf"], "cfg4-pred0.5/svf")


def test_full_config4_next_step_admission_against_stored_oracle_digests():
    """The full heavy-traffic workload under SVF with next-step admission (the
    current-capacity rule: evictions whenever the running set outgrows M), in
    one launch: every instance against the oracle through the digests stored
    per block of 1,024 instances, and properties that hold with preemption."""
    b = W.config(4, policies=("svf+cur",))
    say(f"full config 4 with next-step admission: {b.num_instances} instances")
    t0 = time.time()
    g = gpu_run(b)["svf+cur"]
    say(f"gpu done in {time.time() - t0:.1f}s")
    st = g["stats"]
    assert (st["status"] == 0).all()
    assert (g["finish"] == g["start"] + b.output).all()
    assert (st["peak_mem"] <= b.M).all()
    assert int(st["preemptions"].sum()) == int(g["preempt"].sum()) > 0
    check_block_digests(b, g, "cfg4/svf+cur")


def check_block_digests(b, res, key):
    """Every block of instances of ``res`` against the oracle digests stored
    under ``key`` (tests/golden/make_oracle_digests.py)."""
    data = json.load(open(os.path.join(GOLDEN, "oracle_digests.json")))[key]
    blk = int(data["block"])
    assert sorted(map(int, data["blocks"])) == list(range(0, b.num_instances, blk)), \
        "the stored digests do not cover every block"
    st = res["stats"]
    for lo_s, ent in data["blocks"].items():
        lo = int(lo_s)
        hi = min(lo + blk, b.num_instances)
        a0, a1 = int(b.offsets[lo]), int(b.offsets[hi])
        h = hashlib.sha256()
        for f in FIELDS:
            h.update(np.ascontiguousarray(res[f][a0:a1], dtype=np.int32).tobytes())
        cols = np.stack([st[f][lo:hi].astype(np.int64) for f in SFIELDS], axis=1)
        h.update(np.ascontiguousarray(cols, dtype=np.int64).tobytes())
        assert h.hexdigest() == ent["sha256"], f"{key}: instances {lo}..{hi - 1}"


def test_poisson_geometric_bounds_and_parity():
    """The stochastic model of Section 3.3 on the GPU: sampled instances
    against the oracle, and the measured mean latency against the bounds of
    thm:svf_poisson and thm:svf_1bit_poisson where they apply (rho < 1)."""
    from paper_2606_22327_amd import stochastic as ST
    model = ST.Model()
    say("poisson/geometric: rho 0.5, 0.9, 2.0; 16 x 4000 per setting")
    rows = ST.run(model, (0.5, 0.9, 2.0), instances=16, n=4000, tag=7, keep_outputs=True)
    assert len(rows) == 3 * 5
    for r in rows:
        b, out = r.extra["batch"], r.extra["out"]
        compare(b, dict(out, stats=r.extra["stats"]), r.policy, ids=[0, 9, 15],
                label=f"poisson rho={r.rho} {r.policy} th={r.theta}")
        assert r.ratio >= 1.0
        if r.rho < 1 and r.policy in ("svf", "svf1bit"):
            assert r.mean_latency <= r.latency_bound, r
            assert r.ratio <= r.cr_bound, r


def test_cr_sweep_and_search():
    """Tiny burst instances at several alpha: the GPU's total latencies equal
    the oracle's, each policy is at or above the exact optimum, and SVF stays
    within 1 + 2/(1 - alpha) (Theorem thm:svf-burst), also on the instances
    an evolutionary search drives towards a large ratio."""
    from oracle import opt
    from paper_2606_22327_amd import crsweep as CR
    say("competitive-ratio sweep: alpha 1/2, 1/4, 1/10; 256 instances each")
    for k in (2, 4, 10):
        b = W.tiny_alpha_instances(k, 256, 6, 10, 4, 6, tag=9)
        g = gpu_run(b)
        for pol in b.policies:
            compare(b, g[pol], pol, label=f"alpha1/{k}")
        r = CR.sweep([k], 256, n_hi=10, tag=9)[0]
        for pol in CR.POLICIES:
            assert r.mean_ratio[pol] >= 1.0
        assert r.max_ratio["svf"] <= r.bound
    say("evolutionary search at alpha 1/2: 64 members, 4 generations")
    res = CR.search(2, population=64, generations=4, n_hi=8, threads=8)
    assert 1.0 <= res.max_ratio["svf"] <= res.bound
    s, o = res.worst["svf"]
    want = opt.optimal_total_latency(s, o, res.M)
    bw = W.assemble("worst", [{"arrival": np.zeros(len(s)), "prompt": np.array(s),
                               "output": np.array(o)}], res.M, ("svf",))
    tel = int(oracle.run(bw, "svf")["stats"][0, 2])
    assert tel / want == pytest.approx(res.max_ratio["svf"])
