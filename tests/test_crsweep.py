"""The exact-optimum solver behind the competitive-ratio sweep (host code of
libsvfsim.so) against the oracle's dynamic program, and the sweep's inputs."""

import os

import numpy as np
import pytest

from oracle import bounds, opt
from paper_2606_22327_amd import crsweep as CR
from paper_2606_22327_amd import svfsim as S
from paper_2606_22327_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_native_optimum_matches_the_oracle_dp():
    insts = W.tiny_cr_instances(150)
    b = W.tiny_alpha_instances(2, 40, 3, 7, 4, 6, tag=5)
    insts += [dict(b.instance(i), M=b.M) for i in range(b.num_instances)]
    off = np.concatenate([[0], np.cumsum([len(d["prompt"]) for d in insts])])
    s = np.concatenate([d["prompt"] for d in insts])
    o = np.concatenate([d["output"] for d in insts])
    Ms = np.array([int(d["M"]) for d in insts])
    tot, states, status = S.opt_burst_batch(off, s, o, Ms, threads=4)
    assert (status == 0).all()
    for j, d in enumerate(insts):
        want = opt.optimal_total_latency(d["prompt"], d["output"], int(d["M"]))
        assert int(tot[j]) == want, j
        one, _ = S.opt_burst(d["prompt"], d["output"], int(d["M"]))
        assert one == want


def test_native_optimum_bounds_and_invariance():
    rng = np.random.default_rng(3)
    for _ in range(40):
        n = int(rng.integers(1, 13))
        s = rng.integers(1, 5, n)
        o = rng.integers(1, 7, n)
        pmax = int((s + o).max())
        M = pmax + int(rng.integers(0, 3 * pmax))
        v, _ = S.opt_burst(s, o, M)
        assert v >= bounds.opt_lower_bound_exec(o)                  # Lemma opt_lb_execution
        assert M * v >= bounds.opt_lower_bound_area(s, o, M)        # Proposition opt_lower_bound
        p = rng.permutation(n)
        assert S.opt_burst(s[p], o[p], M)[0] == v
        # more memory never hurts; unbounded memory runs everything at once
        assert S.opt_burst(s, o, M + 5)[0] <= v
    s, o = np.array([2, 3, 1]), np.array([4, 2, 5])
    assert S.opt_burst(s, o, 1000)[0] == int(o.sum())


def test_native_optimum_errors():
    with pytest.raises(S.SvfError) as e:
        S.opt_burst([3], [4], 6)
    assert e.value.name == "SVF_EINFEASIBLE"
    with pytest.raises(S.SvfError) as e:
        S.opt_burst([1], [17], 100)
    assert e.value.name == "SVF_EINVAL"
    with pytest.raises(S.SvfError) as e:
        S.opt_burst([1] * 17, [1] * 17, 100)
    assert e.value.name == "SVF_EINVAL"
    with pytest.raises(S.SvfError) as e:
        S.opt_burst([2] * 8, [3] * 8, 10, state_limit=1)
    assert e.value.name == "SVF_ELIMIT"
    tot, _, status = S.opt_burst_batch([0, 2, 4], [1, 1, 9, 9], [1, 1, 9, 9], [10, 10])
    assert status.tolist() == [0, -4] and tot.tolist() == [2, -1]
    assert S.opt_burst([], [], 5)[0] == 0


def test_alpha_instances_and_bound_table():
    for k in (2, 3, 10):
        b = W.tiny_alpha_instances(k, 50, 6, 12, 4, 6)
        p = b.prompt.astype(np.int64) + b.output
        for i in range(b.num_instances):
            lo, hi = int(b.offsets[i]), int(b.offsets[i + 1])
            assert 6 <= hi - lo <= 12
            assert int(p[lo:hi].max()) * k == b.M
            assert (b.prompt[lo], b.output[lo]) == (4, 6)
            assert (b.arrival[lo:hi] == 0).all()
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "alpha_cr.txt"))
            if ln.strip() and not ln.startswith("#")]
    for num, den, _, printed in rows:
        a = int(num) / int(den)
        assert CR.cr_bound(a) == pytest.approx(bounds.cr_bound(a))
        assert round(CR.cr_bound(a), 2) == pytest.approx(float(printed))


def test_opt_lower_bound_matches_the_paper_and_the_optimum():
    """crsweep.opt_lower_bound is max(area bound of Proposition
    prop:opt_lower_bound, sum o of Lemma lemma:opt_lb_execution): equal to
    the oracle's own implementation of each on random instances, and never
    above the exact optimum of tiny instances."""
    from oracle import bounds, opt as oopt
    from paper_2606_22327_amd import crsweep

    rng = np.random.default_rng(17)
    for _ in range(200):
        n = int(rng.integers(1, 60))
        s = rng.integers(1, 50, n)
        o = rng.integers(1, 50, n)
        M = int((s + o).max()) * int(rng.integers(1, 20))
        want = max(-(-bounds.opt_lower_bound_area(s, o, M) // M), bounds.opt_lower_bound_exec(o))
        assert crsweep.opt_lower_bound(s, o, M) == want
    for inst in W.tiny_cr_instances(60):
        M = int(inst["M"])
        lb = crsweep.opt_lower_bound(inst["prompt"], inst["output"], M)
        assert lb <= oopt.optimal_total_latency(inst["prompt"], inst["output"], M)


@pytest.mark.gpu
def test_lower_bound_sweep_small():
    from paper_2606_22327_amd import crsweep

    rows = crsweep.bound_sweep([2, 10], count=16, n=200)
    for r in rows:
        for p in crsweep.POLICIES:
            assert r.mean_ratio[p] >= 1.0 and r.max_ratio[p] >= r.mean_ratio[p]
        # the proof of thm:svf-burst bounds SVF by these same lower bounds
        assert r.max_ratio["svf"] <= r.bound
