"""The Poisson/geometric harness on the CPU: its closed forms against the
oracle's (themselves pinned by summation over the geometric law) and the
workload generator against the model it stands for."""

import math

import numpy as np
import pytest

from oracle import bounds
from paper_2606_22327_amd import stochastic as ST
from paper_2606_22327_amd import workloads as W


@pytest.mark.parametrize("mu,M,s_max,o_cap", [(1 / 200, 65536, 512, 3000),
                                              (1 / 50, 8192, 100, 900)])
def test_harness_formulas_match_the_oracle(mu, M, s_max, o_cap):
    m = ST.Model(M=M, mu=mu, s_max=s_max, o_cap=o_cap)
    es = (1 + s_max) / 2
    assert m.mean_volume == pytest.approx(bounds.geometric_mean_volume(es, mu), rel=1e-12)
    assert m.rate_floor == pytest.approx(bounds.poisson_capacity(M, m.alpha))
    for rho in (0.2, 0.7, 0.95):
        lam = m.lam_for(rho)
        assert bounds.poisson_rho(lam, m.mean_volume, M, m.alpha) == pytest.approx(rho)
        assert m.w0(lam) == pytest.approx(bounds.poisson_w0(lam, es, mu), rel=1e-12)
        assert m.cr_bound(rho) == pytest.approx(bounds.poisson_cr_bound(m.alpha, mu, rho))
        assert m.latency_bound(rho) == pytest.approx(
            bounds.poisson_svf_latency_bound(lam, es, mu, M, m.alpha), rel=1e-12)
        for th in (10, 100, 400):
            O0, O1, eps = bounds.poisson_conditional_proxies(mu, th)
            assert m.proxies(th) == pytest.approx((O0, O1, eps), rel=1e-12)
            d = m.mean_volume / (m.mean_volume - eps)
            assert m.distortion(th) == pytest.approx(d)
            assert m.cr_bound(rho, d) == pytest.approx(
                bounds.poisson_cr_bound(m.alpha, mu, rho, d))


def test_poisson_geometric_generator_statistics():
    mu, lam = 1 / 200, 0.17
    b = W.poisson_geometric(lam, mu, 512, 3000, 65536, 20000, 4, tag=3, policies=("svf1bit",),
                            theta=200, O0=84, O1=400)
    o = b.output.astype(np.float64)
    assert abs(o.mean() - 1 / mu) < 0.03 / mu
    assert o.min() >= 1 and o.max() <= 3000
    assert (b.prompt >= 1).all() and (b.prompt <= 512).all()
    assert np.array_equal(b.long_bit, (b.output > 200).astype(np.int8))
    for i in range(b.num_instances):
        a = b.arrival[b.offsets[i]:b.offsets[i + 1]].astype(np.float64)
        assert (np.diff(a) >= 0).all()
        assert abs(len(a) / (a[-1] + 1) - lam) < 0.05 * lam
    # the same parameters and tag give the same arrays whatever the policy
    b2 = W.poisson_geometric(lam, mu, 512, 3000, 65536, 20000, 4, tag=3, policies=("svf",))
    assert np.array_equal(b.output, b2.output) and np.array_equal(b.arrival, b2.arrival)
    assert b2.long_bit is None


def test_middle_selection():
    off = np.array([0, 10, 10, 30])
    idx = ST._middle(off)
    assert idx.tolist() == list(range(1, 9)) + list(range(12, 28))
    assert math.isnan(ST.Model().cr_bound(0.5)) is False
