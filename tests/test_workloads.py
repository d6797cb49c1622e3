"""The synthetic workloads: determinism, shapes and distribution sanity."""

import numpy as np
import pytest

from paper_2606_22327_amd import workloads as W


def test_per_instance_streams_are_independent_of_the_sample():
    full = W.config(2, instances=8)
    sub = W.config(2, instances=[5, 2])
    for j, i in enumerate([5, 2]):
        a = full.instance(i)
        b = sub.instance(j)
        for k in ("arrival", "prompt", "output"):
            assert np.array_equal(a[k], b[k])


def test_config3_reuses_config2_arrays():
    b2 = W.config(2, instances=3)
    b3 = W.config(3, instances=3)
    assert np.array_equal(b2.arrival, b3.arrival)
    assert np.array_equal(b2.prompt, b3.prompt)
    assert np.array_equal(b2.output, b3.output)
    assert b3.long_bit is not None and b3.O0 == 16 and b3.O1 == 724


def test_shapes_and_bounds():
    for cfg, n in ((1, 50), (2, 1000), (4, 5000), (5, 200000)):
        b = W.config(cfg, instances=2)
        assert b.num_requests == 2 * n
        assert (b.prompt >= 1).all() and (b.output >= 1).all()
        for i in range(2):
            a = b.instance(i)["arrival"]
            assert (np.diff(a) >= 0).all()
        assert int((b.prompt.astype(np.int64) + b.output).max()) <= b.M


def test_burst_config_statistics():
    b = W.config(1)
    assert (b.arrival == 0).all()
    assert b.prompt.min() == 1 and b.prompt.max() == 32
    assert b.output.min() == 1 and b.output.max() == 64
    assert abs(b.prompt.mean() - 16.5) < 0.5 and abs(b.output.mean() - 32.5) < 1.0


def test_onebit_flip_rate_and_long_fraction():
    b = W.config(3, instances=64)
    truth = b.output > 256
    flip = truth ^ (b.long_bit == 1)
    n = b.num_requests
    assert abs(flip.mean() - 0.1) < 4 * np.sqrt(0.09 / n)
    assert abs(truth.mean() - 0.479) < 0.01


def test_heavy_traffic_mixture_and_rate():
    b = W.config(4, instances=8)
    short = b.output <= 128
    n = b.num_requests
    assert abs(short.mean() - 0.7) < 4 * np.sqrt(0.21 / n)
    assert abs(b.output.mean() - 818.4) < 25
    rate = []
    for i in range(8):
        a = b.instance(i)["arrival"]
        rate.append(len(a) / (a[-1] + 1))
    assert abs(np.mean(rate) - 512 / 818.4) < 0.02


def test_large_queue_mean_volume():
    """Appendix F, Lemma 2: E[vol] = E[s]/mu + 1/mu^2 = 979,400 for the large-
    queue configuration (s uniform on 1..4096, o geometric with mu = 1/400)."""
    b = W.config(5, instances=2)
    s = b.prompt.astype(np.float64)
    o = b.output.astype(np.float64)
    vol = s * o + (o * o + o) / 2
    n = len(vol)
    se = vol.std() / np.sqrt(n)
    assert abs(vol.mean() - 979400.0) < 4 * se
    a = b.instance(0)["arrival"]
    assert np.array_equal(np.unique(a), 500 * np.arange(10))
    assert (np.bincount(a // 500) == 20000).all()


def test_poisson_rate_config2():
    b = W.config(2, instances=16)
    r = [len(b.instance(i)["arrival"]) / (b.instance(i)["arrival"][-1] + 1) for i in range(16)]
    assert abs(np.mean(r) - 2.0) < 0.05


def test_default_step_budget_covers_the_horizon():
    b = W.config(2, instances=4)
    for i in range(4):
        d = b.instance(i)
        assert b.max_steps >= int(d["arrival"].max()) + int(d["output"].astype(np.int64).sum())
    b3 = W.config(3, instances=2)
    assert b3.max_steps > 60 * int(b3.output.astype(np.int64).sum() / 2)


def test_random_small_is_ragged_and_feasible():
    b = W.random_small(1, instances=20, n_max=9, s_max=5, o_max=7, M=12, gap_mean=0.5, bits=True)
    sizes = np.diff(b.offsets)
    assert sizes[0] == 0 and sizes[1] == 1
    assert int((b.prompt + np.maximum(b.output, max(b.O0, b.O1))).max()) <= b.M


def test_predictor_plans_are_feasible_seeded_and_unbiased_in_log():
    b = W.config(2, instances=40, n=500)
    for sigma in (0.25, 0.8):
        p = W.with_predictor(b, sigma)
        cap = np.minimum(W.CONFIGS[2]["o_cap"], b.M - b.prompt.astype(np.int64))
        assert (p.plan_len >= 1).all() and (p.plan_len <= cap).all()
        assert np.array_equal(p.output, b.output) and p.plan_len.dtype == np.int32
        # the same instances drawn on their own get the same predictions
        q = W.with_predictor(W.config(2, instances=[5, 17], n=500), sigma)
        assert np.array_equal(q.plan_len, p.subset([5, 17]).plan_len)
        assert np.array_equal(p.subset([5, 17]).plan_len,
                              W.with_predictor(b.subset([5, 17]), sigma).plan_len)
        # log-ratio: centred, spread close to sigma (requests away from the clips)
        o = b.output.astype(np.float64)
        mid = (o >= 20) & (o * np.exp(3 * sigma) < cap)
        lr = np.log(p.plan_len[mid] / o[mid])
        assert abs(float(np.median(lr))) < 0.05
        assert abs(float(lr.std()) - sigma) < 0.1 * sigma
        assert p.max_steps == 64 * b.max_steps  # room for lost progress
