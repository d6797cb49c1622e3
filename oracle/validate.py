"""Output-only schedule validator: no simulator inside.

TEST INFRASTRUCTURE.  Only the test suite may import this module.

Given one instance (a, s, o, believed lengths o^, policy) and a schedule
(start, admit_seq), it checks, for runs without preemption:

  V1  start_i >= a_i and finish_i = start_i + o_i              (eq:obj)
  V2  the true memory sum_{i: k_i < tau <= k_i+o_i} (s_i+tau-k_i) <= M at every
      step tau (constraint eq:c2 of Section 3.1)
  V3  strict head of line: the requests started at step t are exactly the
      first ones, in priority order, of those waiting at t, and they were
      admitted in that order (Alg. 1, Process 2 pops the head while it fits)
  V4  maximality: after the admissions of step t, the highest-priority request
      still waiting would break the forward-looking check (some future step
      over M, Appendix E.2 proof of the waiting-time lemma)
  V5  every admission passed the forward-looking check against the requests
      running at that moment (with the lengths the scheduler believed)

With rule="current" (Alg. 1's Process 2 read literally) V4 and V5 use the
memory of the next step only, including the candidate's first token.

With V1-V5 the admissions at every step are the longest feasible prefix of the
waiting requests in priority order, so by induction over t they fix the whole
schedule: a simulator that passes the validator on an instance has produced
the one schedule the model allows.  The priority order is computed here from
the volume written as the sum it measures (s+1) + ... + (s+o), not from the
closed form.

The validator also recomputes the run's statistics from the schedule alone
(makespan, latency sum, request-steps, peak memory).
"""

from typing import Dict, Optional

import numpy as np


def _volume_sum(s, o):
    # sum_{x=1..o} (s + x), vectorised as an explicit cumulative sum per row
    return np.array([int(np.arange(sv + 1, sv + ov + 1, dtype=np.int64).sum())
                     for sv, ov in zip(s.tolist(), o.tolist())], dtype=np.int64)


def priority_order(policy: str, a, s, ohat) -> np.ndarray:
    """Indices sorted by (key, arrival, index)."""
    a = np.asarray(a, dtype=np.int64)
    if policy == "fcfs":
        key = a.copy()
    elif policy == "sjf":
        key = np.asarray(ohat, dtype=np.int64)
    else:
        key = _volume_sum(np.asarray(s, dtype=np.int64), np.asarray(ohat, dtype=np.int64))
    idx = np.arange(len(a))
    return np.lexsort((idx, a, key))


def true_profile(s, o, start, horizon):
    """mem[tau] for tau in [0, horizon]; a request started at k adds s+tau-k
    for tau in [k+1, k+o].  Built with two difference arrays (slope and
    intercept), independently of any simulator."""
    s = np.asarray(s, dtype=np.int64)
    o = np.asarray(o, dtype=np.int64)
    k = np.asarray(start, dtype=np.int64)
    keep = k >= 0
    s, o, k = s[keep], o[keep], k[keep]
    lo = k + 1
    hi = np.minimum(k + o, horizon)
    keep = lo <= hi
    s, k, lo, hi = s[keep], k[keep], lo[keep], hi[keep]
    slope = np.zeros(horizon + 2, dtype=np.int64)
    icpt = np.zeros(horizon + 2, dtype=np.int64)
    np.add.at(slope, lo, 1)
    np.add.at(slope, hi + 1, -1)
    np.add.at(icpt, lo, s - k)
    np.add.at(icpt, hi + 1, -(s - k))
    tau = np.arange(horizon + 2, dtype=np.int64)
    return (np.cumsum(slope) * tau + np.cumsum(icpt))[: horizon + 1]


def _planned_ok(t, cand_s, cand_oh, members, s, oh, k, M):
    """Forward-looking check of a candidate started at t against ``members``
    (indices with start k <= t that are running at t), literal over every
    future step up to the last planned finish."""
    if members.size:
        L = np.maximum(oh[members], t - k[members] + 1)
        F = k[members] + L
        horizon = max(int(F.max()), t + cand_oh)
    else:
        horizon = t + cand_oh
    taus = np.arange(t + 1, horizon + 1, dtype=np.int64)
    mem = np.where(taus <= t + cand_oh, cand_s + taus - t, 0)
    for j, Fj in zip(members.tolist(), (F.tolist() if members.size else [])):
        mem = mem + np.where(taus <= Fj, s[j] + taus - k[j], 0)
    return bool((mem <= M).all())


def _current_ok(t, cand_s, members, s, k, M):
    """Next-step memory of the running requests plus the candidate's s + 1."""
    return int((s[members] + t + 1 - k[members]).sum()) + cand_s + 1 <= M


def validate(a, s, o, start, admit_seq, M: int, policy: str, ohat=None,
             finish=None, rule: str = "lookahead") -> Dict:
    """Raise AssertionError on the first violated condition; return the
    statistics recomputed from the schedule."""
    a = np.asarray(a, dtype=np.int64)
    s = np.asarray(s, dtype=np.int64)
    o = np.asarray(o, dtype=np.int64)
    k = np.asarray(start, dtype=np.int64)
    seq = np.asarray(admit_seq, dtype=np.int64)
    oh = o.copy() if ohat is None else np.asarray(ohat, dtype=np.int64)
    n = len(a)
    if n == 0:
        return {"makespan": 0, "sum_latency": 0, "request_steps": 0, "peak_mem": 0}
    assert (k >= 0).all(), "every request must have started"
    # V1
    assert (k >= a).all(), "V1: a request started before it arrived"
    fin = k + o
    if finish is not None:
        assert (np.asarray(finish, dtype=np.int64) == fin).all(), "V1: finish != start + o"
    horizon = int(fin.max()) + 1
    # V2
    prof = true_profile(s, o, k, horizon)
    assert int(prof.max()) <= M, f"V2: memory {int(prof.max())} > M={M} at step {int(prof.argmax())}"
    # admission order must follow start time
    by_seq = np.argsort(seq, kind="stable")
    assert (np.diff(k[by_seq]) >= 0).all(), "admit_seq is not ordered by start"
    assert sorted(seq.tolist()) == list(range(n)), "admit_seq is not a permutation"
    order = priority_order(policy, a, s, oh)
    rank = np.empty(n, dtype=np.int64)
    rank[order] = np.arange(n)
    # V3-V5, step by step over every step where something waits or starts
    t_last = int(k.max())
    for t in range(0, t_last + 1):
        waiting = np.nonzero((a <= t) & (k >= t))[0]
        if waiting.size == 0:
            continue
        w_sorted = waiting[np.argsort(rank[waiting])]
        adm = np.nonzero(k == t)[0]
        adm_sorted = adm[np.argsort(seq[adm])]
        # V3: a prefix of the waiting requests, admitted in priority order
        assert np.array_equal(adm_sorted, w_sorted[: adm.size]), \
            f"V3: step {t}: admitted {adm_sorted.tolist()} is not the head of {w_sorted[:adm.size + 3].tolist()}"
        running = np.nonzero((k < t) & (fin > t))[0]
        members = running
        # V5: each admission fitted against what ran at that moment
        def fits(j, members):
            if rule == "current":
                return _current_ok(t, s[j], members, s, k, M)
            return _planned_ok(t, s[j], oh[j], members, s, oh, k, M)
        for j in adm_sorted.tolist():
            assert fits(j, members), \
                f"V5: step {t}: request {j} was admitted although it did not fit"
            members = np.append(members, j)
        # V4: the next request in line did not fit
        if adm.size < waiting.size:
            h = int(w_sorted[adm.size])
            assert not fits(h, members), \
                f"V4: step {t}: request {h} fitted but was not admitted"
    return {"makespan": int(fin.max()), "sum_latency": int((fin - a).sum()),
            "request_steps": int(o.sum()), "peak_mem": int(prof.max())}
