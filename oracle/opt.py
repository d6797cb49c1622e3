"""Exhaustive optimal schedules for tiny burst instances.

TEST INFRASTRUCTURE.  Only the test suite may import this module.

Solves the integer program of Section 3.1 (objective eq:obj, one start per
request eq:c1, memory at every step eq:c2, binary starts eq:c3) exactly for
burst instances (every a_i = 0) by dynamic programming over the scheduler's
state: which requests have not started, and how far each running request has
got.  At every step any subset of the unstarted requests may start, as long as
the requests already started then fit under M at every future step; idling is
allowed whenever something runs (an empty system never idles, which can only
cost).  The total latency sum_i (k_i + o_i) is accumulated as one unit per
unfinished request per step.

Intended for n <= 8 with small s and o.
"""

from functools import lru_cache
from itertools import combinations
from typing import Sequence


def optimal_total_latency(s: Sequence[int], o: Sequence[int], M: int) -> int:
    s = tuple(int(x) for x in s)
    o = tuple(int(x) for x in o)
    n = len(s)
    assert all(si + oi <= M for si, oi in zip(s, o)), "a request can never fit"

    def fits(running):
        # running: tuple of (i, e) with e = steps already done at the current step
        # future step d >= 1 holds s_i + e + d for e + d <= o_i
        horizon = max((o[i] - e for i, e in running), default=0)
        for d in range(1, horizon + 1):
            tot = 0
            for i, e in running:
                if e + d <= o[i]:
                    tot += s[i] + e + d
            if tot > M:
                return False
        return True

    @lru_cache(maxsize=None)
    def best(unstarted: frozenset, running: tuple) -> int:
        if not unstarted and not running:
            return 0
        here = len(unstarted) + len(running)   # unfinished at this step
        pool = sorted(unstarted)
        result = None
        for r in range(0, len(pool) + 1):
            if r == 0 and not running:
                continue
            for S in combinations(pool, r):
                cand = running + tuple((i, 0) for i in S)
                if not fits(cand):
                    continue
                nxt = tuple(sorted((i, e + 1) for i, e in cand if e + 1 < o[i]))
                v = here + best(unstarted.difference(S), nxt)
                if result is None or v < result:
                    result = v
        assert result is not None
        return result

    return best(frozenset(range(n)), tuple())
