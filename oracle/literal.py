"""Literal pure-Python simulator of the scheduling model (small instances only).

TEST INFRASTRUCTURE.  Only the test suite may import this module.

This is the most direct transcription of the model that the tests hold the C
oracle to.  It differs from the C oracle on purpose in two places: the
forward-looking memory check evaluates the memory at *every* future step tau up
to the last planned finish (the definition, constraint eq:c2 of Section 3.1,
applied to every future step), and the waiting set is ordered with Python tuple
comparison on (key, arrival, index) rather than a hand-written comparator.

Semantics (same step order as the C oracle; readings of the paper are listed in
the design notes):
  1. arrivals a_i = t enter W;
  2. completions t - k_i = o_i leave A;
  3. while the true memory at t+1 exceeds M: evict the largest believed
     remaining volume (latest arrival on ties), eligible again at t+1;
  4. strict head-of-line admission with the forward-looking check (or, for a
     policy name ending in "+cur", the current-capacity rule of Alg. 1 read
     literally: the next step's memory including the candidate stays <= M);
  5. request_steps += |A|; peak = max(peak, memory at t+1); t += 1.
"""

from typing import Dict, Optional

POLICIES = {"fcfs": 0, "sjf": 1, "svf": 2, "svf1bit": 3}


def volume(s: int, o: int) -> int:
    """Section 2.2, Eq. 1, written as the sum it measures: the memory held at
    each of the o decode steps, s + 1, s + 2, ..., s + o."""
    return sum(s + x for x in range(1, o + 1))


def key_of(policy: str, a: int, s: int, ohat: int) -> int:
    if policy == "fcfs":
        return a
    if policy == "sjf":
        return ohat
    return volume(s, ohat)   # "svf" and "svf1bit" (Eq. 2 with ohat = O_b)


def simulate(arrival, prompt, output, M: int, policy: str, plan=None, long_bit=None,
             O0: int = 0, O1: int = 0, max_steps: int = 10 ** 9,
             t_stop: int = 10 ** 18) -> Dict:
    current_rule = policy.endswith("+cur")
    policy = policy[:-4] if current_rule else policy
    n = len(arrival)
    a = [int(x) for x in arrival]
    s = [int(x) for x in prompt]
    o = [int(x) for x in output]
    if policy == "svf1bit":
        oh = [O1 if int(b) else O0 for b in long_bit]
    elif plan is not None:
        oh = [int(x) for x in plan]
    else:
        oh = list(o)
    key = [(key_of(policy, a[i], s[i], oh[i]), a[i], i) for i in range(n)]

    start = [-1] * n
    finish = [-1] * n
    pre = [0] * n
    seqno = [-1] * n
    k = [None] * n
    W = set()
    A = set()
    t = 0
    cursor = 0
    seq = 0
    nfin = 0
    peak = 0
    req_steps = 0

    def planned_finish(i, t):
        return k[i] + max(oh[i], t - k[i] + 1)

    def mem_at(tau, members, t):
        total = 0
        for i in members:
            if k[i] < tau <= planned_finish(i, t):
                total += s[i] + tau - k[i]
        return total

    while True:
        if nfin == n:
            status = 0
            break
        if t > max_steps:
            status = 1
            break
        if t >= t_stop:
            status = 2
            break
        while cursor < n and a[cursor] == t:
            W.add(cursor)
            cursor += 1
        for i in sorted(A):
            if t - k[i] == o[i]:
                A.discard(i)
                finish[i] = t
                nfin += 1
        evicted = []
        while sum(s[i] + t + 1 - k[i] for i in A) > M:
            def remaining(i):
                e = t - k[i]
                L = max(oh[i], e + 1)
                return sum(s[i] + x for x in range(e + 1, L + 1))
            v = max(A, key=lambda i: (remaining(i), a[i], i))
            A.discard(v)
            pre[v] += 1
            k[v] = None
            start[v] = -1
            seqno[v] = -1
            evicted.append(v)
        while W:
            h = min(W, key=lambda i: key[i])
            k[h] = t          # tentatively started at t
            members = A | {h}
            if current_rule:
                ok = sum(s[i] + t + 1 - k[i] for i in members) <= M
            else:
                horizon = max(planned_finish(i, t) for i in members)
                ok = all(mem_at(tau, members, t) <= M for tau in range(t + 1, horizon + 1))
            if not ok:
                k[h] = None
                break
            start[h] = t
            seqno[h] = seq
            seq += 1
            W.discard(h)
            A.add(h)
        W.update(evicted)
        req_steps += len(A)
        peak = max(peak, sum(s[i] + t + 1 - k[i] for i in A))
        t += 1

    fin = [f for f in finish if f >= 0]
    return {
        "start": start, "finish": finish, "preempt": pre, "admit_seq": seqno,
        "makespan": max(fin) if fin else 0, "status": status,
        "sum_latency": sum(finish[i] - a[i] for i in range(n) if finish[i] >= 0),
        "request_steps": req_steps, "peak_mem": peak, "preemptions": sum(pre),
        "t_end": t, "n_finished": len(fin),
    }
