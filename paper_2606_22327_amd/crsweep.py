"""Competitive ratio against alpha on tiny burst instances.

Theorem thm:svf-burst bounds SVF's total latency under burst arrivals by
(1 + 2/(1 - alpha)) times the optimum, alpha = max_i (s_i + o_i) / M; Table
tab:alpha-cr lists the bound at alpha = 1/2, 1/4, 1/10, 1/20, 1/100.  This
module measures the ratio itself: many tiny burst instances (n <= 16) are
simulated on the GPU under SVF, SJF and FCFS in one batch per alpha, and their
exact optima come from the host solver of ``svfopt.h`` (branch and bound over
the integer program of Section 3.1).

Three modes:
  sweep   random instances at each alpha (``workloads.tiny_alpha_instances``);
  search  an evolutionary search for instances with a large SVF / OPT ratio:
          every generation mutates each member once, evaluates all children in
          one GPU batch and one threaded optimum pass, and keeps the worse
          (higher-ratio) of parent and child;
  bound   instances of hundreds to thousands of requests, too large for an
          exact optimum, measured against the lower bound of the optimum that
          the competitive-ratio proof uses (``opt_lower_bound``): TEL / LB is
          an upper estimate of TEL / OPT.  At small alpha a tiny instance fits
          in memory at once and every policy is optimal; these instances keep
          the memory contended at alpha = 1/10, 1/20, 1/100.

Run ``python -m paper_2606_22327_amd.crsweep`` (GPU).
"""

from __future__ import annotations

import argparse
import json
import sys
import time
from dataclasses import dataclass, field
from typing import Dict, List, Sequence

import numpy as np

POLICIES = ("svf", "sjf", "fcfs")


def cr_bound(alpha: float) -> float:
    """Theorem thm:svf-burst: 1 + 2 / (1 - alpha)."""
    return 1.0 + 2.0 / (1.0 - alpha)


@dataclass
class Result:
    k: int
    M: int
    alpha: float
    bound: float
    instances: int
    mean_ratio: Dict[str, float]
    max_ratio: Dict[str, float]
    worst: Dict[str, List[List[int]]] = field(default_factory=dict)
    gpu_ms: float = 0.0
    opt_s: float = 0.0
    states: int = 0


def evaluate(batch, threads: int = 0):
    """Total latency of every policy (GPU) and the optimum (host) per instance."""
    from . import svfsim as S

    sim = S.Simulator.from_batch(batch, POLICIES)
    try:
        sim.set_profiling(True)
        sim.reset()
        sim.run()
        stats = {p: sim.stats(j) for j, p in enumerate(POLICIES)}
        tel = {p: stats[p]["sum_latency"].astype(np.int64) for p in POLICIES}
        status = {p: stats[p]["status"] for p in POLICIES}
        gpu_ms = sim.timings()["sim_ms"]
    finally:
        sim.close()
    for p in POLICIES:
        if (status[p] != 0).any():
            raise RuntimeError(f"{p}: an instance did not finish")
    Ms = np.full(batch.num_instances, batch.M, dtype=np.int64)
    t0 = time.perf_counter()
    opt, states, st = S.opt_burst_batch(batch.offsets, batch.prompt, batch.output, Ms,
                                        threads=threads)
    opt_s = time.perf_counter() - t0
    if (st != 0).any():
        raise RuntimeError(f"optimum not found for {int((st != 0).sum())} instances")
    return tel, opt, gpu_ms, opt_s, int(states.sum())


def opt_lower_bound(prompt, output, M: int) -> int:
    """Lower bound on the optimal total latency of a burst instance: the
    larger of the area bound of Proposition prop:opt_lower_bound (the volumes
    of Eq. 1 in ascending order v_1 <= ... <= v_n; M * TEL(OPT) >=
    sum_j sum_{i <= j} v_i) and Lemma lemma:opt_lb_execution (a request
    cannot finish before o_i steps: TEL(OPT) >= sum_i o_i)."""
    s = np.asarray(prompt, dtype=np.int64)
    o = np.asarray(output, dtype=np.int64)
    v = np.sort(s * o + (o * o + o) // 2)
    n = len(v)
    # sum_j sum_{i <= j} v_i = sum_i v_i (n - i), i counted from 0
    area = int((v * (n - np.arange(n, dtype=np.int64))).sum())
    return max(-(-area // int(M)), int(o.sum()))


def simulate_tel(batch):
    """Total latency of every policy per instance (GPU)."""
    from . import svfsim as S

    sim = S.Simulator.from_batch(batch, POLICIES)
    try:
        sim.set_profiling(True)
        sim.reset()
        sim.run()
        stats = {p: sim.stats(j) for j, p in enumerate(POLICIES)}
        gpu_ms = sim.timings()["sim_ms"]
    finally:
        sim.close()
    for p in POLICIES:
        if (stats[p]["status"] != 0).any():
            raise RuntimeError(f"{p}: an instance did not finish")
    return {p: stats[p]["sum_latency"].astype(np.int64) for p in POLICIES}, gpu_ms


def bound_sweep(ks: Sequence[int], count: int, n: int, s_max: int = 32, o_max: int = 32,
                tag: int = 0) -> List[Result]:
    """Burst instances of n requests at alpha = 1/k (request 0 the largest,
    M = k (s_max + o_max)) under every policy on the GPU; the ratios are total
    latency over ``opt_lower_bound``."""
    from . import workloads as W

    out = []
    for k in ks:
        b = W.tiny_alpha_instances(k, count, n, n, s_max, o_max, tag=2000 + tag)
        tel, gpu_ms = simulate_tel(b)
        lb = np.array([opt_lower_bound(b.instance(i)["prompt"], b.instance(i)["output"], b.M)
                       for i in range(b.num_instances)], dtype=np.int64)
        out.append(_summarise(k, b, tel, lb, gpu_ms, 0.0, 0))
    return out


def _summarise(k, batch, tel, opt, gpu_ms, opt_s, states) -> Result:
    alpha = 1.0 / k
    ratios = {p: tel[p] / opt for p in POLICIES}
    worst = {}
    for p in POLICIES:
        i = int(np.argmax(ratios[p]))
        d = batch.instance(i)
        worst[p] = [d["prompt"].tolist(), d["output"].tolist()]
    return Result(k=k, M=int(batch.M), alpha=alpha, bound=cr_bound(alpha),
                  instances=batch.num_instances, mean_ratio={p: float(ratios[p].mean()) for p in POLICIES},
                  max_ratio={p: float(ratios[p].max()) for p in POLICIES}, worst=worst,
                  gpu_ms=gpu_ms, opt_s=opt_s, states=states)


def sweep(ks: Sequence[int], count: int, n_lo: int = 6, n_hi: int = 12, s_max: int = 4,
          o_max: int = 6, threads: int = 0, tag: int = 0) -> List[Result]:
    from . import workloads as W

    out = []
    for k in ks:
        b = W.tiny_alpha_instances(k, count, n_lo, n_hi, s_max, o_max, tag=tag)
        tel, opt, gpu_ms, opt_s, states = evaluate(b, threads)
        out.append(_summarise(k, b, tel, opt, gpu_ms, opt_s, states))
    return out


def _mutate(rng, s, o, s_max, o_max, n_lo, n_hi):
    s, o = s.copy(), o.copy()
    r = rng.random()
    n = len(s)
    if r < 0.15 and n < n_hi:
        s = np.append(s, rng.integers(1, s_max + 1))
        o = np.append(o, rng.integers(1, o_max + 1))
    elif r < 0.3 and n > max(n_lo, 2):
        j = int(rng.integers(1, n))
        s, o = np.delete(s, j), np.delete(o, j)
    else:
        j = int(rng.integers(1, n))     # request 0 stays the largest one
        if rng.random() < 0.5:
            s[j] = rng.integers(1, s_max + 1)
        else:
            o[j] = rng.integers(1, o_max + 1)
    return s, o


def search(k: int, population: int = 256, generations: int = 30, n_lo: int = 6,
           n_hi: int = 12, s_max: int = 4, o_max: int = 6, threads: int = 0, seed: int = 0,
           log=None) -> Result:
    """Evolutionary search for a large SVF / OPT ratio at alpha = 1/k."""
    from . import workloads as W

    rng = np.random.default_rng([2606, 22327, 8, k, seed])
    b = W.tiny_alpha_instances(k, population, n_lo, n_hi, s_max, o_max, tag=1000 + seed)
    pop = [(b.instance(i)["prompt"].astype(np.int64), b.instance(i)["output"].astype(np.int64))
           for i in range(b.num_instances)]
    tel, opt, gpu_ms, opt_s, states = evaluate(b, threads)
    score = tel["svf"] / opt
    total_gpu, total_opt, total_states = gpu_ms, opt_s, states
    for g in range(generations):
        kids = [_mutate(rng, s, o, s_max, o_max, n_lo, n_hi) for s, o in pop]
        kb = W.assemble("search", [{"arrival": np.zeros(len(s), dtype=np.int64), "prompt": s,
                                    "output": o} for s, o in kids], b.M, POLICIES)
        ktel, kopt, gms, osec, kst = evaluate(kb, threads)
        total_gpu += gms
        total_opt += osec
        total_states += kst
        kscore = ktel["svf"] / kopt
        for i in range(len(pop)):
            if kscore[i] >= score[i]:
                pop[i], score[i] = kids[i], kscore[i]
        if log:
            log(f"alpha 1/{k} generation {g + 1}: best SVF/OPT {score.max():.4f}, "
                f"mean {score.mean():.4f}")
    fb = W.assemble("final", [{"arrival": np.zeros(len(s), dtype=np.int64), "prompt": s,
                               "output": o} for s, o in pop], b.M, POLICIES)
    tel, opt, gms, osec, st = evaluate(fb, threads)
    res = _summarise(k, fb, tel, opt, total_gpu + gms, total_opt + osec, total_states + st)
    return res


def table(rows: Sequence[Result], title: str) -> str:
    lines = [title, "alpha    bound  instances  SVF mean/max     SJF mean/max     "
                    "FCFS mean/max    gpu_ms  opt_s"]
    for r in rows:
        cells = "  ".join(f"{r.mean_ratio[p]:.3f}/{r.max_ratio[p]:.3f}  " for p in POLICIES)
        lines.append(f"1/{r.k:<5d} {r.bound:6.3f} {r.instances:9d}  {cells} "
                     f"{r.gpu_ms:7.1f} {r.opt_s:6.1f}")
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--k", default="2,3,4,6,10,20,100", help="alpha = 1/k values")
    ap.add_argument("--count", type=int, default=4096)
    ap.add_argument("--n-max", type=int, default=12)
    ap.add_argument("--search-generations", type=int, default=30)
    ap.add_argument("--search-k", default="2,3,4,6",
                    help="alpha values searched (at larger k every tiny instance fits at once)")
    ap.add_argument("--population", type=int, default=512)
    ap.add_argument("--threads", type=int, default=0)
    ap.add_argument("--bound-n", type=int, default=2000,
                    help="requests per instance of the lower-bound mode (0: skip it)")
    ap.add_argument("--bound-count", type=int, default=256)
    ap.add_argument("--bound-k", default="2,4,10,20,100")
    ap.add_argument("--json", action="store_true")
    args = ap.parse_args(argv)
    ks = [int(x) for x in args.k.split(",")]

    def log(m):
        print(f"[crsweep] {m}", file=sys.stderr, flush=True)

    t0 = time.perf_counter()
    rows = sweep(ks, args.count, n_hi=args.n_max, threads=args.threads)
    log(f"sweep done in {time.perf_counter() - t0:.1f}s")
    brows = []
    if args.bound_n > 0:
        t0 = time.perf_counter()
        brows = bound_sweep([int(x) for x in args.bound_k.split(",")], args.bound_count,
                            args.bound_n)
        log(f"lower-bound sweep done in {time.perf_counter() - t0:.1f}s")
    found = []
    if args.search_generations > 0:
        for k in [int(x) for x in args.search_k.split(",")]:
            found.append(search(k, args.population, args.search_generations, n_hi=args.n_max,
                                threads=args.threads, log=log))
    if args.json:
        for r in rows + found:
            print(json.dumps(r.__dict__))
        for r in brows:
            print(json.dumps(dict(r.__dict__, mode="lower-bound", n=args.bound_n)))
    else:
        print(table(rows, f"random burst instances (n in 6..{args.n_max}, s <= 4, o <= 6)"))
        if brows:
            print(table(brows, f"n = {args.bound_n} requests, s and o <= 32: total latency over "
                               "the optimum's lower bound (an upper estimate of the ratio)"))
        if found:
            print(table(found, "after the evolutionary search for a large SVF / OPT ratio"))
            for r in found:
                print(f"alpha 1/{r.k}: worst SVF instance s={r.worst['svf'][0]} "
                      f"o={r.worst['svf'][1]} M={r.M}")


if __name__ == "__main__":
    main()
