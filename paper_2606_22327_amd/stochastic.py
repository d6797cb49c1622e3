"""Steady-state check of the Poisson-arrival bounds on the GPU simulator.

Section 3.3 models arrivals as a Poisson process of rate lam and output
lengths as Geometric(mu) on {1, 2, ...} (mean 1/mu), with s + o <= alpha M.
With the worst-case utilisation rho = lam E[vol] / ((1 - alpha) M / 2) < 1,

  SVF     (thm:svf_poisson)      E[CR] <= 1 + 2 / ((1-alpha)(1-mu)(1-rho))
  1-bit   (thm:svf_1bit_poisson) E[CR] <= 1 + E[vol]/(E[vol]-eps) * the same

and, one step before OPT enters their proofs, the mean latency itself obeys

  E[latency] <= 1/mu + d * W_0 / ((1-alpha) M / 2 - lam E[vol]),
  W_0 = lam (E[s]/mu^2 + 2/mu^3)   (Lemma 2 of the stochastic appendix)

with d = 1 for SVF and E[vol] / (E[vol] - eps) for 1-bit SVF.  The 1-bit
variant uses the conditional means of the two classes as proxies,
O_0 = E[o | o <= theta] and O_1 = E[o | o > theta] = theta + 1/mu, and
eps = (theta q^theta / (1 - q^theta))^2 / 2 with q = 1 - mu.

This module draws such workloads (``workloads.poisson_geometric``), runs
them through the C ABI, and sets the measured mean latency (over requests
arriving in the middle 80 % of each instance, away from the empty start and
the drain) against these bounds.  OPT is not computed: E[o] is a lower bound
on OPT's mean latency, so mean latency / E[o] bounds the ratio from above.
The simulator admits integer proxies, so O_0 and O_1 are rounded.

Run ``python -m paper_2606_22327_amd.stochastic`` for the table (GPU).
"""

from __future__ import annotations

import argparse
import json
import math
import sys
import time
from dataclasses import dataclass, field
from typing import Dict, List, Sequence

import numpy as np


@dataclass
class Model:
    """Parameters of the stochastic model."""

    M: int = 65536
    mu: float = 1.0 / 200.0
    s_max: int = 512          # prompts uniform on {1..s_max}
    o_cap: int = 3000         # outputs clipped here (mass (1-mu)^o_cap)
    thetas: Sequence[int] = (200, 600)

    @property
    def mean_s(self) -> float:
        return (1 + self.s_max) / 2.0

    @property
    def alpha(self) -> float:
        return (self.s_max + self.o_cap) / self.M

    @property
    def rate_floor(self) -> float:
        """Lemma 1 of the stochastic appendix: (1 - alpha) M / 2."""
        return 0.5 * self.M * (1.0 - self.alpha)

    @property
    def mean_volume(self) -> float:
        """E[s o + (o^2 + o)/2] for independent s and o ~ Geometric(mu):
        E[s]/mu + (E[o^2] + E[o])/2 with E[o^2] = (2 - mu)/mu^2."""
        mu = self.mu
        return self.mean_s / mu + 0.5 * ((2.0 - mu) / mu ** 2 + 1.0 / mu)

    def lam_for(self, rho: float) -> float:
        return rho * self.rate_floor / self.mean_volume

    def w0(self, lam: float) -> float:
        mu = self.mu
        return lam * (self.mean_s / mu ** 2 + 2.0 / mu ** 3)

    def proxies(self, theta: int):
        """(O_0, O_1, eps) of the 1-bit variant for threshold theta."""
        q_t = (1.0 - self.mu) ** theta
        tail = theta * q_t / (1.0 - q_t)
        return 1.0 / self.mu - tail, theta + 1.0 / self.mu, 0.5 * tail * tail

    def distortion(self, theta: int) -> float:
        eps = self.proxies(theta)[2]
        return self.mean_volume / (self.mean_volume - eps)

    def latency_bound(self, rho: float, d: float = 1.0) -> float:
        lam = self.lam_for(rho)
        return 1.0 / self.mu + d * self.w0(lam) / (self.rate_floor - lam * self.mean_volume)

    def cr_bound(self, rho: float, d: float = 1.0) -> float:
        return 1.0 + d * 2.0 / ((1.0 - self.alpha) * (1.0 - self.mu) * (1.0 - rho))


@dataclass
class Row:
    rho: float
    policy: str
    theta: int
    mean_latency: float
    mean_wait: float
    mean_o: float
    ratio: float                 # mean latency / mean o (>= the CR against OPT)
    latency_bound: float         # nan when rho >= 1 (outside the theorems)
    cr_bound: float
    preemptions: int
    requests: int
    request_steps: int
    sim_ms: float
    extra: Dict = field(default_factory=dict)


def _middle(offsets: np.ndarray, lo_frac=0.1, hi_frac=0.9) -> np.ndarray:
    idx = []
    for i in range(len(offsets) - 1):
        a, b = int(offsets[i]), int(offsets[i + 1])
        n = b - a
        idx.append(np.arange(a + int(lo_frac * n), a + int(hi_frac * n)))
    return np.concatenate(idx) if idx else np.zeros(0, dtype=np.int64)


def run(model: Model, rhos: Sequence[float], instances: int, n: int,
        policies=("svf", "svf1bit", "sjf", "fcfs"), tag: int = 1,
        keep_outputs: bool = False) -> List[Row]:
    """Simulate every (rho, policy[, theta]) on the GPU and summarise."""
    from . import svfsim as S
    from . import workloads as W

    rows: List[Row] = []
    for ri, rho in enumerate(rhos):
        lam = model.lam_for(rho)
        runs = [(p, 0) for p in policies if p != "svf1bit"]
        if "svf1bit" in policies:
            runs += [("svf1bit", th) for th in model.thetas]
        for pol, th in runs:
            O0 = O1 = 0
            if th:
                p0, p1, _ = model.proxies(th)
                O0, O1 = max(1, int(round(p0))), int(round(p1))
            b = W.poisson_geometric(lam, model.mu, model.s_max, model.o_cap, model.M, n,
                                    instances, tag=tag * 100 + ri, policies=(pol,),
                                    theta=th, O0=O0, O1=O1)
            sim = S.Simulator.from_batch(b)
            try:
                sim.set_profiling(True)
                sim.reset()
                sim.run()
                out = sim.read(0)
                st = sim.stats(0)
                tm = sim.timings()
            finally:
                sim.close()
            mid = _middle(b.offsets)
            fin = out["finish"][mid].astype(np.int64)
            a = b.arrival[mid].astype(np.int64)
            o = b.output[mid].astype(np.int64)
            if (fin < 0).any():
                raise RuntimeError(f"rho {rho} {pol}: unfinished requests (step budget)")
            lat = fin - a
            d = model.distortion(th) if th else 1.0
            inside = rho < 1.0
            row = Row(rho=rho, policy=pol, theta=th, mean_latency=float(lat.mean()),
                      mean_wait=float((lat - o).mean()), mean_o=float(o.mean()),
                      ratio=float(lat.mean() / o.mean()),
                      latency_bound=model.latency_bound(rho, d) if inside else math.nan,
                      cr_bound=model.cr_bound(rho, d) if inside else math.nan,
                      preemptions=int(st["preemptions"].sum()), requests=int(mid.size),
                      request_steps=int(st["request_steps"].sum()), sim_ms=tm["sim_ms"],
                      extra={"O0": O0, "O1": O1, "lam": lam})
            if keep_outputs:
                row.extra["batch"] = b
                row.extra["out"] = out
                row.extra["stats"] = st
            rows.append(row)
    return rows


def table(rows: Sequence[Row]) -> str:
    head = ("rho  policy        mean_lat   E[o]  ratio  lat_bound  cr_bound  "
            "wait   preempt  req-steps/s")
    lines = [head]
    for r in rows:
        name = r.policy + (f"(th={r.theta})" if r.theta else "")
        rate = r.request_steps / (r.sim_ms / 1e3) if r.sim_ms > 0 else math.nan
        lines.append(f"{r.rho:4.2f} {name:14s} {r.mean_latency:8.1f} {r.mean_o:6.1f} "
                     f"{r.ratio:6.3f} {r.latency_bound:10.1f} {r.cr_bound:9.2f} "
                     f"{r.mean_wait:6.2f} {r.preemptions:8d} {rate:12.3e}")
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--instances", type=int, default=256)
    ap.add_argument("--n", type=int, default=20000, help="requests per instance")
    ap.add_argument("--rho", default="0.25,0.5,0.75,0.9,1.5,2.0,2.1")
    ap.add_argument("--mu", type=float, default=1.0 / 200.0)
    ap.add_argument("--M", type=int, default=65536)
    ap.add_argument("--json", action="store_true", help="one JSON object per row")
    args = ap.parse_args(argv)
    model = Model(M=args.M, mu=args.mu)
    rhos = [float(x) for x in args.rho.split(",")]
    t0 = time.perf_counter()
    rows = run(model, rhos, args.instances, args.n)
    print(f"model: M={model.M} mu={model.mu:g} s~U{{1..{model.s_max}}} o_cap={model.o_cap} "
          f"alpha={model.alpha:.4f} E[vol]={model.mean_volume:.1f} "
          f"(1-alpha)M/2={model.rate_floor:.1f}; {args.instances} instances x {args.n} "
          f"requests per setting; {time.perf_counter() - t0:.1f}s", file=sys.stderr)
    if args.json:
        for r in rows:
            d = {k: v for k, v in r.__dict__.items() if k != "extra"}
            d.update({k: v for k, v in r.extra.items() if k in ("O0", "O1", "lam")})
            print(json.dumps(d))
    else:
        print(table(rows))


if __name__ == "__main__":
    main()
