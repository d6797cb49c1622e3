"""Seeded synthetic workloads for the batched scheduling simulator.

This module only draws integers.  It holds none of the scheduling arithmetic
(no keys, no volumes, no feasibility test), so that both the GPU path and the
CPU oracle can consume exactly the same arrays without sharing any of the
method's code.

Every instance draws from its own numpy PCG64 stream seeded with
``SeedSequence([2606, 22327, cfg, instance])``, so any subset of instances of a
configuration can be regenerated on its own, bit for bit.

The five configurations stand in for the paper's serving workloads (the paper
samples 2,000 LMSYS-Chat / LongBench requests with a 65,536-token context and a
4,096-token generation cap, burst or Poisson arrivals; Section 4.1).  No item of
those datasets is used or reproduced here; lengths come from the parametric
distributions below.

Request layout (structure of arrays, CSR over instances):
  offsets[i] .. offsets[i+1]  -> the requests of instance i
  arrival  a  int32, nondecreasing inside an instance (requests are indexed in
              arrival order)
  prompt   s  int32 >= 1
  output   o  int32 >= 1   (true output length)
  long_bit b  int8 in {0,1} (only for the 1-bit policy; the scheduler's view)
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

SEED_ROOT = (2606, 22327)

POLICY_NAMES = ("fcfs", "sjf", "svf", "svf1bit")


@dataclass
class Batch:
    """A batch of independent instances sharing one KV budget ``M``."""

    name: str
    offsets: np.ndarray            # int64 [I+1]
    arrival: np.ndarray            # int32 [N]
    prompt: np.ndarray             # int32 [N]
    output: np.ndarray             # int32 [N]
    M: int
    policies: tuple                # policy names, run side by side
    long_bit: Optional[np.ndarray] = None   # int8 [N] or None
    plan_len: Optional[np.ndarray] = None   # int32 [N] or None (None: plan = output)
    O0: int = 0
    O1: int = 0
    max_steps: int = 0
    meta: Dict = field(default_factory=dict)

    @property
    def num_instances(self) -> int:
        return int(self.offsets.shape[0] - 1)

    @property
    def num_requests(self) -> int:
        return int(self.offsets[-1])

    def instance(self, i: int) -> Dict[str, np.ndarray]:
        lo, hi = int(self.offsets[i]), int(self.offsets[i + 1])
        d = {"arrival": self.arrival[lo:hi], "prompt": self.prompt[lo:hi],
             "output": self.output[lo:hi]}
        d["long_bit"] = None if self.long_bit is None else self.long_bit[lo:hi]
        d["plan_len"] = None if self.plan_len is None else self.plan_len[lo:hi]
        return d

    def subset(self, ids: Sequence[int]) -> "Batch":
        """The same batch restricted to the listed instances (order kept)."""
        parts = [self.instance(int(i)) for i in ids]
        return assemble(self.name + "[sub]", parts, self.M, self.policies,
                        O0=self.O0, O1=self.O1, max_steps=self.max_steps,
                        meta=self._subset_meta(ids))

    def _subset_meta(self, ids: Sequence[int]) -> Dict:
        meta = dict(self.meta, subset=list(map(int, ids)))
        if "instance_ids" in meta:
            meta["instance_ids"] = np.asarray(meta["instance_ids"])[np.asarray(ids, dtype=np.int64)]
        return meta


def _rng(cfg: int, inst: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([SEED_ROOT[0], SEED_ROOT[1], int(cfg), int(inst)])))


def _uniform(rng, lo, hi, n):
    """Uniform integers on {lo, ..., hi} (both ends included)."""
    return rng.integers(lo, hi + 1, size=n, dtype=np.int64)


def _lognormal_clipped(rng, mu, sigma, lo, hi, n):
    # clip(rint(exp(N(mu, sigma))), lo, hi); rint rounds half to even.
    x = np.exp(rng.normal(mu, sigma, size=n))
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def _poisson_arrivals(rng, mean_gap, n):
    # A continuous Poisson process read off at integer steps: a_i = floor of
    # the i-th event time.  Rounding each gap instead would raise the rate.
    g = rng.exponential(mean_gap, size=n)
    return np.floor(np.cumsum(g)).astype(np.int64)


def assemble(name, parts: List[Dict[str, np.ndarray]], M, policies, O0=0, O1=0,
             max_steps=0, meta=None) -> Batch:
    """Concatenate per-instance dicts into one CSR batch."""
    sizes = [len(p["arrival"]) for p in parts]
    offsets = np.zeros(len(parts) + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(sizes, dtype=np.int64)

    def cat(key, dtype):
        if not parts or sum(sizes) == 0:
            return np.zeros(0, dtype=dtype)
        return np.ascontiguousarray(np.concatenate(
            [np.asarray(p[key]).astype(dtype, copy=False) for p in parts]))

    a = cat("arrival", np.int32)
    s = cat("prompt", np.int32)
    o = cat("output", np.int32)
    bit = None
    if parts and all(p.get("long_bit") is not None for p in parts):
        bit = cat("long_bit", np.int8)
    plan = None
    if parts and all(p.get("plan_len") is not None for p in parts):
        plan = cat("plan_len", np.int32)
    b = Batch(name=name, offsets=offsets, arrival=a, prompt=s, output=o, M=int(M),
              policies=tuple(policies), long_bit=bit, plan_len=plan, O0=int(O0),
              O1=int(O1), meta=dict(meta or {}))
    b.max_steps = int(max_steps) if max_steps else default_max_steps(b)
    return b


def default_max_steps(b: Batch) -> int:
    """A step budget that a run with known lengths can never exhaust.

    With plan == true length, every step either advances an active request or
    waits for an arrival, so the last finish is at most max(a) + sum(o).  When
    the scheduler plans with other lengths (1-bit policy, predictor noise), or
    admits on the next step's memory only, preemption can waste steps, so the
    budget is widened 64 times.
    """
    worst = 1
    for i in range(b.num_instances):
        lo, hi = int(b.offsets[i]), int(b.offsets[i + 1])
        if hi > lo:
            w = int(b.arrival[lo:hi].max()) + int(b.output[lo:hi].astype(np.int64).sum())
            worst = max(worst, w)
    worst += 1
    planned_differently = any(p.startswith("svf1bit") or p.endswith("+cur")
                              for p in b.policies) or (b.plan_len is not None)
    return worst * 64 if planned_differently else worst


# --------------------------------------------------------------------------
# The configurations
# --------------------------------------------------------------------------

def gen_instance(cfg: int, inst: int, n: Optional[int] = None,
                 burst: int = 20000) -> Dict[str, np.ndarray]:
    """Draw one instance of configuration ``cfg`` (per-instance stream).
    ``burst`` only applies to the large-queue configuration (reduced copies
    for tests keep its burst structure with fewer requests per burst)."""
    rng = _rng(cfg if cfg != 3 else 2, inst)
    if cfg == 1:
        # Offline burst, known outputs: 50 requests at t = 0.
        n = 50 if n is None else n
        a = np.zeros(n, dtype=np.int64)
        s = _uniform(rng, 1, 32, n)
        o = _uniform(rng, 1, 64, n)
        return {"arrival": a, "prompt": s, "output": o}
    if cfg in (2, 3):
        # Online Poisson arrivals, two per step on average; lognormal lengths.
        n = 1000 if n is None else n
        a = _poisson_arrivals(rng, 0.5, n)
        s = _lognormal_clipped(rng, 5.3, 0.8, 1, 2048, n)
        o = _lognormal_clipped(rng, 5.5, 0.9, 1, 2048, n)
        d = {"arrival": a, "prompt": s, "output": o}
        if cfg == 3:
            # The scheduler sees only b = [o > 256], flipped with probability 0.1
            # by an independent per-instance stream.
            r3 = _rng(3, inst)
            flip = r3.random(n) < 0.1
            d["long_bit"] = ((o > 256) ^ flip).astype(np.int8)
        return d
    if cfg == 4:
        # Heavy traffic: arrival rate 512 / E[o] (E[o] = 818.4), bimodal outputs.
        n = 5000 if n is None else n
        lam = 512.0 / 818.4
        a = _poisson_arrivals(rng, 1.0 / lam, n)
        s = _uniform(rng, 64, 1024, n)
        short = rng.random(n) < 0.7
        o_short = _uniform(rng, 16, 128, n)
        o_long = _uniform(rng, 1024, 4096, n)
        o = np.where(short, o_short, o_long)
        return {"arrival": a, "prompt": s, "output": o}
    if cfg == 5:
        # Large queues: bursts of 20,000 arrivals every 500 steps.
        n = 200000 if n is None else n
        a = 500 * (np.arange(n, dtype=np.int64) // burst)
        s = _uniform(rng, 1, 4096, n)
        o = np.clip(rng.geometric(1.0 / 400.0, size=n), 1, 8192).astype(np.int64)
        return {"arrival": a, "prompt": s, "output": o}
    if cfg == 0:
        # Tiny burst instances for exhaustive optimal schedules.
        n = int(_uniform(rng, 2, 8, 1)[0]) if n is None else n
        a = np.zeros(n, dtype=np.int64)
        s = _uniform(rng, 1, 4, n)
        o = _uniform(rng, 1, 4, n)
        pmax = int((s + o).max())
        M = pmax + int(_uniform(rng, 0, 2 * pmax, 1)[0])
        return {"arrival": a, "prompt": s, "output": o, "M": M}
    raise ValueError(f"unknown configuration {cfg}")


# o_cap: the generation cap of each workload (largest output length it draws);
# a length predictor answers inside it.
CONFIGS = {
    1: dict(instances=256, M=512, policies=("svf", "sjf", "fcfs"), o_cap=64),
    2: dict(instances=4096, M=65536, policies=("svf", "sjf", "fcfs"), o_cap=2048),
    3: dict(instances=4096, M=65536, policies=("svf1bit", "svf", "sjf", "fcfs"),
            O0=16, O1=724, o_cap=2048),
    4: dict(instances=16384, M=262144, policies=("svf",), o_cap=4096),
    5: dict(instances=64, M=2 ** 21, policies=("svf",), o_cap=8192),
}

CONFIG_TITLES = {
    1: "offline burst, 256 x 50, M=512",
    2: "online Poisson, 4096 x 1000, M=65536, SVF/SJF/FCFS",
    3: "1-bit SVF with noisy bit, 4096 x 1000, M=65536",
    4: "heavy traffic, 16384 x 5000, M=262144, SVF",
    5: "large queues, 64 x 200000 in bursts of 20000, M=2^21, SVF",
}


def config(cfg: int, instances=None, n: Optional[int] = None,
           policies: Optional[Sequence[str]] = None, burst: int = 20000) -> Batch:
    """Build configuration ``cfg``.

    ``instances``: None for the full count, an int for the first k instances,
    or an explicit list of instance ids (each drawn from its own stream, so a
    sample of a full-size configuration is identical to the same instances of
    the full batch).  ``n`` overrides the per-instance request count (smaller
    cases for the oracle).
    """
    spec = CONFIGS[cfg]
    if instances is None:
        ids = range(spec["instances"])
    elif isinstance(instances, int):
        ids = range(instances)
    else:
        ids = list(instances)
    parts = [gen_instance(cfg, int(i), n, burst) for i in ids]
    b = assemble(f"cfg{cfg}", parts, spec["M"], tuple(policies or spec["policies"]),
                 O0=spec.get("O0", 0), O1=spec.get("O1", 0),
                 meta={"cfg": cfg, "ids": list(map(int, ids)) if not isinstance(ids, range)
                       else [ids.start, ids.stop], "n": n,
                       "instance_ids": np.asarray(list(ids), dtype=np.int64)})
    return b


def with_predictor(b: Batch, sigma: float) -> Batch:
    """The same batch planned with predicted output lengths (a stand-in for the
    paper's length regressor, Alg. 1's Process 1): o^ = rint(o * e^Z),
    Z ~ Normal(0, sigma), clipped to [1, generation cap] and to M - s so that
    every request stays feasible.  Each instance draws from its own stream
    (its configuration stream with one more word), so samples of a
    configuration get the same predictions as the full batch."""
    cfg = int(b.meta["cfg"])
    ids = b.meta["instance_ids"]
    cap = CONFIGS[cfg]["o_cap"]
    plan = np.empty(b.num_requests, dtype=np.int32)
    for j in range(b.num_instances):
        lo, hi = int(b.offsets[j]), int(b.offsets[j + 1])
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([SEED_ROOT[0], SEED_ROOT[1], cfg, int(ids[j]), 1])))
        o = b.output[lo:hi].astype(np.float64)
        z = rng.normal(0.0, sigma, hi - lo)
        hi_cap = np.minimum(cap, b.M - b.prompt[lo:hi].astype(np.int64))
        plan[lo:hi] = np.clip(np.rint(o * np.exp(z)), 1, hi_cap)
    out = Batch(b.name + f"+pred{sigma:g}", b.offsets, b.arrival, b.prompt, b.output, b.M,
                b.policies, long_bit=b.long_bit, plan_len=plan, O0=b.O0, O1=b.O1,
                meta=dict(b.meta, predictor_sigma=float(sigma)))
    out.max_steps = default_max_steps(out)
    return out


def poisson_geometric(lam: float, mu: float, s_max: int, o_cap: int, M: int, n: int,
                      instances: int, tag: int = 0, policies=("svf",), theta: int = 0,
                      O0: int = 0, O1: int = 0, first: int = 0) -> Batch:
    """The stochastic model of the Poisson-arrival theorems (Section 3.3):
    arrivals of rate ``lam`` per step (continuous Poisson process read off at
    integer steps), prompts uniform on {1..s_max}, outputs Geometric(mu) on
    {1, 2, ...} clipped at ``o_cap`` (so s + o <= s_max + o_cap; the clipped
    mass is (1 - mu)^o_cap).  ``theta`` > 0 adds the exact 1-bit labels
    b = [o > theta] with proxies O0, O1 given by the caller.  Instance i draws
    from its own stream (``tag`` separates parameter sets)."""
    parts = []
    for i in range(first, first + instances):
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([SEED_ROOT[0], SEED_ROOT[1], 6, int(tag), int(i)])))
        a = _poisson_arrivals(rng, 1.0 / lam, n)
        s_ = _uniform(rng, 1, s_max, n)
        o = np.minimum(rng.geometric(mu, size=n), o_cap).astype(np.int64)
        d = {"arrival": a, "prompt": s_, "output": o}
        if theta > 0:
            d["long_bit"] = (o > theta).astype(np.int8)
        parts.append(d)
    return assemble(f"poisson-geo{tag}", parts, M, tuple(policies), O0=O0, O1=O1,
                    meta={"lam": lam, "mu": mu, "s_max": s_max, "o_cap": o_cap,
                          "theta": theta, "tag": tag, "first": first})


def tiny_cr_instances(count: int, start: int = 0) -> List[Dict]:
    """Configuration 0: tiny burst instances with their own budgets."""
    return [gen_instance(0, i) for i in range(start, start + count)]


def tiny_alpha_instances(k: int, count: int, n_lo: int, n_hi: int, s_max: int, o_max: int,
                         tag: int = 0) -> Batch:
    """Burst instances for a competitive-ratio sweep at alpha = 1/k: n drawn
    from {n_lo..n_hi}, s from {1..s_max}, o from {1..o_max}; request 0 is the
    largest possible one (s_max, o_max), and every instance shares the budget
    M = k (s_max + o_max), so max_i (s_i + o_i) / M = 1/k exactly."""
    parts = []
    for i in range(count):
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([SEED_ROOT[0], SEED_ROOT[1], 7, int(k), int(tag), int(i)])))
        n = int(_uniform(rng, n_lo, n_hi, 1)[0])
        s_ = _uniform(rng, 1, s_max, n)
        o = _uniform(rng, 1, o_max, n)
        s_[0], o[0] = s_max, o_max
        parts.append({"arrival": np.zeros(n, dtype=np.int64), "prompt": s_, "output": o})
    return assemble(f"alpha1/{k}", parts, k * (s_max + o_max), ("svf", "sjf", "fcfs"),
                    meta={"k": k, "s_max": s_max, "o_max": o_max, "tag": tag})


def random_small(seed: int, instances: int, n_max: int, s_max: int, o_max: int,
                 M: int, gap_mean: float = 0.0, bits: bool = False,
                 plan_noise: bool = False, ragged: bool = True) -> Batch:
    """Small random batches for parity tests: ragged sizes (0 and 1 included),
    optional arrivals, optional 1-bit labels or noisy plan lengths.  Every
    request satisfies s + max(o, plan) <= M."""
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([SEED_ROOT[0], SEED_ROOT[1], 9000 + int(seed)])))
    parts = []
    for i in range(instances):
        if ragged:
            n = int(rng.integers(0, n_max + 1))
            if i == 0:
                n = 0
            elif i == 1:
                n = 1
        else:
            n = n_max
        if gap_mean > 0:
            a = _poisson_arrivals(rng, gap_mean, n)
        else:
            a = np.zeros(n, dtype=np.int64)
        o = _uniform(rng, 1, o_max, n)
        s = _uniform(rng, 1, s_max, n)
        d = {"arrival": a, "prompt": s, "output": o}
        if bits:
            d["long_bit"] = (rng.random(n) < 0.5).astype(np.int8)
        if plan_noise:
            d["plan_len"] = np.clip(np.rint(o * np.exp(rng.normal(0.0, 0.5, n))), 1, o_max).astype(np.int64)
        parts.append(d)
    pol = ("svf1bit", "svf", "sjf", "fcfs") if bits else ("svf", "sjf", "fcfs")
    return assemble(f"rand{seed}", parts, M, pol,
                    O0=max(1, o_max // 8) if bits else 0,
                    O1=max(1, (o_max * 3) // 4) if bits else 0)
