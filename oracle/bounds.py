"""Closed-form quantities from the paper, used as pins by the tests.

TEST INFRASTRUCTURE.  Only the test suite may import this module.
"""

import math
from typing import Sequence


def cr_bound(alpha: float) -> float:
    """Theorem thm:svf-burst: TEL(SVF)/TEL(OPT) <= 1 + 2/(1 - alpha),
    alpha = max_i (s_i + o_i) / M."""
    return 1.0 + 2.0 / (1.0 - alpha)


def cr_bound_holds(tel_svf: int, opt: int, M: int, pmax: int) -> bool:
    """The same inequality in exact integers:
    TEL * (M - P_max) <= (3M - P_max) * OPT."""
    return tel_svf * (M - pmax) <= (3 * M - pmax) * opt


def volume_closed(s: int, o: int) -> int:
    """Eq. 1 in the form v = s*o + (o^2 + o)/2."""
    return s * o + (o * o + o) // 2


def volume_peak_form(s: int, o: int) -> float:
    """The equivalent form used in Appendix E.2: p*o - o^2/2 + o/2, p = s + o."""
    p = s + o
    return p * o - o * o / 2 + o / 2


def opt_lower_bound_area(s: Sequence[int], o: Sequence[int], M: int) -> int:
    """Proposition prop:opt_lower_bound in integers: M * TEL(OPT) >=
    sum_j sum_{i<=j} vol_(i) with volumes sorted ascending.  Returns the
    double sum (compare against M * OPT)."""
    vols = sorted(volume_closed(int(a), int(b)) for a, b in zip(s, o))
    total, prefix = 0, 0
    for v in vols:
        prefix += v
        total += prefix
    return total


def opt_lower_bound_exec(o: Sequence[int]) -> int:
    """Lemma lemma:opt_lb_execution: TEL(OPT) >= sum_i o_i."""
    return int(sum(int(x) for x in o))


def onebit_minimax(T: int):
    """Theorem thm:svf_1bit_burst: threshold sqrt(T), proxies T^(1/4), T^(3/4)
    (geometric means of [1, theta] and (theta, T])."""
    theta = math.isqrt(T)
    return theta, math.isqrt(theta), math.isqrt(theta * T)


def geometric_mean_volume(mean_s: float, mu: float) -> float:
    """Appendix F, Lemma 2: E[vol] = E[s]/mu + 1/mu^2 for o ~ Geometric(mu)
    independent of s."""
    return mean_s / mu + 1.0 / (mu * mu)


def poisson_conditional_proxies(mu: float, theta: int):
    """Theorem thm:svf_1bit_poisson: O_0 = 1/mu - theta q^theta/(1-q^theta),
    O_1 = theta + 1/mu, eps = (theta q^theta/(1-q^theta))^2 / 2, q = 1 - mu."""
    q = 1.0 - mu
    r = theta * q ** theta / (1.0 - q ** theta)
    return 1.0 / mu - r, theta + 1.0 / mu, 0.5 * r * r


# ---- Poisson arrivals, geometric outputs (Section 3.3; proofs in the appendix
#      on the stochastic bounds).  q = 1 - mu; alpha = max (s + o) / M;
#      C = (1 - alpha) M / 2 is the processing rate of Lemma 1 there.

def poisson_capacity(M: float, alpha: float) -> float:
    """Lemma 1 of the stochastic appendix: with a non-empty queue the rate of
    processed volume exceeds (1 - alpha) M / 2."""
    return (1.0 - alpha) * M / 2.0


def poisson_rho(lam: float, mean_vol: float, M: float, alpha: float) -> float:
    """Worst-case utilisation rho = lam E[vol] / ((1 - alpha) M / 2)."""
    return lam * mean_vol / poisson_capacity(M, alpha)


def poisson_w0(lam: float, mean_s: float, mu: float) -> float:
    """Lemma 2 of the stochastic appendix: W_0 = lam (E[s]/mu^2 + 2/mu^3)."""
    return lam * (mean_s / mu ** 2 + 2.0 / mu ** 3)


def poisson_w_exact(lam: float, mean_s: float, mu: float) -> float:
    """W_exact = (1 - mu) W_0 (end of the proof of thm:svf_poisson)."""
    return (1.0 - mu) * poisson_w0(lam, mean_s, mu)


def poisson_svf_latency_bound(lam, mean_s, mu, M, alpha, distortion=1.0):
    """The step of the proof before OPT enters: E[latency] <= E[o] + factor *
    W_0 / ((1 - alpha) M / 2 - lam E[vol]), factor = 1 for SVF and
    E[vol] / (E[vol] - eps) for 1-bit SVF."""
    ev = geometric_mean_volume(mean_s, mu)
    slack = poisson_capacity(M, alpha) - lam * ev
    return 1.0 / mu + distortion * poisson_w0(lam, mean_s, mu) / slack


def poisson_cr_bound(alpha: float, mu: float, rho: float, distortion: float = 1.0) -> float:
    """Theorems thm:svf_poisson (distortion 1) and thm:svf_1bit_poisson
    (distortion E[vol] / (E[vol] - eps)): 1 + d * 2 / ((1-alpha)(1-mu)(1-rho))."""
    return 1.0 + distortion * 2.0 / ((1.0 - alpha) * (1.0 - mu) * (1.0 - rho))
