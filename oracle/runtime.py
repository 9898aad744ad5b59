"""Runtime model of coded and uncoded distributed computation (fp64 CPU oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Follows Sec. III-B to
III-D of Lee et al., "Speeding Up Distributed Machine Learning Using Codes":

* a job split into l subtasks: each subtask takes T0 / l, with the mother
  runtime T0 = shift + E / mu, E ~ Exp(1) (eq. shifted_exp, Sec. III-C);
* uncoded: n subtasks, the job ends with the slowest (eq. uncoded);
* n/k-repetition: k subtasks, each replicated on n/k consecutive workers,
  the job ends when every subtask has one finished replica (eq. rep_coded);
* (n,k) MDS: k-sized subtasks on n workers, the job ends with the k-th
  finisher (eq. mds_coded);
* expected runtimes, their distributions (eq. F_rep, F_mds) and the optimal
  MDS code dimension k* through the lower branch of Lambert W (Lemma 2).

Worker runtimes come from the same counter-based SplitMix64 words as the
survivor draw of the coded product (oracle/coded.py), so one draw gives the
three schemes common random numbers.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

from .coded import RUNTIME_STREAM, SPLITMIX_GAMMA

_M64 = np.uint64(0xFFFFFFFFFFFFFFFF)


def harmonic(n: int) -> float:
    """H_n = sum_{i<=n} 1/i, exactly (the paper approximates it by log n)."""
    return float(sum(Fraction(1, i) for i in range(1, n + 1)))


def expected_uncoded(n: int, mu: float, shift: float = 1.0) -> float:
    """E[max of n subtasks of T0/n] = (shift + H_n / mu) / n."""
    return (shift + harmonic(n) / mu) / n


def expected_repetition(n: int, k: int, mu: float, shift: float = 1.0) -> float:
    """E[max over k tasks of the min over n/k replicas of T0/k]: the minimum of
    n/k exponentials of rate mu is exponential of rate (n/k) mu, and the mean
    maximum of k of those is H_k / ((n/k) mu)."""
    if n % k:
        raise ValueError("repetition needs k | n")
    return (shift + harmonic(k) * k / (n * mu)) / k


def expected_mds(n: int, k: int, mu: float, shift: float = 1.0) -> float:
    """E[k-th smallest of n subtasks of T0/k] = (shift + (H_n - H_{n-k}) / mu) / k."""
    return (shift + (harmonic(n) - harmonic(n - k)) / mu) / k


def _F(t, mu, shift):
    t = np.asarray(t, dtype=np.float64)
    return np.where(t >= shift, 1.0 - np.exp(-mu * (t - shift)), 0.0)


def cdf_uncoded(t, n: int, mu: float, shift: float = 1.0):
    """[F(n t)]^n."""
    return _F(n * np.asarray(t, dtype=np.float64), mu, shift) ** n


def cdf_repetition(t, n: int, k: int, mu: float, shift: float = 1.0):
    """eq. F_rep: [1 - (1 - F(k t))^(n/k)]^k."""
    Fk = _F(k * np.asarray(t, dtype=np.float64), mu, shift)
    return (1.0 - (1.0 - Fk) ** (n // k)) ** k


def cdf_mds(t, n: int, k: int, mu: float, shift: float = 1.0):
    """eq. F_mds, in its binomial form: P(at least k of n finish by t)."""
    Fk = _F(k * np.asarray(t, dtype=np.float64), mu, shift)
    return sum(math.comb(n, j) * Fk ** j * (1.0 - Fk) ** (n - j) for j in range(k, n + 1))


def lambert_w_lower(x: float) -> float:
    """W_{-1}(x) for -1/e <= x < 0, from its definition: the solution w <= -1
    of w e^w = x (Lemma 2 uses this lower real branch).

    On (-inf, -1] the map f(w) = w e^w decreases monotonically from 0 (as
    w -> -inf) to -1/e (at w = -1), so the root is unique.  It is bracketed
    by [lo, -1] with lo pushed left until f(lo) > x, then found by plain
    bisection: the bracket is halved until no fp64 value lies strictly
    inside it, and the end whose f is nearer x is returned."""
    if not (-1.0 / math.e <= x < 0.0):
        raise ValueError("W_{-1} is real on [-1/e, 0)")

    def f(w):
        return w * math.exp(w)

    hi = -1.0
    if f(hi) >= x:                    # x at the branch point (within rounding)
        return hi
    lo = -2.0
    while f(lo) <= x:                 # f(lo) must lie above x (nearer 0)
        lo *= 2.0
    # invariant: lo < hi, f(lo) > x >= f(hi)
    while True:
        mid = 0.5 * (lo + hi)
        if not (lo < mid < hi):
            break
        if f(mid) > x:
            lo = mid
        else:
            hi = mid
    return lo if abs(f(lo) - x) < abs(f(hi) - x) else hi


def optimal_mds(n: int, mu: float):
    """Lemma 2: k* = [1 + 1/W_{-1}(-e^{-mu-1})] n and T* = -W_{-1}(-e^{-mu-1}) / (mu n).
    Returns (k*, T*, n T*)."""
    w = lambert_w_lower(-math.exp(-mu - 1.0))
    return (1.0 + 1.0 / w) * n, -w / (mu * n), -w / mu


def best_integer_k(n: int, mu: float, shift: float = 1.0) -> int:
    """The k in [1, n] with the smallest exact expected MDS runtime (ties: smaller k)."""
    vals = [expected_mds(n, k, mu, shift) for k in range(1, n + 1)]
    return int(np.argmin(vals)) + 1


def runtime_words(n: int, seed: int, first_draw: int, draws: int) -> np.ndarray:
    """(draws, n) uint64 SplitMix64 words of the runtime stream: word (d, i) is
    output number (4<<56 | d<<16 | i) of SplitMix64 seeded with `seed`."""
    d = np.arange(first_draw, first_draw + draws, dtype=np.uint64)[:, None]
    i = np.arange(n, dtype=np.uint64)[None, :]
    ctr = (np.uint64(RUNTIME_STREAM) << np.uint64(56)) | (d << np.uint64(16)) | i
    with np.errstate(over="ignore"):
        z = np.uint64(seed) + (ctr + np.uint64(1)) * np.uint64(SPLITMIX_GAMMA)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def mother_runtimes(words: np.ndarray, mu: float, shift: float = 1.0) -> np.ndarray:
    """T0 = shift - ln(U) / mu with U = ((u >> 11) + 0.5) 2^-53."""
    u = ((words >> np.uint64(11)).astype(np.float64) + 0.5) * 2.0 ** -53
    return shift - np.log(u) / mu


def simulate(n: int, k: int, seed: int, first_draw: int, draws: int, mu: float = 1.0, shift: float = 1.0):
    """Overall runtimes of one job per draw under the three schemes, from the
    same worker samples: (uncoded, repetition or None if k does not divide n, MDS)."""
    T0 = mother_runtimes(runtime_words(n, seed, first_draw, draws), mu, shift)
    uncoded = np.max(T0 / n, axis=1)
    mds = np.sort(T0 / k, axis=1)[:, k - 1]
    rep = None
    if n % k == 0:
        groups = (T0 / k).reshape(draws, k, n // k)      # consecutive workers replicate one task
        rep = np.max(np.min(groups, axis=2), axis=1)
    return uncoded, rep, mds
