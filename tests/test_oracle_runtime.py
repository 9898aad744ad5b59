"""Pins of the runtime-model oracle (Sec. III-B..III-D) against closed forms,
library routines, the paper's printed number and exact per-draw relations."""
import json
import math
import os

import numpy as np
import pytest
import scipy.optimize
import scipy.special
import scipy.stats

from oracle import coded as oc
from oracle import runtime as rt

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("x", [-1.0 / math.e + 1e-12, -0.3, -0.2, -0.1, -1e-3, -1e-9, -math.exp(-3.0)])
def test_lambert_w_lower_branch(x):
    w = rt.lambert_w_lower(x)
    ref = scipy.special.lambertw(x, -1).real
    assert w <= -1.0
    assert abs(w - ref) <= 1e-6 * abs(ref) if x > -1.0 / math.e + 1e-10 else abs(w + 1) < 1e-4
    assert abs(w * math.exp(w) - x) <= 1e-13


@pytest.mark.parametrize("eps", [1e-12, 1e-9, 1e-6])
def test_lambert_w_lower_near_the_branch_point(eps):
    """Near x = -1/e the lower branch has the expansion
    W_{-1}(-1/e + eps) = -1 - p - p^2/3 - 11 p^3/72 + O(p^4), p = sqrt(2 e eps)
    (a closed form independent of both the bisection and scipy, which loses
    accuracy here)."""
    x = -math.exp(-1.0) + eps
    p = math.sqrt(2.0 * math.e * eps)
    series = -1.0 - p - p * p / 3.0 - 11.0 * p ** 3 / 72.0
    w = rt.lambert_w_lower(x)
    assert abs(w - series) <= 2.0 * p ** 4 + 1e-7


def test_library_optimal_k_agrees_with_the_bisection_oracle():
    """The library's k* and T* (its own W_{-1}) against the oracle's definition-based root."""
    from paper_1512_02673_amd import binding as lib
    try:
        lib.lib()
    except (OSError, RuntimeError) as e:
        pytest.skip(f"library not built: {e}")
    for n, mu in [(10, 1.0), (64, 0.25), (1000, 1.0), (100, 5.0), (7, 0.05)]:
        ks, ts, kb = lib.coded_optimal_k(n, mu)
        k_ref, t_ref, _ = rt.optimal_mds(n, mu)
        assert ks == pytest.approx(k_ref, rel=1e-12) and ts == pytest.approx(t_ref, rel=1e-12)
        assert kb == rt.best_integer_k(n, mu)


def test_optimal_runtime_factor_printed_in_paper():
    g = json.load(open(os.path.join(GOLDEN, "optimal_mds_mu1.json")))
    _, _, nT = rt.optimal_mds(1000, g["mu"])
    assert round(nT, g["printed_decimals"]) == g["n_times_T_star"]


@pytest.mark.parametrize("mu", [0.25, 0.5, 1.0, 2.0, 5.0])
def test_k_star_minimises_the_continuous_runtime(mu):
    """Lemma 2's k* against direct minimisation of (1/k)(1 + (1/mu) log(n/(n-k)))."""
    n = 1000
    k_star, T_star, _ = rt.optimal_mds(n, mu)
    f = lambda k: (1.0 + math.log(n / (n - k)) / mu) / k
    res = scipy.optimize.minimize_scalar(f, bounds=(1e-6, n - 1e-6), method="bounded",
                                         options={"xatol": 1e-9})
    assert abs(res.x - k_star) <= 1e-4 * n
    assert abs(res.fun - T_star) <= 1e-9
    # the exact-harmonic optimum over integer k sits next to it
    assert abs(rt.best_integer_k(n, mu) - k_star) <= 2.0


def test_expected_runtimes_against_monte_carlo():
    n, k, draws = 10, 5, 200_000
    unc, rep, mds = rt.simulate(n, k, 31, 0, draws, mu=1.0)
    for sample, mean in ((unc, rt.expected_uncoded(n, 1.0)), (rep, rt.expected_repetition(n, k, 1.0)),
                         (mds, rt.expected_mds(n, k, 1.0))):
        assert abs(sample.mean() - mean) <= 5 * sample.std() / math.sqrt(draws)


@pytest.mark.parametrize("n,k,mu,shift", [(10, 5, 1.0, 1.0), (12, 4, 0.5, 2.0)])
def test_runtime_distributions_match_closed_forms(n, k, mu, shift):
    unc, rep, mds = rt.simulate(n, k, 7, 1000, 20_000, mu, shift)
    assert scipy.stats.kstest(unc, lambda t: rt.cdf_uncoded(t, n, mu, shift)).pvalue > 1e-3
    assert scipy.stats.kstest(rep, lambda t: rt.cdf_repetition(t, n, k, mu, shift)).pvalue > 1e-3
    assert scipy.stats.kstest(mds, lambda t: rt.cdf_mds(t, n, k, mu, shift)).pvalue > 1e-3


def test_mds_never_slower_than_repetition_per_draw():
    """The MDS decodable sets contain the repetition ones (remark after eq. F_mds),
    so on every draw the MDS job ends no later."""
    unc, rep, mds = rt.simulate(20, 5, 3, 0, 5000)
    assert np.all(mds <= rep)
    t = np.linspace(0.1, 2.0, 50)
    assert np.all(rt.cdf_mds(t, 20, 5, 1.0) >= rt.cdf_repetition(t, 20, 5, 1.0) - 1e-15)


def test_vectorised_words_match_scalar_generator():
    w = rt.runtime_words(16, 2, 5, 40)
    for d in range(40):
        for i in range(16):
            assert int(w[d, i]) == oc.runtime_word(2, oc.RUNTIME_STREAM, 5 + d, i)
    _, _, mds = rt.simulate(16, 12, 2, 5, 40)
    for d in range(40):
        assert mds[d] == pytest.approx(oc.draw_survivors(16, 12, 2, 5 + d)[1], rel=1e-15)
