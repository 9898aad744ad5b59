"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: the paper's
worked example, brute force in exact integer/rational arithmetic, closed forms
of the runtime model, library solvers, or published generator outputs.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.integrate
import scipy.linalg.lapack
import scipy.special
import scipy.stats

from oracle import coded as oc
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def int_matmul(A, X):
    """Exact product of integer nested lists (brute force)."""
    return [[sum(int(A[i][t]) * int(X[t][j]) for t in range(len(X))) for j in range(len(X[0]))]
            for i in range(len(A))]


def vandermonde_parity(n, k):
    """Integer parity rows P[i][j] = (j+1)^i.  Vandermonde matrices on positive
    nodes are totally positive, so every square sub-matrix of P is invertible
    and [I; P] is MDS (checked by brute force in test_vandermonde_codes_are_mds)."""
    return np.array([[float((j + 1) ** i) for j in range(k)] for i in range(n - k)])


def frac_det(M):
    M = [[Fraction(v) for v in row] for row in M]
    m = len(M)
    det = Fraction(1)
    for j in range(m):
        p = next((i for i in range(j, m) if M[i][j] != 0), None)
        if p is None:
            return Fraction(0)
        if p != j:
            M[j], M[p] = M[p], M[j]
            det = -det
        det *= M[j][j]
        for i in range(j + 1, m):
            f = M[i][j] / M[j][j]
            M[i] = [a - f * b for a, b in zip(M[i], M[j])]
    return det


# ---------------------------------------------------------------------------
# The paper's worked example
# ---------------------------------------------------------------------------

def test_toy_example_worker3_stores_sum_and_any_two_decode():
    toy = load("toy_3_2.json")
    G = np.array(toy["G"], dtype=np.float64)
    A, x = toy["A"], toy["x"]
    q = len(A)
    blocks = oc.pad_and_split(np.array(A, dtype=np.float64), toy["k"])
    coded = oc.encode(G, blocks)
    half = q // 2
    # worker 3 stores A1 + A2, computed here element by element with Python ints
    w3 = [[A[i][j] + A[half + i][j] for j in range(len(A[0]))] for i in range(half)]
    assert coded[2].tolist() == w3
    assert coded[0].tolist() == A[:half] and coded[1].tolist() == A[half:]
    Y = oc.worker_products(coded, np.array(x, dtype=np.float64))
    expect = int_matmul(A, x)
    # A2 x = (A1 + A2) x - A1 x, the subtraction the paper describes
    a2x = int_matmul(A[half:], x)
    assert (Y[2] - Y[0]).tolist() == a2x
    for S in itertools.combinations(range(3), 2):
        out = oc.decode_from_all(G, S, Y, q)
        assert out.tolist() == expect, S


# ---------------------------------------------------------------------------
# Decoding from every k-subset of tiny codes, against exact brute force
# ---------------------------------------------------------------------------

TINY = [(3, 2), (4, 2), (5, 3), (6, 4), (6, 3), (7, 4)]


@pytest.mark.parametrize("n,k", TINY)
def test_vandermonde_codes_are_mds(n, k):
    G = oc.systematic_generator(vandermonde_parity(n, k))
    for S in itertools.combinations(range(n), k):
        assert frac_det(G[list(S)].tolist()) != 0


@pytest.mark.parametrize("n,k", TINY)
@pytest.mark.parametrize("q", [None, "ragged"])
def test_every_k_subset_decodes_to_brute_force_product(n, k, q):
    r, s = 5, 3
    qq = 4 * k if q is None else 4 * k - 1 - (k > 2)       # ragged: not a multiple of k
    A = synth.integers((qq, r), 11, synth.STREAM_A, n, k)
    X = synth.integers((r, s), 11, synth.STREAM_X, n, k)
    G = oc.systematic_generator(vandermonde_parity(n, k))
    expect = np.array(int_matmul(A.astype(int).tolist(), X.astype(int).tolist()), dtype=np.float64)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    for S in itertools.combinations(range(n), k):
        out = oc.decode_from_all(G, S, Y, qq)
        assert out.shape == (qq, s)
        err = np.max(np.abs(out - expect))
        assert err <= 1e-9 * max(1.0, np.max(np.abs(expect))), (S, err)


def test_decode_uses_first_k_in_arrival_order_and_ignores_order():
    n, k = 6, 3
    A = synth.integers((9, 4), 3, synth.STREAM_A)
    X = synth.integers((4, 2), 3, synth.STREAM_X)
    G = oc.systematic_generator(vandermonde_parity(n, k))
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    expect = A.astype(np.float64) @ X
    arrivals = [5, 1, 3, 0, 2]          # more than k: only the first k count
    out = oc.decode(G, arrivals, [Y[i] for i in arrivals], 9)
    assert np.allclose(out, expect, atol=1e-10)
    # a poisoned result after the first k must not matter
    res = [Y[i] for i in arrivals]
    res[3] = np.full_like(res[3], np.nan)
    assert np.allclose(oc.decode(G, arrivals, res, 9), expect, atol=1e-10)
    with pytest.raises(oc.DecodeError):
        oc.decode(G, [1, 2], [Y[1], Y[2]], 9)
    with pytest.raises(oc.DecodeError):
        oc.decode(G, [1, 1, 2], [Y[1], Y[1], Y[2]], 9)


def test_systematic_survivors_reduce_to_identity():
    n, k, q, r, s = 16, 12, 200, 33, 2
    P = synth.parity_matrix(n, k, 1)
    G = oc.systematic_generator(P)
    A = synth.gaussian((q, r), 1, synth.STREAM_A)
    X = synth.gaussian((r, s), 1, synth.STREAM_X)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    out = oc.decode_from_all(G, list(range(k)), Y, q)
    qb = oc.block_rows(q, k)
    assert np.array_equal(out, Y[:k].reshape(k * qb, s)[:q])
    # and the systematic blocks are A's own blocks, untouched (Sec. III-A)
    coded = oc.encode(G, oc.pad_and_split(A, k))
    assert np.array_equal(coded[:k].reshape(k * qb, r)[:q], A.astype(np.float64))


def test_encode_is_linear():
    n, k = 7, 4
    G = oc.systematic_generator(vandermonde_parity(n, k))
    A = synth.integers((10, 6), 5, synth.STREAM_A)
    B = synth.integers((10, 6), 6, synth.STREAM_A)
    lhs = oc.encode(G, oc.pad_and_split(3 * A - 2 * B, k))
    rhs = 3 * oc.encode(G, oc.pad_and_split(A, k)) - 2 * oc.encode(G, oc.pad_and_split(B, k))
    assert np.array_equal(lhs, rhs)
    # the parity rows are the exact integer combinations of the blocks
    blocks = oc.pad_and_split(A, k)
    for p in range(n - k):
        manual = sum(int(G[k + p, j]) * blocks[j].astype(int) for j in range(k))
        assert np.array_equal(oc.encode(G, blocks)[k + p], manual)


@pytest.mark.parametrize("n,k,q", [(4, 2, 10), (16, 12, 50), (8, 5, 23)])
def test_decode_of_encode_is_identity(n, k, q):
    """With X = I every worker returns its own coded block; decoding any k of
    them gives A back (padding rows dropped)."""
    r = 7
    P = synth.parity_matrix(n, k, 9)
    G = oc.systematic_generator(P)
    A = synth.gaussian((q, r), 9, synth.STREAM_A)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), np.eye(r))
    rng = np.random.default_rng(0)
    for _ in range(20):
        S = sorted(rng.choice(n, size=k, replace=False).tolist())
        out = oc.decode_from_all(G, S, Y, q)
        kappa = np.linalg.cond(G[S])
        assert np.max(np.abs(out - A)) <= 1e-14 * kappa * np.max(np.abs(A)) * k


# ---------------------------------------------------------------------------
# The hand-written LU against LAPACK
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("m", [1, 2, 5, 16, 33])
def test_lu_matches_lapack_getrf_and_solves(m):
    rng = np.random.default_rng(m)
    M = rng.standard_normal((m, m))
    LU, piv, info = oc.lu_factor(M)
    lu_ref, ipiv_ref, info_ref = scipy.linalg.lapack.dgetrf(M)
    assert info == info_ref == 0
    assert np.array_equal(piv, ipiv_ref)
    assert np.allclose(LU, lu_ref, rtol=1e-12, atol=1e-12)
    B = rng.standard_normal((m, 4))
    assert np.allclose(oc.lu_solve(LU, piv, B), np.linalg.solve(M, B), rtol=1e-10, atol=1e-10)


def test_lu_reports_first_zero_pivot_like_getrf():
    M = np.array([[1.0, 2.0, 3.0], [2.0, 4.0, 6.0], [1.0, 0.0, 1.0]])
    _, _, info = oc.lu_factor(M)
    _, _, info_ref = scipy.linalg.lapack.dgetrf(M)
    assert info == info_ref and info > 0
    # a non-MDS code (two equal parity rows) gives a singular survivor matrix
    G = oc.systematic_generator(np.array([[1.0, 2.0], [1.0, 2.0]]))
    with pytest.raises(oc.DecodeError) as e:
        oc.decode(G, [2, 3], [np.ones((2, 1)), np.ones((2, 1))], 4)
    assert e.value.info == 2


# ---------------------------------------------------------------------------
# The counter-based generator behind the runtime draw
# ---------------------------------------------------------------------------

def test_splitmix64_published_outputs():
    ref = load("splitmix64_seed1234567.json")
    state = ref["seed"]
    for want in ref["outputs"]:
        state, z = oc.splitmix64_next(state)
        assert z == int(want)
    for i, want in enumerate(ref["outputs"]):
        assert oc.splitmix64_output(ref["seed"], i) == int(want)


def test_counter_layout_matches_sequential_stepping():
    seed = 987654321
    state = seed
    seq = []
    for _ in range(40):
        state, z = oc.splitmix64_next(state)
        seq.append(z)
    for w in range(40):
        assert oc.runtime_word(seed, 0, 0, w) == seq[w]
    # draw d, worker w of stream s sits at counter s*2^56 + d*2^16 + w
    assert oc.runtime_counter(4, 3, 7) == (4 << 56) + 3 * 65536 + 7


# ---------------------------------------------------------------------------
# The runtime model: closed forms of Sec. III-C/III-D
# ---------------------------------------------------------------------------

def harmonic(n):
    return sum(Fraction(1, i) for i in range(1, n + 1))


def sample_tk(n, k, draws, shift=1.0, rate=1.0, seed=77):
    return np.array([oc.draw_survivors(n, k, seed, d, shift, rate)[1] for d in range(draws)])


@pytest.mark.parametrize("n,k,shift,rate", [(16, 12, 1.0, 1.0), (10, 5, 1.0, 1.0), (64, 48, 1.0, 1.0),
                                            (10, 10, 1.0, 1.0), (12, 4, 2.0, 0.5)])
def test_mean_of_kth_order_statistic_matches_closed_form(n, k, shift, rate):
    """E[T_(k)] = (1/k)(shift + (H_n - H_{n-k})/mu) (Sec. III-D, exact harmonic
    form of eq. mds_coded_2; k = n is the uncoded case (1/n)(1 + H_n/mu))."""
    draws = 6000 if n <= 16 else 2000
    T = sample_tk(n, k, draws, shift, rate)
    mean = (shift + float(harmonic(n) - harmonic(n - k)) / rate) / k
    var = sum(1.0 / i ** 2 for i in range(n - k + 1, n + 1)) / (rate * k) ** 2
    assert abs(T.mean() - mean) < 5 * math.sqrt(var / draws)
    assert T.min() >= shift / k


def test_kth_order_statistic_follows_F_mds():
    """KS test of T_(k) against eq. F_mds at n=10, k=5 (the setting of the runtime-distribution figure),
    integrating the printed density numerically."""
    n, k, mu = 10, 5, 1.0
    F = lambda t: 1.0 - math.exp(-mu * (t - 1.0)) if t >= 1.0 else 0.0
    f = lambda t: mu * math.exp(-mu * (t - 1.0)) if t >= 1.0 else 0.0

    def F_mds(t):
        integrand = lambda tau: n * k * f(k * tau) * math.comb(n - 1, k - 1) * F(k * tau) ** (k - 1) \
            * (1.0 - F(k * tau)) ** (n - k)
        return scipy.integrate.quad(integrand, 1.0 / k, max(t, 1.0 / k), limit=200)[0]

    # the printed integral agrees with the binomial form of the k-th order statistic
    for t in [0.21, 0.25, 0.3, 0.5]:
        assert abs(F_mds(t) - scipy.special.betainc(k, n - k + 1, F(k * t))) < 1e-8
    T = sample_tk(n, k, 3000, seed=5)
    stat, p = scipy.stats.kstest(T, np.vectorize(F_mds))
    assert p > 1e-3, (stat, p)


@pytest.mark.parametrize("n,k", [(4, 2), (16, 12)])
def test_parity_survivor_count_is_hypergeometric(n, k):
    """Runtimes are i.i.d., so the first k of n is a uniform k-subset and the
    number of parity survivors m is hypergeometric."""
    draws = 6000
    counts = np.zeros(min(k, n - k) + 1)
    for d in range(draws):
        S, _ = oc.draw_survivors(n, k, 3, d)
        counts[int(np.sum(S >= k))] += 1
    probs = np.array([math.comb(n - k, m) * math.comb(k, k - m) / math.comb(n, k) for m in range(len(counts))])
    keep = probs * draws >= 5
    obs = np.append(counts[keep], counts[~keep].sum())
    exp = np.append(probs[keep] * draws, probs[~keep].sum() * draws)
    if exp[-1] == 0:
        obs, exp = obs[:-1], exp[:-1]
    assert scipy.stats.chisquare(obs, exp).pvalue > 1e-3


def test_accepted_survivor_sets_follow_the_conditioned_hypergeometric_law():
    """The decode-heavy rule keeps sequential draws whose set has m >= 8 parity
    workers and that differ from every kept set.  With C(64,48) ~ 4.9e14 sets,
    repeats are negligible, so the kept sets' parity counts must follow the
    law of the k fastest of n i.i.d. runtimes (Sec. III-B: every k-subset is
    equally likely, m is hypergeometric) conditioned on m >= 8."""
    n, k, m_min, B = 64, 48, 8, 4000
    sets, _ = oc.draw_survivor_sets(n, k, 11, B, min_parity=m_min)
    m = (sets >= k).sum(axis=1)
    support = np.arange(m_min, n - k + 1)
    w = np.array([math.comb(n - k, j) * math.comb(k, k - j) for j in support], dtype=np.float64)
    probs = w / w.sum()
    counts = np.array([np.sum(m == j) for j in support])
    assert counts.sum() == B
    keep = probs * B >= 5
    obs, exp = counts[keep], probs[keep] * B
    if np.any(~keep):
        obs, exp = np.append(obs, counts[~keep].sum()), np.append(exp, probs[~keep].sum() * B)
    assert scipy.stats.chisquare(obs, exp).pvalue > 1e-3


def test_survivor_set_batch_limited_by_the_number_of_qualifying_sets():
    """sum_{m >= m_min} C(k,m) C(n-k,m) sets exist; all of them come back when
    that many are asked for, and one more is refused instead of drawing forever."""
    n, k, m_min = 6, 3, 2
    total = sum(math.comb(k, j) * math.comb(n - k, j) for j in range(m_min, min(k, n - k) + 1))
    assert total == 10
    sets, _ = oc.draw_survivor_sets(n, k, 5, total, min_parity=m_min)
    every = {c for c in itertools.combinations(range(n), k) if sum(v >= k for v in c) >= m_min}
    assert {tuple(int(v) for v in s) for s in sets} == every
    with pytest.raises(ValueError):
        oc.draw_survivor_sets(n, k, 5, total + 1, min_parity=m_min)
    with pytest.raises(ValueError):
        oc.draw_survivor_sets(4, 2, 0, 7)


def test_survivor_sets_with_min_parity_are_distinct_and_qualify():
    n, k = 64, 48
    sets, nxt = oc.draw_survivor_sets(n, k, 4, 300, min_parity=8)
    assert sets.shape == (300, k)
    assert len({tuple(s) for s in sets}) == 300
    assert all(np.all(np.diff(s) > 0) for s in sets)
    assert all(np.sum(s >= k) >= 8 for s in sets)
    assert nxt >= 300


# ---------------------------------------------------------------------------
# Coded gradient descent (Sec. III-E)
# ---------------------------------------------------------------------------

def test_coded_gd_tracks_plain_gd_and_reaches_least_squares():
    q, r = 96, 8
    A = synth.gaussian((q, r), 2, synth.STREAM_A, std=1.0 / math.sqrt(r)).astype(np.float64)
    w = synth.gaussian((r,), 2, synth.STREAM_WSTAR).astype(np.float64)
    y = A @ w + 0.1 * synth.gaussian((q,), 2, synth.STREAM_NOISE).astype(np.float64)
    G1 = oc.systematic_generator(synth.parity_matrix(6, 4, 2))
    G2 = oc.systematic_generator(synth.parity_matrix(6, 4, 2, synth.STREAM_PT))
    lam = np.linalg.eigvalsh(A.T @ A)
    eta = 1.0 / lam.max()
    rec = []
    oc.coded_gd(A, y, np.zeros(r), G1, G2, eta, 60, seed=2, record=rec)
    x = np.zeros(r)
    for t in range(60):
        x = x - eta * (A.T @ (A @ x - y))
        assert np.allclose(rec[t], x, rtol=1e-9, atol=1e-11), t
    x_ls = np.linalg.lstsq(A, y, rcond=None)[0]
    assert np.allclose(rec[-1], x_ls, rtol=1e-6, atol=1e-8)


@pytest.mark.parametrize("which", ["A", "T"])
def test_conditioned_gd_generators_certificate(which):
    """The coded gradient-descent codes' certified generators (code of A and of
    A^T): every one of the C(20,16) = 4845 survivor sets has a decode system
    with condition number at most the recorded bound, which is attained, and
    the plain draw of the same stream is worse."""
    w = synth.WORKLOADS["gd20x16_conditioned_262144x4096"]
    PA, PT, planes = synth.gd_codes(w)
    assert planes == 1
    P = PA if which == "A" else PT
    bound = w.extra["worst_condition" if which == "A" else "worst_condition_T"]
    G = oc.systematic_generator(P)
    k = w.k
    seen = 0.0
    for S in itertools.combinations(range(w.n), k):
        par = [i for i in S if i >= k]
        miss = [j for j in range(k) if j not in S]
        if par:
            seen = max(seen, np.linalg.cond(G[np.array(par)][:, miss]))
    assert abs(seen - bound) <= 0.05 and abs(synth.worst_decode_condition(P) - seen) <= 1e-6 * seen
    plain = synth.parity_matrix(w.n, w.k, w.seed, synth.STREAM_P if which == "A" else synth.STREAM_PT)
    assert synth.worst_decode_condition(plain) > 2 * bound


def test_conditioned_generator_certificate():
    """The GEMV regime's conditioned generator: every one of the C(16,12) survivor
    sets of G = [I; P] has a decode system (parity survivors x missing blocks)
    with 2-norm condition number at most the recorded bound, checked here by
    walking the survivor sets themselves (not the sub-blocks of P)."""
    w = synth.WORKLOADS["gemv16x12_conditioned_65536x8192"]
    P, c, worst = synth.conditioned_parity_matrix(w.n, w.k, w.seed, w.extra["candidates"],
                                                  pick=w.extra["parity_candidate"])
    assert c == w.extra["parity_candidate"] and abs(worst - w.extra["worst_condition"]) < 0.1
    G = oc.systematic_generator(P)
    k = w.k
    seen = 0
    for S in itertools.combinations(range(w.n), k):
        par = [i for i in S if i >= k]
        miss = [j for j in range(k) if j not in S]
        if par:
            kap = np.linalg.cond(G[np.array(par)][:, miss])
            assert kap <= worst * (1 + 1e-9), S
            seen = max(seen, kap)
    assert abs(seen - worst) <= 1e-6 * worst           # the bound is attained
    # and the plain seed-2 draw of the same workload is worse
    assert synth.worst_decode_condition(synth.parity_matrix(w.n, w.k, w.seed)) > 4 * worst
