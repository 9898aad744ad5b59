"""Pins of the coded-shuffling oracle (Sec. IV) against the paper's examples,
its rate theorem and corollaries, and the invariants of the cache rule."""
import itertools
import math

import numpy as np
import pytest

from oracle import coded as oc
from oracle import shuffle as sh


def test_vectorised_words_match_the_scalar_generator():
    rng = np.random.default_rng(0)
    ctr = rng.integers(0, 2 ** 63, size=50, dtype=np.uint64)
    got = sh.splitmix_words(1234567, ctr)
    assert [int(v) for v in got] == [oc.splitmix64_output(1234567, int(c)) for c in ctr]


def test_toy_example_two_workers():
    """Sec. I's illustration: W1 holds A1, A2 and W2 holds A3, A4; W1 now needs A3 and W2
    needs A2.  One multicast row A2 + A3 replaces two unicast rows."""
    A = np.array([[1, 2], [3, 4], [5, 6], [7, 8]], dtype=np.float32)
    st = sh.State(2, 4, 2, 0, 0, np.array([0, 0, 1, 1], dtype=np.int32),
                  np.array([[1, 1, 0, 0], [0, 0, 1, 1]], dtype=bool))
    p = sh.plan(st, np.array([0, 1, 0, 1], dtype=np.int32))
    assert p.coded_rows == 1 and p.uncoded_rows == 2
    M = sh.encode(A, p)
    assert np.array_equal(M[0], A[1] + A[2])
    out = sh.decode(A, M, p)
    for d in range(2):
        assert np.array_equal(out[d], A[p.enc_rows[d]])
    assert sorted(zip(p.term_worker.tolist(), p.enc_rows.tolist())) == [(0, 2), (1, 1)]


def test_three_worker_example_message_parts():
    """Sec. IV's example (n = 3): the message has a part for each of {1,2}, {1,3},
    {2,3} and {1,2,3}, and part I sums the rows of S_i cached exactly by I - {i}."""
    n, q = 3, 18
    # signature of each row (workers caching it) and the new owner of each row
    sigs = [0b001, 0b010, 0b100, 0b011, 0b101, 0b110] * 3
    cached = np.array([[(sg >> i) & 1 for sg in sigs] for i in range(n)], dtype=bool)
    new = np.array([(int(np.nonzero([(sg >> i) & 1 == 0 for i in range(n)])[0][j % 2 if bin(sg).count("1") == 1 else 0]))
                    for j, sg in enumerate(sigs)], dtype=np.int32)
    st = sh.State(n, q, 6, 0, 0, np.zeros(q, dtype=np.int32), cached)
    p = sh.plan(st, new)
    keys = [g[0] for g in p.groups]
    assert keys == sorted(set(keys)) and set(keys) <= {0b011, 0b101, 0b110, 0b111}
    assert set(keys) == {0b011, 0b101, 0b110, 0b111}
    for key, lists, length in p.groups:
        for i, rows in lists.items():
            assert (key >> i) & 1
            for r in rows:
                assert new[r] == i and not cached[i, r]
                assert sigs[r] == key & ~(1 << i)          # r lies in C~_{I - {i}}
        assert length == max(len(v) for v in lists.values())


@pytest.mark.parametrize("n,frac", [(50, 0.1), (10, 0.3), (20, 0.08), (3, 0.5), (64, 0.02)])
def test_rate_closed_form_equals_sum(n, frac):
    q = 1000 * n
    s = frac * q
    assert sh.rate_coded_closed(n, q, s) == pytest.approx(sh.rate_coded_sum(n, q, s), rel=1e-10)


def test_rate_corollaries():
    # Corollary 2: caches that just hold the data in use halve the rate
    for n in (2, 5, 50):
        q = 100 * n
        assert sh.rate_coded_sum(n, q, q / n) == pytest.approx(sh.rate_uncoded(n, q, q / n) / 2, rel=1e-12)
    # the figure's setting: n = 50, q = 1000, s/q = 0.1 cuts the rate by more than 81%
    assert 1 - sh.rate_coded_sum(50, 1000, 100) / sh.rate_uncoded(50, 1000, 100) > 0.81
    # Corollary 3: for large n the gain approaches n s/q
    n, q, s = 4000, 4_000_000, 400_000
    assert sh.rate_coded_sum(n, q, s) == pytest.approx(sh.rate_uncoded(n, q, s) / (n * s / q), rel=2e-2)


def test_simulated_rates_follow_the_theorem():
    """Law of large numbers: a simulated iteration sends close to R_u unique rows
    uncoded and close to R_c rows coded (padding to the longest list adds a little)."""
    n, q, s = 8, 40000, 10000
    st = sh.initial_state(n, q, s, 11)
    for _ in range(2):
        p = sh.plan(st)
        assert p.uncoded_rows == pytest.approx(sh.rate_uncoded(n, q, s), rel=0.02)
        assert p.coded_rows >= 0.98 * sh.rate_coded_sum(n, q, s)
        assert p.coded_rows <= 1.10 * sh.rate_coded_sum(n, q, s)
        st = sh.commit(st, p)


def test_cache_rule_invariants_and_complete_delivery():
    n, q, s = 5, 200, 70
    st = sh.initial_state(n, q, s, 3)
    A = np.arange(q * 3, dtype=np.float32).reshape(q, 3)        # integer rows: sums are exact
    for _ in range(4):
        assert np.all(np.bincount(st.assign, minlength=n) == q // n)
        for i in range(n):
            assert st.cached[i].sum() == s and np.all(st.cached[i][st.assign == i])
        p = sh.plan(st)
        out = sh.decode(A, sh.encode(A, p), p)
        assert np.array_equal(out, A[p.enc_rows])                 # every row decodes exactly
        for i in range(n):
            got = set(np.nonzero(st.cached[i])[0]) | set(p.enc_rows[p.term_worker == i].tolist())
            assert set(np.nonzero(p.new_assign == i)[0]) <= got   # the new set is complete
        nxt = sh.commit(st, p)
        for i in range(n):
            extra = nxt.cached[i] & (nxt.assign != i)
            assert np.all(st.cached[i][extra])                   # kept rows come from the old cache
        st = nxt


def test_decode_rounding_with_real_rows():
    """Over floats the sums round: a decoded row is within the rounding of its
    message, and it equals the oracle's own arithmetic to the bit."""
    n, q, s = 6, 600, 200
    st = sh.initial_state(n, q, s, 5)
    rng = np.random.default_rng(1)
    A = rng.standard_normal((q, 16)).astype(np.float32)
    p = sh.plan(st)
    M = sh.encode(A, p)
    out = sh.decode(A, M, p)
    for d in range(len(p.enc_rows)):
        m = p.term_msg[d]
        terms = p.enc_rows[p.enc_off[m]:p.enc_off[m + 1]]
        bound = 2 * len(terms) * np.finfo(np.float32).eps * np.sum(np.abs(A[terms]), axis=0)
        assert np.all(np.abs(out[d] - A[p.enc_rows[d]]) <= bound)
