"""Coded shuffling (CPU oracle, test infrastructure only).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Follows Sec. IV of Lee
et al., "Speeding Up Distributed Machine Learning Using Codes":

* setup: before every iteration the q data rows are partitioned uniformly at
  random into n sets S_i of q/n rows, one per worker; worker i holds a cache
  C_i of s rows with S_i inside it;
* cache update rule: the new cache is the new S_i plus s - q/n rows drawn
  uniformly without replacement from the old cache minus the new S_i;
* coded transmission (Algorithm 1): for every worker group I with |I| >= 2
  the master multicasts the sum over i in I of the rows A(S_i cap C~_{I-i}),
  each list zero-padded to the longest, where C~_J holds the rows cached by
  exactly the workers of J;
* decoding: worker i subtracts the other members' rows, which it caches by the
  definition of C~, and keeps its own;
* rates: uncoded R_u = q (1 - s/q) (eq. r1) and coded R_c (eq. r2 / rate1).

Reading of the paper used here (no other source fixes them):
* the rows are coded over their own representation (fp32 data, fp32 sums);
  sums and differences run over the members of a group in increasing worker
  index, so a decoded row equals the oracle's to the bit;
* Algorithm 1 iterates over |I| > 2 but the text and the example use
  |I| >= 2; every group that has a row to send is used;
* the random partition and cache draws are taken from counter-based
  SplitMix64 words (stream 8: partition of iteration t, rank by word of
  (t, row); stream 9: cache keep draw of iteration t, rank by word of
  (t, row, worker)); the initial caches are the keep draw of iteration 0
  applied to the whole data set.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from .coded import MASK64, SPLITMIX_GAMMA

PARTITION_STREAM = 8
CACHE_STREAM = 9


def _mix(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def splitmix_words(seed: int, counters: np.ndarray) -> np.ndarray:
    """SplitMix64 output number c for every counter c (vectorised)."""
    c = np.asarray(counters, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & MASK64) + (c + np.uint64(1)) * np.uint64(SPLITMIX_GAMMA)
    return _mix(z)


def partition(n: int, q: int, seed: int, t: int) -> np.ndarray:
    """S^t: worker of every row.  The rows ranked by their stream-8 word of
    (t, row), ties to the lower row, are dealt out q/n at a time."""
    if q % n:
        raise ValueError("q must be a multiple of n")
    rows = np.arange(q, dtype=np.uint64)
    w = splitmix_words(seed, (np.uint64(PARTITION_STREAM) << np.uint64(56)) | (np.uint64(t) << np.uint64(40)) | rows)
    order = np.argsort(w, kind="stable")
    assign = np.empty(q, dtype=np.int32)
    assign[order] = np.arange(q) // (q // n)
    return assign


def keep_draw(rows: np.ndarray, worker: int, t: int, seed: int, count: int) -> np.ndarray:
    """`count` of `rows` uniformly without replacement: the smallest stream-9
    words of (t, row, worker), ties to the lower row."""
    rows = np.sort(np.asarray(rows, dtype=np.int64))
    if count > len(rows):
        raise ValueError("not enough rows to draw from")
    ctr = (np.uint64(CACHE_STREAM) << np.uint64(56)) | (np.uint64(t) << np.uint64(40)) | \
        (rows.astype(np.uint64) << np.uint64(6)) | np.uint64(worker)
    order = np.argsort(splitmix_words(seed, ctr), kind="stable")
    return np.sort(rows[order[:count]])


@dataclass
class State:
    n: int
    q: int
    cache_rows: int
    seed: int
    t: int
    assign: np.ndarray          # S^t: worker of each row
    cached: np.ndarray          # n x q bool: C_i^t


def _apply_cache_rule(n, q, cache_rows, seed, t, assign, old_cached):
    """C_i = S_i plus (s - q/n) rows drawn from old C_i minus S_i."""
    cached = np.zeros((n, q), dtype=bool)
    extra = cache_rows - q // n
    for i in range(n):
        mine = assign == i
        cached[i, mine] = True
        pool = np.nonzero(old_cached[i] & ~mine)[0]
        cached[i, keep_draw(pool, i, t, seed, extra)] = True
    return cached


def initial_state(n: int, q: int, cache_rows: int, seed: int) -> State:
    if not (1 <= n <= 64) or q % n or not (q // n <= cache_rows <= q):
        raise ValueError("need 1 <= n <= 64, n | q and q/n <= cache_rows <= q")
    assign = partition(n, q, seed, 0)
    cached = _apply_cache_rule(n, q, cache_rows, seed, 0, assign, np.ones((n, q), dtype=bool))
    return State(n, q, cache_rows, seed, 0, assign, cached)


def signatures(cached: np.ndarray) -> np.ndarray:
    """Bit i of a row's signature is set when worker i caches it."""
    n = cached.shape[0]
    sig = np.zeros(cached.shape[1], dtype=np.uint64)
    for i in range(n):
        sig |= cached[i].astype(np.uint64) << np.uint64(i)
    return sig


@dataclass
class Plan:
    new_assign: np.ndarray      # S^{t+1}
    groups: list                # [(I mask, {worker: rows}, padded length)] in increasing I
    enc_off: np.ndarray         # message m's terms: enc_rows[enc_off[m]:enc_off[m+1]]
    enc_rows: np.ndarray        # row of A of every term
    term_worker: np.ndarray     # the worker that needs that row
    term_msg: np.ndarray        # the message the term belongs to
    coded_rows: int             # rows multicast with coding (sum of padded lengths)
    uncoded_rows: int           # rows sent one by one without coding


def plan(state: State, new_assign: np.ndarray | None = None) -> Plan:
    """Algorithm 1 for the next partition (drawn, or given): worker i lacks
    the rows of its new S_i outside C_i; such a row with signature J goes into
    the message of group I = J + {i} (its rows lie in S_i cap C~_{I-i}).  The
    messages of a group are padded to its longest list; message rows sum the
    members' j-th rows in increasing worker order."""
    n, q = state.n, state.q
    if new_assign is None:
        new_assign = partition(n, q, state.seed, state.t + 1)
    sig = signatures(state.cached)
    groups = {}
    for i in range(n):
        need = np.nonzero((new_assign == i) & ~state.cached[i])[0]
        for r in need:
            key = int(sig[r]) | (1 << i)
            groups.setdefault(key, {}).setdefault(i, []).append(int(r))
    out_groups, enc_off, enc_rows, term_worker, term_msg = [], [0], [], [], []
    m = 0
    for key in sorted(groups):
        lists = groups[key]
        length = max(len(v) for v in lists.values())
        out_groups.append((key, {i: list(v) for i, v in sorted(lists.items())}, length))
        for j in range(length):
            for i in sorted(lists):
                if j < len(lists[i]):
                    enc_rows.append(lists[i][j])
                    term_worker.append(i)
                    term_msg.append(m)
            enc_off.append(len(enc_rows))
            m += 1
    return Plan(new_assign, out_groups, np.array(enc_off, dtype=np.int64), np.array(enc_rows, dtype=np.int32),
                np.array(term_worker, dtype=np.int32), np.array(term_msg, dtype=np.int32), m, len(enc_rows))


def encode(A: np.ndarray, p: Plan) -> np.ndarray:
    """The multicast rows: message m is the fp32 sum of its terms' rows, in order."""
    A = np.asarray(A, dtype=np.float32)
    M = np.zeros((p.coded_rows, A.shape[1]), dtype=np.float32)
    for m in range(p.coded_rows):
        terms = p.enc_rows[p.enc_off[m]:p.enc_off[m + 1]]
        acc = A[terms[0]].copy()
        for r in terms[1:]:
            acc = acc + A[r]
        M[m] = acc
    return M


def decode(A: np.ndarray, M: np.ndarray, p: Plan) -> np.ndarray:
    """Worker term_worker[d] recovers row enc_rows[d]: its message minus the
    other members' rows (all in its cache), subtracted in order."""
    A = np.asarray(A, dtype=np.float32)
    out = np.empty((len(p.enc_rows), A.shape[1]), dtype=np.float32)
    for d in range(len(p.enc_rows)):
        m = p.term_msg[d]
        acc = M[m].copy()
        for t in range(p.enc_off[m], p.enc_off[m + 1]):
            if t != d:
                acc = acc - A[p.enc_rows[t]]
        out[d] = acc
    return out


def commit(state: State, p: Plan) -> State:
    """The cache update rule for iteration t+1."""
    cached = _apply_cache_rule(state.n, state.q, state.cache_rows, state.seed, state.t + 1, p.new_assign,
                               state.cached)
    return State(state.n, state.q, state.cache_rows, state.seed, state.t + 1, p.new_assign, cached)


def rate_uncoded(n: int, q: int, s: float) -> float:
    """eq. r1: R_u = q (1 - s/q) rows per iteration."""
    return q * (1.0 - s / q)


def _p(n: int, q: int, s: float) -> float:
    return (s - q / n) / (q - q / n)


def rate_coded_sum(n: int, q: int, s: float) -> float:
    """eq. rate1: R_c = sum_{i>=2} C(n,i) (q/n) ((i-1)/n) p^(i-2) (1-p)^(n-i+1)."""
    p = _p(n, q, s)
    if p == 0.0:                       # only the pairs' term is left
        return math.comb(n, 2) * (q / n) * (1 / n)
    if p == 1.0:                       # every cache holds everything: nothing to send
        return 0.0
    total = 0.0
    for i in range(2, n + 1):          # terms in log space: C(n, i) overflows a double for large n
        lc = math.lgamma(n + 1) - math.lgamma(i + 1) - math.lgamma(n - i + 1)
        total += math.exp(lc + (i - 2) * math.log(p) + (n - i + 1) * math.log1p(-p)) * (q / n) * ((i - 1) / n)
    return total


def rate_coded_closed(n: int, q: int, s: float) -> float:
    """eq. r2: R_c = q/(n p)^2 [(1-p)^(n+1) + (n-1) p (1-p) - (1-p)^2], p > 0."""
    p = _p(n, q, s)
    return q / (n * p) ** 2 * ((1 - p) ** (n + 1) + (n - 1) * p * (1 - p) - (1 - p) ** 2)
