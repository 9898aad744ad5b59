"""Plain fp64 CPU oracle for (n,k) MDS-coded matrix multiplication.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the library's product
path never calls it and shares no code with it.

It follows Lee, Lam, Pedarsani, Papailiopoulos, Ramchandran, "Speeding Up
Distributed Machine Learning Using Codes" (IEEE Trans. IT; arXiv 1512.02673):

* Sec. III-A (coded computation; the (n,k) MDS construction and its footnote
  on zero-row padding): pad A with zero rows to a multiple of k, split it into
  k row-blocks, apply the code to each element of the blocks to get n coded
  blocks (the first k equal the originals for a systematic code), let worker i
  compute its coded block times X, and recover A.X from any k results by
  decoding and concatenating.
* Sec. III-B, eq. (mds_coded): the MDS-coded runtime is the k-th order
  statistic of the n worker runtimes, so the survivors are the k fastest.
* Sec. III-C and eq. (shifted_exp): a task split into l pieces takes T0/l with
  P(T0 <= t) = 1 - exp(-mu (t - 1)); coded tasks use l = k.
* Sec. III-E, eq. (exact_gradient): gradient descent for least squares with
  the two products A.x and A^T.z each computed by its own coded product.

Everything is computed in float64 from inputs that are exactly representable
in the device dtype.  There is no blocking, fusion or reordering beyond the
definitions above.
"""
from __future__ import annotations

import math

import numpy as np

MASK64 = (1 << 64) - 1
SPLITMIX_GAMMA = 0x9E3779B97F4A7C15

# ---------------------------------------------------------------------------
# Sec. III-A: padding, splitting, systematic generator, encoding
# ---------------------------------------------------------------------------


def block_rows(q: int, k: int) -> int:
    """Rows per block after zero-row padding of q rows to a multiple of k (Sec. III-A footnote)."""
    return -(-q // k)


def pad_and_split(A: np.ndarray, k: int) -> np.ndarray:
    """Append zero rows to A until k divides its row count, then cut it into k
    equal row-blocks A_1..A_k (Sec. III-A and its footnote).  Returns (k, qb, r) float64."""
    A = np.asarray(A, dtype=np.float64)
    q, r = A.shape
    qb = block_rows(q, k)
    padded = np.zeros((k * qb, r), dtype=np.float64)
    padded[:q] = A
    return padded.reshape(k, qb, r)


def systematic_generator(P: np.ndarray) -> np.ndarray:
    """Generator G = [I_k; P] of a systematic code: coded block i equals A_i for
    i <= k (Sec. III-A), the n-k parity rows come from P."""
    P = np.asarray(P, dtype=np.float64)
    k = P.shape[1]
    return np.vstack([np.eye(k), P])


def encode(G: np.ndarray, blocks: np.ndarray) -> np.ndarray:
    """Coded blocks A'_i = sum_j G[i, j] A_j: the (n,k) code applied to every
    element of the k sub-matrices (Sec. III-A).  Returns (n, qb, r) float64."""
    n, k = G.shape
    assert blocks.shape[0] == k
    coded = np.zeros((n,) + blocks.shape[1:], dtype=np.float64)
    for i in range(n):
        for j in range(k):
            if G[i, j] != 0.0:
                coded[i] += G[i, j] * blocks[j]
    return coded


def worker_products(coded: np.ndarray, X: np.ndarray) -> np.ndarray:
    """Local function of worker i: its stored coded block times the multicast
    input, y_i = A'_i X (Sec. III-A, protocol paragraph).  Returns (n, qb, s)."""
    X = np.asarray(X, dtype=np.float64)
    if X.ndim == 1:
        X = X[:, None]
    return np.stack([coded[i] @ X for i in range(coded.shape[0])])


# ---------------------------------------------------------------------------
# Sec. III-B/III-C: runtimes and the survivor set
# ---------------------------------------------------------------------------


def splitmix64_next(state: int) -> tuple[int, int]:
    """One step of SplitMix64 (Steele, Lea, Flood, OOPSLA 2014): advance the
    state by the golden-ratio increment, then apply the 64-bit finaliser."""
    state = (state + SPLITMIX_GAMMA) & MASK64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return state, z ^ (z >> 31)


def splitmix64_output(seed: int, index: int) -> int:
    """Output number `index` (0-based) of SplitMix64 seeded with `seed`.

    Its state after index+1 steps is seed + (index+1)*gamma, so any output can
    be produced directly: the generator is counter-based by construction."""
    state = (seed + (index * SPLITMIX_GAMMA)) & MASK64
    return splitmix64_next(state)[1]


def runtime_counter(stream: int, draw: int, worker: int) -> int:
    """Counter of worker `worker` in draw `draw` of random stream `stream`."""
    if not (0 <= worker < (1 << 16) and 0 <= draw < (1 << 40) and 0 <= stream < 256):
        raise ValueError("counter field out of range")
    return (stream << 56) | (draw << 16) | worker


def runtime_word(seed: int, stream: int, draw: int, worker: int) -> int:
    return splitmix64_output(seed & MASK64, runtime_counter(stream, draw, worker))


def uniform_open01(word: int) -> float:
    """A uniform on (0,1) from the top 53 bits of a 64-bit word."""
    return ((word >> 11) + 0.5) * 2.0 ** -53


RUNTIME_STREAM = 4


def worker_runtimes(n: int, k: int, seed: int, draw: int, shift: float = 1.0, rate: float = 1.0,
                    stream: int = RUNTIME_STREAM) -> np.ndarray:
    """Runtimes of the n coded tasks of one product (Sec. III-C): the mother
    runtime is shifted-exponential, T0 = shift + E/rate with E ~ Exp(1)
    (eq. shifted_exp), and each of the n tasks carries 1/k of the work, so it
    takes T0/k (the scaled distribution F(k t))."""
    T = np.empty(n, dtype=np.float64)
    for i in range(n):
        u = uniform_open01(runtime_word(seed, stream, draw, i))
        T[i] = (shift + (-math.log(u)) / rate) / k
    return T


def draw_survivors(n: int, k: int, seed: int, draw: int, shift: float = 1.0, rate: float = 1.0,
                   stream: int = RUNTIME_STREAM) -> tuple[np.ndarray, float]:
    """The first k workers to finish and the overall runtime T_(k) (Sec. III-B,
    eq. mds_coded).  Equal runtimes go to the lower worker index.  Returns the
    survivor indices in ascending order (0-based) and T_(k)."""
    T = worker_runtimes(n, k, seed, draw, shift, rate, stream)
    order = sorted(range(n), key=lambda i: (T[i], i))
    S = np.array(sorted(order[:k]), dtype=np.int32)
    return S, float(T[order[k - 1]])


def draw_survivor_sets(n: int, k: int, seed: int, batch: int, min_parity: int = 0, first_draw: int = 0,
                       shift: float = 1.0, rate: float = 1.0) -> tuple[np.ndarray, int]:
    """`batch` distinct survivor sets with at least `min_parity` parity workers:
    draws first_draw, first_draw+1, ... are taken in order and a set is kept
    when it qualifies and differs from every set kept before.  Returns
    (batch, k) int32 sets and the next unused draw index.  Asking for more
    sets than exist (sum over m >= min_parity of C(k, m) C(n-k, m): m parity
    workers in, m systematic ones out) raises ValueError."""
    available = sum(math.comb(k, m) * math.comb(n - k, m) for m in range(min_parity, min(k, n - k) + 1))
    if batch > available:
        raise ValueError(f"only {available} distinct survivor sets have >= {min_parity} parity workers")
    seen = set()
    sets = []
    d = first_draw
    while len(sets) < batch:
        S, _ = draw_survivors(n, k, seed, d, shift, rate)
        d += 1
        if int(np.sum(S >= k)) < min_parity:
            continue
        key = tuple(int(v) for v in S)
        if key in seen:
            continue
        seen.add(key)
        sets.append(S)
    return np.array(sets, dtype=np.int32).reshape(batch, k), d


# ---------------------------------------------------------------------------
# Decoding: dec(indices, results) of Sec. III-A (the paper leaves the algorithm
# open; any k coded results determine the k blocks because every k x k
# sub-matrix of an MDS generator is invertible, so decoding is the solution of
# G_S B = Y_S, computed here by Gaussian elimination with partial pivoting).
# ---------------------------------------------------------------------------


def lu_factor(M: np.ndarray) -> tuple[np.ndarray, np.ndarray, int]:
    """Doolittle LU with partial pivoting (largest |entry| in the column, lowest
    row on ties).  Returns (LU packed, pivot row of each step, info) where info
    is 0 or the 1-based step whose pivot is exactly zero (LAPACK getrf's rule)."""
    LU = np.array(M, dtype=np.float64, copy=True)
    m = LU.shape[0]
    piv = np.arange(m)
    info = 0
    for j in range(m):
        p = j
        for i in range(j + 1, m):
            if abs(LU[i, j]) > abs(LU[p, j]):
                p = i
        piv[j] = p
        if p != j:
            LU[[j, p]] = LU[[p, j]]
        if LU[j, j] == 0.0:
            if info == 0:
                info = j + 1
            continue
        for i in range(j + 1, m):
            LU[i, j] /= LU[j, j]
            LU[i, j + 1:] -= LU[i, j] * LU[j, j + 1:]
    return LU, piv, info


def lu_solve(LU: np.ndarray, piv: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Solve M Z = B from lu_factor's output (row swaps, then L, then U)."""
    Z = np.array(B, dtype=np.float64, copy=True)
    m = LU.shape[0]
    for j in range(m):
        if piv[j] != j:
            Z[[j, piv[j]]] = Z[[piv[j], j]]
    for i in range(m):
        for j in range(i):
            Z[i] -= LU[i, j] * Z[j]
    for i in range(m - 1, -1, -1):
        for j in range(i + 1, m):
            Z[i] -= LU[i, j] * Z[j]
        Z[i] /= LU[i, i]
    return Z


class DecodeError(ValueError):
    def __init__(self, msg, info=0):
        super().__init__(msg)
        self.info = info


def decode(G: np.ndarray, indices, results, q: int) -> np.ndarray:
    """dec(indices, results) (Sec. III-A): `indices` is the sequence of worker
    indices in arrival order and `results[c]` is worker indices[c]'s product.
    The first k results form a decodable set of the MDS code; solving
    G_S B = Y_S recovers the k block products A_j X, whose concatenation
    without the padding rows is A X (q x s)."""
    n, k = G.shape
    idx = [int(i) for i in indices]
    if len(idx) < k:
        raise DecodeError("fewer than k results")
    idx = idx[:k]
    if len(set(idx)) != k or min(idx) < 0 or max(idx) >= n:
        raise DecodeError("indices must be k distinct workers in [0, n)")
    Ys = [np.asarray(results[c], dtype=np.float64) for c in range(k)]
    Ys = [y[:, None] if y.ndim == 1 else y for y in Ys]
    qb, s = Ys[0].shape
    GS = G[idx, :]
    LU, piv, info = lu_factor(GS)
    if info:
        raise DecodeError("singular survivor sub-matrix", info)
    B = lu_solve(LU, piv, np.stack([y.reshape(-1) for y in Ys]))
    return B.reshape(k * qb, s)[:q]


def decode_from_all(G: np.ndarray, S, Y: np.ndarray, q: int) -> np.ndarray:
    """decode() with the survivors' rows taken from the full (n, qb, s) result array."""
    return decode(G, list(S), [Y[i] for i in S], q)


def coded_matmul(A: np.ndarray, X: np.ndarray, G: np.ndarray, seed: int, draw: int,
                 shift: float = 1.0, rate: float = 1.0):
    """One coded product (Sec. III-A protocol): encode, all n worker products,
    wait for the first k (Sec. III-B), decode.  Returns (A X, survivors, T_(k))."""
    n, k = G.shape
    coded = encode(G, pad_and_split(A, k))
    Y = worker_products(coded, X)
    S, T = draw_survivors(n, k, seed, draw, shift, rate)
    return decode_from_all(G, S, Y, A.shape[0]), S, T


def plain_product(A: np.ndarray, X: np.ndarray) -> np.ndarray:
    """The uncoded result A X in float64: what every decodable set must return."""
    X = np.asarray(X, dtype=np.float64)
    if X.ndim == 1:
        X = X[:, None]
    return np.asarray(A, dtype=np.float64) @ X


# ---------------------------------------------------------------------------
# Sec. III-E: coded gradient descent for least squares
# ---------------------------------------------------------------------------


def coded_gd(A: np.ndarray, y: np.ndarray, x0: np.ndarray, G1: np.ndarray, G2: np.ndarray, eta: float,
             iters: int, seed: int, shift: float = 1.0, rate: float = 1.0, record=None):
    """x(t+1) = x(t) - eta A^T (A x(t) - y) (eq. exact_gradient), where A x(t)
    is an (n,k1)-coded product of A and A^T z(t) an (n,k2)-coded product of
    A^T (Sec. III-E).  The product in iteration t uses survivor draw 2t, the
    transposed product draw 2t+1.  Returns the final x."""
    A = np.asarray(A, dtype=np.float64)
    q, r = A.shape
    k1, k2 = G1.shape[1], G2.shape[1]
    n1, n2 = G1.shape[0], G2.shape[0]
    coded1 = encode(G1, pad_and_split(A, k1))
    coded2 = encode(G2, pad_and_split(A.T, k2))
    x = np.asarray(x0, dtype=np.float64).reshape(r, 1).copy()
    yv = np.asarray(y, dtype=np.float64).reshape(q, 1)
    for t in range(iters):
        S1, _ = draw_survivors(n1, k1, seed, 2 * t, shift, rate)
        Ax = decode_from_all(G1, S1, worker_products(coded1, x), q)
        z = Ax - yv
        S2, _ = draw_survivors(n2, k2, seed, 2 * t + 1, shift, rate)
        g = decode_from_all(G2, S2, worker_products(coded2, z), r)
        x = x - eta * g
        if record is not None:
            record.append(x[:, 0].copy())
    return x[:, 0]
