"""Seeded input generators (NumPy PCG64, one SeedSequence per (seed, stream, chunk)).

Every array the tests and the benchmark feed to the coded pipeline comes from
these functions, so the oracle and the GPU path see identical values.  Nothing
here encodes, multiplies or decodes.
"""
from __future__ import annotations

import concurrent.futures as _cf
import itertools
import os

import numpy as np

# Stream identifiers: one independent random stream per role.
STREAM_A = 1        # data matrix A
STREAM_X = 2        # right-hand side X (product t uses chunk key t)
STREAM_P = 3        # parity rows P of the generator G = [I_k; P]
STREAM_RUNTIME = 4  # worker runtimes (consumed by the counter-based SplitMix64, not by NumPy)
STREAM_NOISE = 5    # label noise of the least-squares workload
STREAM_WSTAR = 6    # ground-truth weights of the least-squares workload
STREAM_PT = 7       # parity rows of the second code (the one applied to A^T)
STREAM_SETS = 10    # survivor sets with a fixed number of parity survivors

ROW_CHUNK = 4096    # rows per independently seeded chunk of a large matrix


def generator(seed: int, stream: int, *extra: int) -> np.random.Generator:
    """A PCG64 generator keyed by (seed, stream, *extra)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), int(stream), *map(int, extra)])))


def gaussian(shape, seed: int, stream: int, *extra: int, std: float = 1.0) -> np.ndarray:
    """float32 i.i.d. N(0, std^2) array drawn from one generator."""
    out = generator(seed, stream, *extra).standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def _chunk_rows(seed, stream, c, cols, std):
    g = generator(seed, stream, 1_000_000 + c)
    out = g.standard_normal((ROW_CHUNK, cols), dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def gaussian_rows(rows: int, cols: int, seed: int, stream: int, *, row0: int = 0,
                  nrows: int | None = None, std: float = 1.0, threads: int | None = None) -> np.ndarray:
    """Rows [row0, row0+nrows) of a rows x cols float32 N(0, std^2) matrix.

    The matrix is defined chunk by chunk (ROW_CHUNK rows per chunk, each chunk
    its own generator), so any row range can be regenerated without drawing
    the whole matrix, and chunks can be drawn in parallel.
    """
    if nrows is None:
        nrows = rows - row0
    if row0 < 0 or nrows < 0 or row0 + nrows > rows:
        raise ValueError("row range outside the matrix")
    out = np.empty((nrows, cols), dtype=np.float32)
    if nrows == 0:
        return out
    c_first, c_last = row0 // ROW_CHUNK, (row0 + nrows - 1) // ROW_CHUNK

    def fill(c):
        blk = _chunk_rows(seed, stream, c, cols, std)
        lo = max(row0, c * ROW_CHUNK)
        hi = min(row0 + nrows, (c + 1) * ROW_CHUNK)
        out[lo - row0:hi - row0] = blk[lo - c * ROW_CHUNK:hi - c * ROW_CHUNK]

    chunks = range(c_first, c_last + 1)
    nthreads = threads or min(16, len(os.sched_getaffinity(0)))
    if len(chunks) > 1 and nthreads > 1:
        with _cf.ThreadPoolExecutor(nthreads) as ex:
            list(ex.map(fill, chunks))
    else:
        for c in chunks:
            fill(c)
    return out


def integers(shape, seed: int, stream: int, *extra: int, lo: int = -3, hi: int = 3) -> np.ndarray:
    """float32 array of i.i.d. integers uniform on [lo, hi] (exact in bf16/fp32)."""
    return generator(seed, stream, *extra).integers(lo, hi + 1, size=shape).astype(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bfloat16 bit patterns of float32 x, rounded to nearest even."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_from_bits(bits: np.ndarray) -> np.ndarray:
    """float32 values of uint16 bfloat16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 array holding x rounded to bfloat16 (round to nearest even)."""
    return bf16_from_bits(bf16_bits(x))


def parity_matrix(n: int, k: int, seed: int, stream: int = STREAM_P, dtype: str = "f32") -> np.ndarray:
    """(n-k) x k float64 array of i.i.d. N(0,1) parity coefficients.

    The values are rounded to the device compute dtype ("f32" or "bf16") so the
    encoder and every decoder use exactly the same code.
    """
    p = gaussian((n - k, k), seed, stream)
    if dtype == "bf16":
        p = bf16_round(p)
    elif dtype != "f32":
        raise ValueError(dtype)
    return p.astype(np.float64)


def integer_parity_matrix(n: int, k: int, seed: int, stream: int = STREAM_P, lo: int = -2, hi: int = 2) -> np.ndarray:
    """(n-k) x k float64 array of small integers (exact encode in fp32/bf16)."""
    return integers((n - k, k), seed, stream, lo=lo, hi=hi).astype(np.float64)


def worst_decode_condition(P: np.ndarray) -> float:
    """Largest 2-norm condition number over every square sub-block of P.

    For a systematic code G = [I_k; P] the decode system of a survivor set is
    the sub-block of P on the parity survivors' rows and the missing
    systematic blocks' columns, so this bounds every decode of the code.
    The enumeration is exhaustive (sum over m of C(n-k, m) C(k, m) blocks),
    meant for small codes.
    """
    p, k = P.shape
    worst = 1.0
    for m in range(1, p + 1):
        cols = np.array(list(itertools.combinations(range(k), m)))
        for rows in itertools.combinations(range(p), m):
            sv = np.linalg.svd(P[list(rows)][:, cols].transpose(1, 0, 2), compute_uv=False)
            worst = max(worst, float(np.max(sv[:, 0] / sv[:, -1])))
    return worst


def conditioned_parity_matrix(n: int, k: int, seed: int, candidates: int, stream: int = STREAM_P,
                              dtype: str = "f32", pick: int | None = None):
    """The best of `candidates` seeded N(0,1) parity matrices by worst decode
    condition number (candidate c is drawn with key c and rounded to dtype).
    With `pick`, only that candidate is drawn and certified.
    Returns (P, candidate, worst condition number)."""
    best = None
    for c in ([pick] if pick is not None else range(candidates)):
        P = gaussian((n - k, k), seed, stream, c)
        if dtype == "bf16":
            P = bf16_round(P)
        elif dtype != "f32":
            raise ValueError(dtype)
        P = P.astype(np.float64)
        w = worst_decode_condition(P)
        if best is None or w < best[2]:
            best = (P, c, w)
    return best



def exact_parity_sets(n: int, k: int, m: int, batch: int, seed: int) -> np.ndarray:
    """batch x k int32 survivor sets, each with exactly m parity workers (of
    k..n-1) and k - m systematic ones (of 0..k-1), drawn uniformly and
    independently (repeats allowed), each row in a random order.  Inputs for
    measuring the decode's cost against the number of missing blocks."""
    if not (0 <= m <= min(k, n - k)):
        raise ValueError("need 0 <= m <= min(k, n - k)")
    g = generator(seed, STREAM_SETS, m)
    out = np.empty((batch, k), dtype=np.int32)
    for b in range(batch):
        sys_ = g.choice(k, size=k - m, replace=False)
        par = k + g.choice(n - k, size=m, replace=False)
        row = np.concatenate([sys_, par]).astype(np.int32)
        g.shuffle(row)
        out[b] = row
    return out
