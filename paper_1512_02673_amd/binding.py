"""ctypes binding of libcoded_mi355x.so: the C ABI's calls under the same names.

Argument marshalling only: shapes, strides and data pointers are read from
torch tensors, the current torch stream is passed as the HIP stream, and every
step of the coded product runs in the library.  Loading fails loudly when the
library has not been built.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

from .build import LIB_PATH

CODED_OK, CODED_ERR_ARG, CODED_ERR_SHAPE, CODED_ERR_TOO_FEW, CODED_ERR_SINGULAR, CODED_ERR_HIP, \
    CODED_ERR_UNSUPPORTED = range(7)
CODED_F32, CODED_BF16, CODED_F64 = 0, 1, 2
CODED_MAX_N = 128
CODED_NOALLOC_SCRATCH_BYTES = 64 << 20
CODED_PLANES_LO_BF16 = 3   # fp32 codes: hi plane fp32, lo plane bfloat16

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "coded.h")

_c_i32, _c_i64, _c_u64, _c_dbl, _c_p = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p

_SIGNATURES = {
    "coded_code_bytes": (_c_i32, [_c_i32, _c_i32, _c_p]),
    "coded_code_create": (_c_i32, [_c_i32, _c_i32, _c_p, _c_i32, _c_p, _c_i64, ctypes.POINTER(_c_p)]),
    "coded_code_destroy": (_c_i32, [_c_p]),
    "coded_code_info": (_c_i32, [_c_p, _c_p, _c_p, _c_p]),
    "coded_sizes": (_c_i32, [_c_p, _c_i32, _c_i32, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p]),
    "coded_encode": (_c_i32, [_c_p, _c_i32, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p]),
    "coded_worker_mm": (_c_i32, [_c_p, _c_i32, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_i64, _c_i64, _c_p,
                                 _c_p, _c_i32, _c_p, _c_p]),
    "coded_encode_worker_mm": (_c_i32, [_c_p, _c_i32, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_i64, _c_i64,
                                        _c_p, _c_i32, _c_p, _c_p]),
    "coded_decode": (_c_i32, [_c_p, _c_p, _c_i32, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_i64, _c_p, _c_p]),
    "coded_decode_batched": (_c_i32, [_c_p, _c_p, _c_i32, _c_p, _c_i32, _c_i64, _c_i64, _c_p, _c_i64, _c_i64,
                                      _c_p, _c_p]),
    "coded_draw_survivors": (_c_i32, [_c_i32, _c_i32, _c_u64, _c_u64, _c_dbl, _c_dbl, _c_p, _c_p]),
    "coded_draw_survivor_sets": (_c_i32, [_c_i32, _c_i32, _c_u64, _c_u64, _c_i32, _c_i32, _c_p, _c_p]),
    "coded_matmul": (_c_i32, [_c_p, _c_i32, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_i32, _c_p, _c_i64, _c_i64,
                              _c_u64, _c_u64, _c_dbl, _c_dbl, _c_p, _c_p, _c_p, _c_i64, _c_p, _c_p, _c_p]),
    "coded_matmul_noalloc": (_c_i32, [_c_p, _c_i32, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_i32, _c_p, _c_i64, _c_i64,
                                      _c_u64, _c_u64, _c_dbl, _c_dbl, _c_p, _c_p, _c_p, _c_i64, _c_p, _c_p]),
    "coded_straggler_matmul": (_c_i32, [_c_p, _c_i32, _c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_i64, _c_i64,
                                        _c_u64, _c_u64, _c_dbl, _c_dbl, _c_dbl, _c_i32, _c_p, _c_i32, _c_p, _c_p,
                                        _c_i64, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "coded_transpose": (_c_i32, [_c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_i64, _c_p]),
    "coded_shuffle_create": (_c_i32, [_c_i32, _c_i64, _c_i64, _c_u64, _c_p]),
    "coded_shuffle_destroy": (_c_i32, [_c_p]),
    "coded_shuffle_state": (_c_i32, [_c_p, _c_p, _c_p, _c_p]),
    "coded_shuffle_plan": (_c_i32, [_c_p, _c_p, _c_p]),
    "coded_shuffle_tables": (_c_i32, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "coded_shuffle_commit": (_c_i32, [_c_p]),
    "coded_shuffle_encode": (_c_i32, [_c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_i64, _c_i64, _c_p, _c_i64, _c_p]),
    "coded_shuffle_decode": (_c_i32, [_c_p, _c_i64, _c_i64, _c_i64, _c_p, _c_i64, _c_p, _c_p, _c_p, _c_i64, _c_i64,
                                      _c_p, _c_i64, _c_p]),
    "coded_gd_sizes": (_c_i32, [_c_p, _c_p, _c_i64, _c_i64, _c_p]),
    "coded_gd_step": (_c_i32, [_c_p, _c_p, _c_p, _c_i64, _c_p, _c_p, _c_i64, _c_p, _c_i64, _c_i64, _c_p, _c_p, _c_dbl,
                               _c_u64, _c_u64, _c_dbl, _c_dbl, _c_p, _c_p, _c_p, _c_p]),
    "coded_simulate_runtimes": (_c_i32, [_c_i32, _c_i32, _c_u64, _c_u64, _c_i64, _c_dbl, _c_dbl, _c_p, _c_p, _c_p,
                                         _c_p]),
    "coded_optimal_k": (_c_i32, [_c_i32, _c_dbl, _c_p, _c_p, _c_p]),
    "coded_status_string": (ctypes.c_char_p, [_c_i32]),
    "coded_last_error": (ctypes.c_char_p, []),
    "coded_version": (ctypes.c_char_p, []),
}

_lib = None


class CodedError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run paper_1512_02673_amd.build.build() "
                               "(or __graft_entry__.build()) first")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(h, name)
            f.restype = res
            f.argtypes = args
        _lib = h
    return _lib


def header_functions() -> list[str]:
    """Names of the functions include/coded.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(coded_[a-z0-9_]+)\s*\(", text)))


def status_string(status: int) -> str:
    return lib().coded_status_string(status).decode()


def last_error() -> str:
    return lib().coded_last_error().decode()


def version() -> str:
    return lib().coded_version().decode()


def _check(status: int) -> None:
    if status != CODED_OK:
        raise CodedError(status, last_error())


# ---------------------------------------------------------------- host-only calls

def coded_draw_survivors(n: int, k: int, seed: int, draw: int, shift: float = 1.0, rate: float = 1.0):
    """(survivors ascending int32[k], T_(k)) of one draw."""
    out = np.zeros(k, dtype=np.int32)
    t = ctypes.c_double()
    _check(lib().coded_draw_survivors(n, k, seed, draw, shift, rate, out.ctypes.data, ctypes.addressof(t)))
    return out, t.value


def coded_draw_survivor_sets(n: int, k: int, seed: int, batch: int, min_parity: int = 0, first_draw: int = 0):
    """(sets int32[batch, k], next unused draw)."""
    out = np.zeros((batch, k), dtype=np.int32)
    nxt = ctypes.c_uint64()
    _check(lib().coded_draw_survivor_sets(n, k, seed, first_draw, batch, min_parity, out.ctypes.data,
                                          ctypes.addressof(nxt)))
    return out, nxt.value


def coded_optimal_k(n: int, rate: float):
    """(k*, T*, best integer k) of Lemma 2."""
    ks, ts, kb = ctypes.c_double(), ctypes.c_double(), ctypes.c_int32()
    _check(lib().coded_optimal_k(n, rate, ctypes.addressof(ks), ctypes.addressof(ts), ctypes.addressof(kb)))
    return ks.value, ts.value, kb.value


# ---------------------------------------------------------------- device calls

def _torch():
    import torch
    return torch


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t) -> int:
    torch = _torch()
    return {torch.float32: CODED_F32, torch.bfloat16: CODED_BF16, torch.float64: CODED_F64}[t.dtype]


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _matrix(t, name):
    """(rows, cols, row stride) of a 1-D (column) or row-major 2-D tensor."""
    if t.dim() == 1:
        if t.stride(0) != 1:
            raise ValueError(f"{name} must be contiguous")
        return t.shape[0], 1, 1
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be 1-D or row-major 2-D")
    return t.shape[0], t.shape[1], max(t.stride(0), 1)


def coded_code_bytes(n: int, k: int) -> int:
    """Bytes of the device buffer an (n,k) code needs."""
    b = ctypes.c_int64()
    _check(lib().coded_code_bytes(n, k, ctypes.addressof(b)))
    return b.value


class Code:
    """An (n,k) code: G = [I_k; P] on host, and on the device in a buffer this
    object owns (a torch tensor on the current device) and passes to
    coded_code_create."""

    def __init__(self, n: int, k: int, G: np.ndarray, planes: int = 2):
        G = np.ascontiguousarray(G, dtype=np.float64)
        if G.shape != (n, k):
            raise ValueError("G must be n x k")
        nbytes = coded_code_bytes(n, k)
        self.device_buf = _torch().empty(nbytes, dtype=_torch().uint8, device="cuda")
        h = ctypes.c_void_p()
        _check(lib().coded_code_create(n, k, G.ctypes.data, planes, ctypes.c_void_p(self.device_buf.data_ptr()),
                                       nbytes, ctypes.byref(h)))
        self.handle = h
        self.n, self.k, self.planes = n, k, planes
        self.G = G

    @classmethod
    def systematic(cls, P: np.ndarray, planes: int = 2) -> "Code":
        P = np.asarray(P, dtype=np.float64)
        k = P.shape[1]
        return cls(k + P.shape[0], k, np.vstack([np.eye(k), P]), planes)

    def qb(self, q: int) -> int:
        return -(-q // self.k)

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            lib().coded_code_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def coded_sizes(code: Code, dt: int, y_dt: int, q: int, r: int, s: int):
    """(parity_bytes, y_bytes, matmul workspace_bytes, worker workspace_bytes)."""
    pb, yb, wb, ww = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(lib().coded_sizes(code.handle, dt, y_dt, q, r, s, ctypes.addressof(pb), ctypes.addressof(yb),
                             ctypes.addressof(wb), ctypes.addressof(ww)))
    return pb.value, yb.value, wb.value, ww.value


def coded_encode(code: Code, A, parity, stream=None) -> None:
    q, r, lda = _matrix(A, "A")
    _check(lib().coded_encode(code.handle, _dtype_code(A), _ptr(A), q, r, lda, _ptr(parity), _stream(stream)))


def worker_workspace(code: Code, A, X):
    """A device buffer of the worker workspace size for these operands (None if 0 bytes)."""
    torch = _torch()
    q, r, _ = _matrix(A, "A")
    _, s, _ = _matrix(X, "X")
    y_dt = CODED_F32 if _dtype_code(A) == CODED_BF16 else CODED_F64
    nbytes = coded_sizes(code, _dtype_code(A), y_dt, q, r, s)[3]
    return torch.empty(nbytes, dtype=torch.uint8, device=A.device) if nbytes else None


def matmul_workspace(code: Code, A, X):
    """A device buffer of coded_matmul's workspace size for these operands."""
    torch = _torch()
    q, r, _ = _matrix(A, "A")
    _, s, _ = _matrix(X, "X")
    y_dt = CODED_F32 if _dtype_code(A) == CODED_BF16 else CODED_F64
    nbytes = coded_sizes(code, _dtype_code(A), y_dt, q, r, s)[2]
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=A.device)


def coded_worker_mm(code: Code, A, parity, X, Y, worker_mask=None, workspace="auto", stream=None) -> None:
    """workspace: a device buffer of coded_sizes' worker workspace bytes, None (bf16: vector
    kernel), or "auto" (allocated here when needed)."""
    q, r, lda = _matrix(A, "A")
    rx, s, ldx = _matrix(X, "X")
    if rx != r:
        raise ValueError("X must have r rows")
    mask = None
    if worker_mask is not None:
        m = np.ascontiguousarray(worker_mask, dtype=np.uint8)
        if m.shape != (code.n,):
            raise ValueError("worker_mask must have n entries")
        mask = m.ctypes.data_as(ctypes.c_void_p)
    if isinstance(workspace, str):
        workspace = worker_workspace(code, A, X)
    _check(lib().coded_worker_mm(code.handle, _dtype_code(A), _ptr(A), q, r, lda, _ptr(parity), _ptr(X), s, ldx,
                                 mask, _ptr(Y), _dtype_code(Y), _ptr(workspace), _stream(stream)))


def coded_encode_worker_mm(code: Code, A, parity, X, Y, workspace="auto", stream=None) -> None:
    """Parity blocks and every worker's product in one call (coded_encode, then
    coded_worker_mm for all workers; one pass over A where the kernel serves the shape)."""
    q, r, lda = _matrix(A, "A")
    rx, s, ldx = _matrix(X, "X")
    if rx != r:
        raise ValueError("X must have r rows")
    if isinstance(workspace, str):
        workspace = worker_workspace(code, A, X)
    _check(lib().coded_encode_worker_mm(code.handle, _dtype_code(A), _ptr(A), q, r, lda, _ptr(parity), _ptr(X), s,
                                        ldx, _ptr(Y), _dtype_code(Y), _ptr(workspace), _stream(stream)))


def coded_decode(code: Code, survivors, Y, q: int, out, info, stream=None) -> None:
    sv = np.ascontiguousarray(survivors, dtype=np.int32)
    _, s, ldo = _matrix(out, "out")
    _check(lib().coded_decode(code.handle, sv.ctypes.data_as(ctypes.c_void_p), len(sv), _ptr(Y), _dtype_code(Y), q,
                              s, _ptr(out), ldo, _ptr(info), _stream(stream)))


def coded_decode_batched(code: Code, sets, Y, q: int, out, info, stream=None) -> None:
    """sets: device int32 (batch, k); out: (batch, q) or (batch, q, s) float32."""
    batch = sets.shape[0]
    if out.dim() == 2:
        s, ldo = 1, 1
    else:
        s, ldo = out.shape[2], out.stride(1)
    _check(lib().coded_decode_batched(code.handle, _ptr(sets), batch, _ptr(Y), _dtype_code(Y), q, s, _ptr(out), ldo,
                                      out.stride(0), _ptr(info), _stream(stream)))


def coded_matmul(code: Code, A, parity, X, out, workspace, info, seed: int, draw: int, parity_ready: bool = True,
                 shift: float = 1.0, rate: float = 1.0, stream=None):
    """One coded product; returns (survivors int32[k], T_(k))."""
    q, r, lda = _matrix(A, "A")
    rx, s, ldx = _matrix(X, "X")
    if rx != r:
        raise ValueError("X must have r rows")
    _, so, ldo = _matrix(out, "out")
    surv = np.zeros(code.k, dtype=np.int32)
    t = ctypes.c_double()
    _check(lib().coded_matmul(code.handle, _dtype_code(A), _ptr(A), q, r, lda, _ptr(parity), int(bool(parity_ready)),
                              _ptr(X), s, ldx, seed, draw, shift, rate, surv.ctypes.data_as(ctypes.c_void_p),
                              ctypes.addressof(t), _ptr(out), ldo, _ptr(workspace), _ptr(info), _stream(stream)))
    return surv, t.value


def coded_matmul_noalloc(code: Code, A, parity, X, out, info, seed: int, draw: int, parity_ready: bool = True,
                         shift: float = 1.0, rate: float = 1.0, stream=None):
    """coded_matmul on the library's static device scratch (no workspace argument,
    nothing allocated); returns (survivors int32[k], T_(k))."""
    q, r, lda = _matrix(A, "A")
    rx, s, ldx = _matrix(X, "X")
    if rx != r:
        raise ValueError("X must have r rows")
    _, so, ldo = _matrix(out, "out")
    surv = np.zeros(code.k, dtype=np.int32)
    t = ctypes.c_double()
    _check(lib().coded_matmul_noalloc(code.handle, _dtype_code(A), _ptr(A), q, r, lda, _ptr(parity),
                                      int(bool(parity_ready)), _ptr(X), s, ldx, seed, draw, shift, rate,
                                      surv.ctypes.data_as(ctypes.c_void_p), ctypes.addressof(t), _ptr(out), ldo,
                                      _ptr(info), _stream(stream)))
    return surv, t.value


def coded_straggler_matmul(code: Code, A, parity, X, Y, out, info, seed: int, draw: int, time_unit_us: float,
                           launch_all: bool = False, workspace="auto", shift: float = 1.0, rate: float = 1.0,
                           stream=None):
    """One coded product with real, timed straggling (blocks until the decode is done).
    Returns (survivors int32[k] in arrival order, timeline float64[n, 3] in microseconds:
    start time, enqueue time, completion seen, -1 where it did not happen, latency in microseconds)."""
    q, r, lda = _matrix(A, "A")
    rx, s, ldx = _matrix(X, "X")
    if rx != r:
        raise ValueError("X must have r rows")
    _, so, ldo = _matrix(out, "out")
    if isinstance(workspace, str):
        workspace = worker_workspace(code, A, X)
    surv = np.zeros(code.k, dtype=np.int32)
    timeline = np.zeros((code.n, 3), dtype=np.float64)
    lat = ctypes.c_double()
    _check(lib().coded_straggler_matmul(code.handle, _dtype_code(A), _ptr(A), q, r, lda, _ptr(parity), _ptr(X), s,
                                        ldx, seed, draw, shift, rate, time_unit_us, int(bool(launch_all)), _ptr(Y),
                                        _dtype_code(Y), _ptr(workspace), _ptr(out), ldo, _ptr(info),
                                        surv.ctypes.data_as(ctypes.c_void_p),
                                        timeline.ctypes.data_as(ctypes.c_void_p), ctypes.addressof(lat),
                                        _stream(stream)))
    return surv, timeline, lat.value


def coded_transpose(A, AT, stream=None) -> None:
    q, r, lda = _matrix(A, "A")
    r2, q2, ldat = _matrix(AT, "AT")
    if (r2, q2) != (r, q):
        raise ValueError("AT must be r x q")
    _check(lib().coded_transpose(_ptr(A), q, r, lda, _ptr(AT), ldat, _stream(stream)))


def coded_gd_sizes(codeA: Code, codeAT: Code, q: int, r: int) -> int:
    wb = ctypes.c_int64()
    _check(lib().coded_gd_sizes(codeA.handle, codeAT.handle, q, r, ctypes.addressof(wb)))
    return wb.value


def coded_gd_step(codeA: Code, codeAT: Code, A, parityA, AT, parityAT, y, x, eta: float, seed: int, iteration: int,
                  workspace, info, shift: float = 1.0, rate: float = 1.0, stream=None):
    """One coded gradient-descent iteration (x updated in place); returns both survivor sets."""
    q, r, lda = _matrix(A, "A")
    _, _, ldat = _matrix(AT, "AT")
    surv = np.zeros(codeA.k + codeAT.k, dtype=np.int32)
    _check(lib().coded_gd_step(codeA.handle, codeAT.handle, _ptr(A), lda, _ptr(parityA), _ptr(AT), ldat,
                               _ptr(parityAT), q, r, _ptr(y), _ptr(x), eta, seed, iteration, shift, rate,
                               _ptr(workspace), _ptr(info), surv.ctypes.data_as(ctypes.c_void_p), _stream(stream)))
    return surv[:codeA.k], surv[codeA.k:]


def coded_simulate_runtimes(n: int, k: int, seed: int, first_draw: int, t_uncoded=None, t_repetition=None,
                            t_mds=None, shift: float = 1.0, rate: float = 1.0, stream=None) -> None:
    """Fill the given device fp64 tensors (equal lengths) with per-draw overall runtimes."""
    outs = [t for t in (t_uncoded, t_repetition, t_mds) if t is not None]
    if not outs:
        return
    count = outs[0].numel()
    if any(t.numel() != count for t in outs):
        raise ValueError("output tensors must have equal lengths")
    _check(lib().coded_simulate_runtimes(n, k, seed, first_draw, count, shift, rate, _ptr(t_uncoded),
                                         _ptr(t_repetition), _ptr(t_mds), _stream(stream)))


# ---------------------------------------------------------------- buffer helpers

def alloc_parity(code: Code, q: int, r: int, dtype, device="cuda"):
    """Parity planes of a q x r input: (planes, n-k, qb, r) of `dtype`; for a
    CODED_PLANES_LO_BF16 code (fp32 only) a flat uint8 buffer holding the fp32
    hi plane followed by the bfloat16 lo plane (see parity_planes)."""
    torch = _torch()
    qb = code.qb(q)
    if code.planes == CODED_PLANES_LO_BF16:
        if dtype != torch.float32:
            raise ValueError("a bfloat16 lo plane is for fp32 inputs")
        return torch.empty(6 * (code.n - code.k) * qb * r, dtype=torch.uint8, device=device)
    return torch.empty((code.planes, code.n - code.k, qb, r), dtype=dtype, device=device)


def parity_planes(code: Code, par, q: int, r: int):
    """(hi, lo) views of a CODED_PLANES_LO_BF16 parity buffer: hi float32 and
    lo bfloat16, each (n-k, qb, r)."""
    torch = _torch()
    shape = (code.n - code.k, code.qb(q), r)
    hb = 4 * shape[0] * shape[1] * shape[2]
    hi = par[:hb].view(torch.float32).view(shape)
    lo = par[hb:].view(torch.bfloat16).view(shape)
    return hi, lo


def alloc_y(code: Code, q: int, s: int, dtype, device="cuda"):
    torch = _torch()
    return torch.empty((code.n, code.qb(q), s), dtype=dtype, device=device)


class Shuffle:
    """Coded-shuffling master state (coded_shuffle_create): n workers, q rows, caches of cache_rows rows."""

    def __init__(self, n: int, q: int, cache_rows: int, seed: int):
        h = ctypes.c_void_p()
        _check(lib().coded_shuffle_create(n, q, cache_rows, seed, ctypes.byref(h)))
        self.handle = h
        self.n, self.q, self.cache_rows, self.seed = n, q, cache_rows, seed

    def state(self):
        """(t, partition int32[q], cache signatures uint64[q])."""
        t = ctypes.c_int64()
        assign = np.zeros(self.q, dtype=np.int32)
        sig = np.zeros(self.q, dtype=np.uint64)
        _check(lib().coded_shuffle_state(self.handle, ctypes.byref(t), assign.ctypes.data_as(ctypes.c_void_p),
                                         sig.ctypes.data_as(ctypes.c_void_p)))
        return t.value, assign, sig

    def plan(self):
        """Plans iteration t+1: (coded_rows, terms)."""
        m, t = ctypes.c_int64(), ctypes.c_int64()
        _check(lib().coded_shuffle_plan(self.handle, ctypes.byref(m), ctypes.byref(t)))
        self.coded_rows, self.terms = m.value, t.value
        return m.value, t.value

    def tables(self):
        """The pending plan: dict of enc_off, enc_rows, term_worker, term_msg, next_assign (host arrays)."""
        out = {"enc_off": np.zeros(self.coded_rows + 1, dtype=np.int64),
               "enc_rows": np.zeros(self.terms, dtype=np.int32),
               "term_worker": np.zeros(self.terms, dtype=np.int32),
               "term_msg": np.zeros(self.terms, dtype=np.int32),
               "next_assign": np.zeros(self.q, dtype=np.int32)}
        _check(lib().coded_shuffle_tables(self.handle, *(out[k].ctypes.data_as(ctypes.c_void_p) for k in
                                                         ("enc_off", "enc_rows", "term_worker", "term_msg",
                                                          "next_assign"))))
        return out

    def commit(self):
        _check(lib().coded_shuffle_commit(self.handle))

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            lib().coded_shuffle_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def coded_shuffle_encode(A, enc_off, enc_rows, M, stream=None) -> None:
    """M (coded_rows x r) from A (q x r fp32) and device copies of the plan's tables."""
    q, r, lda = _matrix(A, "A")
    coded_rows, _, ldm = _matrix(M, "M")
    _check(lib().coded_shuffle_encode(_ptr(A), q, r, lda, _ptr(enc_off), _ptr(enc_rows), coded_rows,
                                      enc_rows.numel(), _ptr(M), ldm, _stream(stream)))


def coded_shuffle_decode(A, M, enc_off, enc_rows, term_msg, out, stream=None) -> None:
    """out (terms x r): each worker's decoded copy of the rows it lacked."""
    q, r, lda = _matrix(A, "A")
    coded_rows, _, ldm = _matrix(M, "M")
    _, _, ldo = _matrix(out, "out")
    _check(lib().coded_shuffle_decode(_ptr(A), q, r, lda, _ptr(M), ldm, _ptr(enc_off), _ptr(enc_rows), _ptr(term_msg),
                                      coded_rows, enc_rows.numel(), _ptr(out), ldo, _stream(stream)))

