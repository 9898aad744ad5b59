"""Device ceilings of the GPU the library runs on (calib/ceilings.hip), the
figures the kernels' design notes compare against besides the published
peaks: HBM read and write bandwidth, the row-window read patterns of the
worker kernels, the memory pattern of the bf16 single pass, and sustained
matrix-instruction and fp64 vector rates."""
from __future__ import annotations

import ctypes
import os

from .build import CALIB_PATH

_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(CALIB_PATH):
            raise OSError(f"{CALIB_PATH} is not built (run __graft_entry__.build())")
        _lib = ctypes.CDLL(CALIB_PATH)
        p, i32, i64, f = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        _lib.calib_read.argtypes = [p, i64, i32, i32, p, f]
        _lib.calib_write.argtypes = [p, i64, i32, i32, i32, f]
        _lib.calib_read_rows.argtypes = [p, i64, i32, i32, i32, p, f]
        _lib.calib_rate.argtypes = [i32, i32, i32, i32, p, p, f]
        _lib.calib_tile_pattern.argtypes = [p, p, i64, i64, i32, i32, i32, i32, f]
        for fn in ("calib_read", "calib_write", "calib_read_rows", "calib_rate", "calib_tile_pattern"):
            getattr(_lib, fn).restype = ctypes.c_int32
    return _lib


def _ms(fn, *args) -> float:
    ms = ctypes.c_float()
    rc = fn(*args, ctypes.byref(ms))
    if rc:
        raise RuntimeError(f"{fn.__name__} failed ({rc})")
    return ms.value


def ceilings(read_bytes: int = 3 * 2 ** 30, reps: int = 20) -> dict:
    """Measures every ceiling once; returns a JSON-ready dict."""
    import torch

    h = lib()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    scratch = torch.zeros(16, dtype=torch.float32, device="cuda")
    buf = torch.ones(read_bytes // 4, dtype=torch.float32, device="cuda")
    out = {"device": torch.cuda.get_device_name(0), "compute_units": cus}
    rd = {}
    for size in (448 * 2 ** 20, read_bytes):
        best = None
        for blocks in (cus * 4, cus * 8, cus * 16):
            ms = _ms(h.calib_read, ctypes.c_void_p(buf.data_ptr()), size, blocks, reps, ctypes.c_void_p(scratch.data_ptr()))
            gbs = size / (ms * 1e-3) / 1e9
            best = max(best or 0.0, gbs)
        rd[f"{size // 2 ** 20} MiB"] = best
    out["hbm_read_gbs"] = rd
    wr = {}
    for nt in (0, 1):
        best = 0.0
        for blocks in (cus * 4, cus * 8, cus * 16):
            ms = _ms(h.calib_write, ctypes.c_void_p(buf.data_ptr()), read_bytes, blocks, nt, reps)
            best = max(best, read_bytes / (ms * 1e-3) / 1e9)
        wr["nontemporal" if nt else "plain"] = best
    out["hbm_write_gbs"] = wr
    rows, r = (448 * 2 ** 20) // (4 * 4096), 4096
    names = ["1 row x 16 KB", "4 rows x 4 KB (2 in flight)", "8 rows x 1 KB (8 in flight, LDS)",
             "16 rows x 512 B (4 in flight, LDS)"]
    out["row_window_read_gbs_448MiB"] = {
        names[pat]: rows * r * 4 / (_ms(h.calib_read_rows, ctypes.c_void_p(buf.data_ptr()), rows, r, pat, reps,
                                        ctypes.c_void_p(scratch.data_ptr())) * 1e-3) / 1e9
        for pat in range(4)}
    del buf
    # the bf16 single pass's memory pattern at the dense workload's shape
    q, r = 131072, 16384
    qb = -(-q // 24)
    A = torch.ones(q * r, dtype=torch.bfloat16, device="cuda")
    P = torch.empty(2 * 8 * qb * r, dtype=torch.bfloat16, device="cuda")
    moved = 2 * q * r + 4 * 8 * qb * r
    out["single_pass_pattern_gbs"] = {
        f"reads {1024 // rr} rows x {rr} B, writes {1024 // rw} rows x {rw} B per wave instruction":
            moved / (_ms(h.calib_tile_pattern, ctypes.c_void_p(A.data_ptr()), ctypes.c_void_p(P.data_ptr()), q, r, rr,
                         rw, cus, 5) * 1e-3) / 1e9
        for rr, rw in ((128, 128), (256, 256), (512, 512), (512, 128), (512, 256))}
    del A, P
    rates = {}
    kinds = [("v_mfma_f64_16x16x4f64", 0, 2000), ("v_mfma_f64_4x4x4f64", 1, 4000),
             ("v_mfma_f32_16x16x32_bf16", 2, 4000), ("v_fma_f64", 3, 20000)]
    for name, kind, iters in kinds:
        res = {}
        for wps in (1, 2, 4):
            blocks = cus * wps
            o = torch.empty(blocks * 256, dtype=torch.float64, device="cuda")
            flops = ctypes.c_double()
            ms = _ms(h.calib_rate, kind, blocks, iters, 5, ctypes.c_void_p(o.data_ptr()), ctypes.byref(flops))
            res[f"{wps} wave/SIMD"] = flops.value / (ms * 1e-3) / 1e12
        rates[name] = res
    out["rate_tflops"] = rates
    return out
