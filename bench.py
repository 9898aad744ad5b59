"""Benchmark of (n,k) MDS-coded matrix multiplication on one MI355X.

Default workload (the GEMV regime): A 65536 x 8192 fp32 N(0,1) in k = 12
row-blocks, a systematic (16,12) code with N(0,1) parity, a fresh x (8192)
and a fresh shifted-exponential survivor draw per product, encode done once
before timing.  One step = one coded product: the survivor draw (host), the
16 worker products (one GEMV launch over all blocks) and the decode launch;
the decode of product t overlaps the worker products of product t+1.

Prints one JSON line with the throughput (decoded products/s), the worker
GEMV's HBM roofline fraction (kernel time from HIP events recorded on the
launch stream around every GEMV launch of the timed region) and the fp64
oracle timed on a bounded sample of the same workload on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = "coded A·X decoded products/sec + achieved HBM GB/s (GEMV) / MFMA % (GEMM)"
HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "worker_gemv_traffic_gemv16x12.json")
KERNEL_SOURCES = ["paper_1512_02673_amd/csrc/worker.hip", "paper_1512_02673_amd/csrc/worker_common.h",
                  "paper_1512_02673_amd/csrc/internal.h"]


# Runtime-model kernel: executed VALU instructions per launch from a committed
# rocprofv3 counter summary (SQ_INSTS_VALU), valid for this source hash only.
VALU_FILE = os.path.join(ROOT, "profiles", "runtime_sim_valu_10x5.json")
RUNTIME_SOURCES = ["paper_1512_02673_amd/csrc/runtime.hip", "paper_1512_02673_amd/csrc/internal.h"]
# Vector-issue peak: 256 CUs x 4 SIMDs, one wave64 VALU instruction per SIMD
# every 4 cycles (16 lanes wide) at 2.4 GHz = 614.4 G wave-instructions/s.
ALU_PEAK_G = 256 * 4 * 2.4 / 4


def kernel_source_hash(sources=None) -> str:
    h = hashlib.sha256()
    for p in sources or KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


# Single-pass bf16 encode + worker products: the same kind of summary.
DENSE_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fused_traffic_dense32x24.json")
DENSE_SOURCES = ["paper_1512_02673_amd/csrc/fused_bf16.hip", "paper_1512_02673_amd/csrc/internal.h"]


def measured_traffic(per_launch_algorithmic: float, path=TRAFFIC_FILE, sources=None):
    """HBM bytes per launch of a kernel from a committed rocprofv3 counter
    summary, or None when it is missing or was taken on a different kernel
    source (the GEMV's by default)."""
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash(sources):
        return None
    if abs(float(t.get("algorithmic_bytes_per_launch", -1.0)) - per_launch_algorithmic) > 1.0:
        return None                      # counters of another launch shape
    return float(t["hbm_bytes_per_launch"])


def measured_kernel_traffic(workload: str, kernel: str, per_launch_algorithmic: float):
    """HBM bytes per launch of one kernel of a workload from its committed
    rocprofv3 summary (profiles/traffic_<workload>.json), or None when it is
    missing, was taken on different kernel sources, or on another launch shape."""
    try:
        with open(os.path.join(ROOT, "profiles", f"traffic_{workload}.json")) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash(t.get("sources")):
        return None
    kt = t.get("kernels", {}).get(kernel)
    if not kt:
        return None
    alg = float(kt.get("algorithmic_bytes_per_launch", -1.0))
    if abs(alg - per_launch_algorithmic) > 1e-9 * max(alg, 1.0) + 1.0:
        return None
    return float(kt["hbm_bytes_per_launch"])


def measured_mfma(workload: str, kernel: str):
    """Matrix-core counters of one kernel of a workload from its committed
    rocprofv3 summary (profiles/mfma_<workload>.json): flops issued per launch
    (SQ_INSTS_VALU_MFMA_MOPS_* x 512) and the busy fraction of the matrix
    cores at the clock the launch ran at (SQ_VALU_MFMA_BUSY_CYCLES over
    GRBM_GUI_ACTIVE per XCC x SIMDs).  None when missing or taken on other
    kernel sources."""
    try:
        with open(os.path.join(ROOT, "profiles", f"mfma_{workload}.json")) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash(t.get("sources")):
        return None
    kt = t.get("kernels", {}).get(kernel)
    if not kt:
        return None
    return {"kernel": kernel, "issued_flops_per_launch": kt["issued_flops_per_dispatch"],
            "busy_frac": kt["mfma_util"]}


def measured_valu(draws: int):
    """Executed VALU wave-instructions per runtime-model launch of `draws`
    draws, or None when the summary is missing or for another source."""
    try:
        with open(VALU_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash(RUNTIME_SOURCES) or t.get("draws_per_launch") != draws:
        return None
    return float(t["valu_insts_per_launch"])


def host_info() -> dict:
    """The host the oracle baseline ran on: cores this process may use, BLAS
    library and its thread count, RAM and CPU model."""
    info = {"host_cores_available": len(os.sched_getaffinity(0)), "host_cpu_count": os.cpu_count()}
    try:
        from threadpoolctl import threadpool_info
        info["blas"] = [{"library": p.get("internal_api"), "version": p.get("version"),
                         "threads": p.get("num_threads")}
                        for p in threadpool_info() if p.get("user_api") == "blas"]
    except Exception:
        info["blas"] = None
    try:
        info["host_ram_gib"] = round(os.sysconf("SC_PAGE_SIZE") * os.sysconf("SC_PHYS_PAGES") / 2 ** 30, 1)
    except (ValueError, OSError, AttributeError):
        info["host_ram_gib"] = None
    try:
        with open("/proc/cpuinfo") as f:
            info["host_cpu"] = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        info["host_cpu"] = None
    return info


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        info = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if info:
            return int(max(p["num_threads"] for p in info))
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


# Compute- and latency-bound steps run faster once the GPU's clocks have
# ramped under load (the dense single pass: 1.545 ms per pass after three
# calls, 1.44 ms after half a second of them; the (4,2) one-launch product:
# 7.33 against 7.21 us).  Those workloads call their step, untimed, for
# CLOCK_RAMP_S before the timed steps, so that the timed steps measure the
# steady state; the memory-bound GEMV workloads do not need it.
CLOCK_RAMP_S = 1.0


def ramp_clocks(call, seconds: float = CLOCK_RAMP_S) -> None:
    import torch
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for i in range(8):
            call(i)
        torch.cuda.synchronize()


def gemv_workload(args):
    import torch

    from paper_1512_02673_amd import binding as lib

    w = synth.WORKLOADS[args.workload if args.workload.startswith("gemv16x12") else "gemv16x12_65536x8192"]
    n, k, q, r, seed = w.n, w.k, w.q, w.r, w.seed
    K, W = args.steps, args.warmup
    t0 = time.time()
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    if "parity_candidate" in w.extra:
        # the certified generator (worst decode condition number over every survivor set)
        P = synth.conditioned_parity_matrix(n, k, seed, w.extra["candidates"], pick=w.extra["parity_candidate"])[0]
    else:
        P = synth.parity_matrix(n, k, seed)
    planes = w.extra.get("planes", 2)
    xs = np.stack([synth.gaussian((r,), seed, synth.STREAM_X, t) for t in range(K + W)])
    print(f"[bench] inputs drawn in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    code = lib.Code.systematic(P, planes=planes)
    dA = torch.from_numpy(A).cuda()
    dX = torch.from_numpy(xs).cuda()
    par = lib.alloc_parity(code, q, r, torch.float32)
    Y = lib.alloc_y(code, q, 1, torch.float64)
    out = torch.empty((K + W, q), dtype=torch.float32, device="cuda")
    info = torch.zeros(K + W, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(1_000_000)             # the encode is queued before the first event fires
    e0.record()
    lib.coded_encode(code, dA, par)
    e1.record()
    torch.cuda.synchronize()
    encode_ms = e0.elapsed_time(e1)

    # One step is one coded_matmul call (survivor draw, all n worker products,
    # decode), made through the C ABI with its arguments converted once, so
    # that Python overhead stays far below the GPU time of a step.  The timed
    # loop records no per-step events: timing events and cross-stream waits
    # between the workers and the decode measured about 12 us per product
    # (2%), and a two-stream pipeline of workers and decode gained nothing
    # over the calls back to back.
    import ctypes
    h = lib.lib()
    vp = ctypes.c_void_p
    ws = lib.matmul_workspace(code, dA, dX[0])
    code_h, st_h, ws_p = code.handle, vp(stream.cuda_stream), vp(ws.data_ptr())
    A_p, par_p = vp(dA.data_ptr()), vp(par.data_ptr())
    x_p = [vp(dX[t].data_ptr()) for t in range(K + W)]
    out_p = [vp(out[t].data_ptr()) for t in range(K + W)]
    info_p = [vp(info[t:t + 1].data_ptr()) for t in range(K + W)]
    tk = ctypes.c_double()
    tk_p = ctypes.addressof(tk)

    def step(t):
        rc = h.coded_matmul(code_h, lib.CODED_F32, A_p, q, r, r, par_p, 1, x_p[t], 1, 1, seed, t, 1.0, 1.0, None,
                            tk_p, out_p[t], 1, ws_p, info_p[t], st_h)
        if rc:
            raise RuntimeError(lib.last_error())

    for t in range(W):
        step(t)
    torch.cuda.synchronize()
    start = time.perf_counter()
    for i in range(K):
        step(W + i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - start
    if int(info.abs().sum().item()) != 0:
        raise RuntimeError("a decode reported a singular or invalid survivor set")

    # Per-kernel times, in a separate pass: the same products as separate
    # worker and decode calls with events around each (these also check that
    # coded_matmul equals the decomposed step bit for bit).
    m_steps = min(K, 200)
    Y2 = lib.alloc_y(code, q, 1, torch.float64)
    one = torch.empty(q, dtype=torch.float32, device="cuda")
    inf1 = torch.zeros(1, dtype=torch.int32, device="cuda")
    surv = np.zeros(k, dtype=np.int32)
    surv_p = surv.ctypes.data_as(vp)
    Y2_p, one_p, inf1_p = vp(Y2.data_ptr()), vp(one.data_ptr()), vp(inf1.data_ptr())
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(m_steps)]
    for i in range(m_steps):
        t = W + i
        h.coded_draw_survivors(n, k, seed, t, 1.0, 1.0, surv_p, None)
        evs[i][0].record(stream)
        h.coded_worker_mm(code_h, lib.CODED_F32, A_p, q, r, r, par_p, x_p[t], 1, 1, None, Y2_p, lib.CODED_F64, None,
                          st_h)
        evs[i][1].record(stream)
        h.coded_decode(code_h, surv_p, k, Y2_p, lib.CODED_F64, q, 1, one_p, 1, inf1_p, st_h)
        evs[i][2].record(stream)
        if i in (0, m_steps - 1):
            torch.cuda.synchronize()
            if not torch.equal(one, out[t]):
                raise RuntimeError("coded_matmul differs from the decomposed step")
    torch.cuda.synchronize()
    gemv_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    dec_ms = np.array([e[1].elapsed_time(e[2]) for e in evs])
    matmul_ms = elapsed * 1e3 / K

    qb = code.qb(q)
    lo16 = planes == lib.CODED_PLANES_LO_BF16
    # bytes per parity element: fp32 planes, or an fp32 hi and a bf16 lo plane
    par_elem = 6.0 if lo16 else 4.0 * planes
    algo_bytes = 4.0 * q * r + par_elem * (n - k) * qb * r + 4.0 * r + 8.0 * n * qb
    gemv_mean_ms = float(gemv_ms.mean())
    achieved = algo_bytes / (gemv_mean_ms * 1e-3) / 1e9
    kname = f"gemv_wg_kernel<4, 8, 256, {'true' if lo16 else 'false'}>"
    if w.name == "gemv16x12_65536x8192":
        traffic = measured_traffic(algo_bytes)
    else:
        traffic = measured_kernel_traffic(w.name, kname, algo_bytes)
    result = {
        "metric": METRIC,
        "value": K / elapsed,
        "unit": "products/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": elapsed * 1e3 / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": w.name, "n": n, "k": k, "q": q, "r": r, "s": 1, "input_dtype": "f32",
                   "parity_planes": ("fp32 hi + bf16 lo (6 bytes per element)" if lo16 else planes),
                   "worker_accumulate": "f64", "encode": "once, before timing",
                   "survivors": "fresh shifted-exponential draw per product (shift 1, rate 1)"},
        "encode_ms": encode_ms,
        "gemv_ms_mean": gemv_mean_ms,
        "gemv_ms_p5_p95": [float(np.percentile(gemv_ms, 5)), float(np.percentile(gemv_ms, 95))],
        "decode_ms_mean": float(dec_ms.mean()),
        "coded_matmul_ms_per_call": matmul_ms,
        "roofline": {"bound": "hbm", "kernel": kname, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "algorithmic_bytes_per_launch": algo_bytes,
                     "traffic": traffic, "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE)"},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_gemv(w, A, P, xs, W, out, min(args.cpu_products, K))
    return result


def cpu_baseline_gemv(w, A, P, xs, first, out_dev, products):
    """The fp64 oracle on a bounded sample of the same workload: one encode of
    the full A, then `products` coded products (fresh x and draw each).  Its
    outputs also check the GPU's outputs for the same steps."""
    from oracle import coded as oc

    n, k, q, seed = w.n, w.k, w.q, w.seed
    G = oc.systematic_generator(P)
    t0 = time.perf_counter()
    coded = oc.encode(G, oc.pad_and_split(A, k))
    t_enc = time.perf_counter() - t0
    worst = 0.0
    t1 = time.perf_counter()
    for i in range(products):
        t = first + i
        Yo = oc.worker_products(coded, xs[t])
        S, _ = oc.draw_survivors(n, k, seed, t)
        ref = oc.decode_from_all(G, S, Yo, q)[:, 0]
        got = out_dev[t].cpu().numpy().astype(np.float64)
        worst = max(worst, float(np.max(np.abs(got - ref)) / np.max(np.abs(ref))))
    t_prod = time.perf_counter() - t1
    return {"value": products / t_prod, "unit": "products/s", "cores": blas_threads(), "kind": "oracle",
            "sample": f"{w.name}: one fp64 encode of the full A ({t_enc:.1f} s, not in value) then {products} "
                      f"coded products (all {n} worker products, draw, LU decode) in {t_prod:.1f} s",
            "encode_s": t_enc, "gpu_vs_oracle_max_rel_err": worst}


def mds_small_workload(args):
    """The (4,2) code on A 2048 x 512 fp32 with x 512 x 1, a fresh code and fresh
    inputs for each of 100 seeds (Sec. III-A's systematic MDS product at the
    smallest configured size).  One step is one coded_matmul of the next seed
    (encode + 4 worker products + draw + decode), seeds taken in turn; every
    seed's inputs are resident before timing.  The whole product touches about
    25 MB, so it is bound by launch latency, not by HBM."""
    import ctypes

    import torch

    from paper_1512_02673_amd import binding as lib

    w = synth.WORKLOADS["mds4x2_2048x512"]
    n, k, q, r = w.n, w.k, w.q, w.r
    seeds = w.extra["seeds"]
    K, W = args.steps, args.warmup
    codes, dA, dx, par = [], [], [], []
    hostA, hostP, hostx = [], [], []
    for sd in seeds:
        P = synth.parity_matrix(n, k, sd)
        A = synth.gaussian((q, r), sd, synth.STREAM_A)
        x = synth.gaussian((r, 1), sd, synth.STREAM_X)[:, 0]
        hostA.append(A), hostP.append(P), hostx.append(x)
        codes.append(lib.Code.systematic(P, planes=2))
        dA.append(torch.from_numpy(A).cuda())
        dx.append(torch.from_numpy(x).cuda())
        par.append(lib.alloc_parity(codes[-1], q, r, torch.float32))
    ws = lib.matmul_workspace(codes[0], dA[0], dx[0])
    out = torch.empty((len(seeds), q), dtype=torch.float32, device="cuda")
    info = torch.zeros(len(seeds), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    h = lib.lib()
    vp = ctypes.c_void_p
    st_h, ws_p = vp(stream.cuda_stream), vp(ws.data_ptr())
    args_c = [(codes[i].handle, vp(dA[i].data_ptr()), vp(par[i].data_ptr()), vp(dx[i].data_ptr()),
               vp(out[i].data_ptr()), vp(info[i:i + 1].data_ptr())) for i in range(len(seeds))]
    surv = np.zeros(k, dtype=np.int32)
    surv_p = surv.ctypes.data_as(vp)
    tk = ctypes.c_double()

    def step(t):
        i = t % len(seeds)
        c, A_p, P_p, x_p, o_p, inf_p = args_c[i]
        rc = h.coded_matmul(c, lib.CODED_F32, A_p, q, r, r, P_p, 0, x_p, 1, 1, seeds[i], 0, 1.0, 1.0, surv_p,
                            ctypes.addressof(tk), o_p, 1, ws_p, inf_p, st_h)
        if rc:
            raise RuntimeError(lib.last_error())

    for t in range(W):
        step(t)
    torch.cuda.synchronize()
    ramp_clocks(step)
    # Events only around the whole timed loop: per-step events would sit
    # between the launches (about 1.7 us each here).  Device time per product
    # is the loop's event interval over the steps.
    e_start, e_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start = time.perf_counter()
    e_start.record(stream)
    for i in range(K):
        step(W + i)
    e_end.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - start
    if int(info.abs().sum().item()) != 0:
        raise RuntimeError("a decode reported a singular or invalid survivor set")
    gpu_us = e_start.elapsed_time(e_end) * 1e3 / K
    qb = codes[0].qb(q)
    planes_b = 4.0 * 2 * (n - k) * qb * r
    # one launch: A read once, both planes written once, x, Y and the output
    prod_bytes = 4.0 * q * r + planes_b + 4.0 * r + 8.0 * n * qb + 4.0 * q
    result = {
        "metric": METRIC, "value": K / elapsed, "unit": "products/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": elapsed * 1e3 / K, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {"workload": w.name, "n": n, "k": k, "q": q, "r": r, "s": 1, "seeds": len(seeds),
                   "per_step": "coded_matmul of the next seed: encode + 4 worker products + draw + decode, "
                               "one launch"},
        "us_per_product_wall": elapsed * 1e6 / K, "us_per_product_gpu_events": gpu_us,
        "gpu_events_note": "events around the whole timed loop, interval / steps",
        "roofline": {"bound": "latency", "kernel": "onepass_f32_kernel (encode + 4 worker products + decode)",
                     "note": "about 12.6 MB per product in one launch of 1024 short workgroups: bound by launch "
                             "and memory latency; the HBM fraction below is for context",
                     "achieved": prod_bytes / (gpu_us * 1e-6) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": prod_bytes / (gpu_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     "algorithmic_bytes_per_launch": prod_bytes, "traffic": None},
    }
    if not args.no_cpu_baseline:
        from oracle import coded as oc
        worst, cnt = 0.0, 0
        t0 = time.perf_counter()
        while cnt < 40 * len(seeds) and time.perf_counter() - t0 < 15.0:
            i = cnt % len(seeds)
            G = oc.systematic_generator(hostP[i])
            coded = oc.encode(G, oc.pad_and_split(hostA[i], k))
            Yo = oc.worker_products(coded, hostx[i])
            S, _ = oc.draw_survivors(n, k, seeds[i], 0)
            ref = oc.decode_from_all(G, S, Yo, q)[:, 0]
            if cnt < len(seeds):
                got = out[i].cpu().numpy().astype(np.float64)
                worst = max(worst, float(np.max(np.abs(got - ref)) / np.max(np.abs(ref))))
            cnt += 1
        el = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": cnt / el, "unit": "products/s", "cores": blas_threads(), "kind": "oracle",
                                  "sample": f"{cnt} coded products of the same seeds (encode, 4 worker products, "
                                            f"draw, LU decode) in {el:.1f} s",
                                  "gpu_vs_oracle_max_rel_err": worst}
    result["clock_ramp_s"] = CLOCK_RAMP_S     # untimed calls before the timed steps
    return result


def decode_workload(args):
    """Decode-heavy workload: (64,48) code, A 16384 x 4096 fp32, X 4096 x 8; the
    64 worker products are computed once, then one step decodes A X from each
    of 10000 distinct survivor sets (each with >= 8 parity survivors) in one
    batched launch.  Unit: one decoded A X."""
    import torch

    from paper_1512_02673_amd import binding as lib

    w = synth.WORKLOADS["decode64x48_16384x4096x8"]
    n, k, q, r, s, seed, B = w.n, w.k, w.q, w.r, w.s, w.seed, w.units
    K, W = args.steps, args.warmup
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    X = synth.gaussian((r, s), seed, synth.STREAM_X)
    P = synth.parity_matrix(n, k, seed)
    code = lib.Code.systematic(P, planes=2)
    dA, dX = torch.from_numpy(A).cuda(), torch.from_numpy(X).cuda()
    par = lib.alloc_parity(code, q, r, torch.float32)
    Y = lib.alloc_y(code, q, s, torch.float64)
    lib.coded_encode(code, dA, par)
    lib.coded_worker_mm(code, dA, par, dX, Y)
    # The 64 worker products (s = 8 columns, fp64 matrix cores), timed on their own.
    stream = torch.cuda.current_stream()
    pev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(20)]
    for e0, e1 in pev:
        e0.record(stream)
        lib.coded_worker_mm(code, dA, par, dX, Y)
        e1.record(stream)
    torch.cuda.synchronize()
    prod_ms = np.array([a.elapsed_time(b) for a, b in pev])
    qb = code.qb(q)
    prod_bytes = 4.0 * q * r + 4.0 * code.planes * (n - k) * qb * r + 4.0 * r * s + 8.0 * n * qb * s
    prod_flops = 2.0 * (k * qb + code.planes * (n - k) * qb) * r * s
    if args.exact_parity is None:
        sets, _ = lib.coded_draw_survivor_sets(n, k, seed, B, min_parity=w.extra["min_parity"])
    else:
        # cost against the number of missing blocks: every set has exactly that many
        sets = synth.exact_parity_sets(n, k, args.exact_parity, B, seed)
    dsets = torch.from_numpy(sets).cuda()
    out = torch.empty((B, q, s), dtype=torch.float32, device="cuda")
    info = torch.zeros(B, dtype=torch.int32, device="cuda")
    for _ in range(W):
        lib.coded_decode_batched(code, dsets, Y, q, out, info)
    torch.cuda.synchronize()
    ramp_clocks(lambda i: lib.coded_decode_batched(code, dsets, Y, q, out, info))
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    start = time.perf_counter()
    for i in range(K):
        evs[i][0].record(stream)
        lib.coded_decode_batched(code, dsets, Y, q, out, info)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - start
    if int(info.abs().sum().item()) != 0:
        raise RuntimeError("a decode reported a singular or invalid survivor set")
    ms = np.array([a.elapsed_time(b) for a, b in evs])
    m = (sets >= k).sum(axis=1)
    algo_bytes = 4.0 * B * q * s + 8.0 * n * qb * s + 4.0 * B * k + 4.0 * B
    flops = float(np.sum(2.0 * m * k * qb * s))
    mean_s = float(ms.mean()) * 1e-3
    achieved = algo_bytes / mean_s / 1e9
    result = {
        "metric": METRIC, "value": B * K / elapsed, "unit": "decodes/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": elapsed * 1e3 / K, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "launch_ms_mean": float(ms.mean()), "launch_ms_p5_p50_p95": [float(np.percentile(ms, p)) for p in (5, 50, 95)],
        "config": {"workload": w.name, "n": n, "k": k, "q": q, "r": r, "s": s, "sets_per_step": B,
                   "min_parity": w.extra["min_parity"], "mean_parity_survivors": float(m.mean()),
                   "sets": ("distinct drawn sets (shifted-exponential runtimes) with >= min_parity parity survivors"
                            if args.exact_parity is None else
                            f"uniform random sets with exactly {args.exact_parity} parity survivors (repeats allowed)")},
        "roofline": {"bound": "hbm", "kernel": "decode_mfma_kernel", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "algorithmic_bytes_per_launch": algo_bytes,
                     "traffic": measured_kernel_traffic(w.name, "decode_mfma_kernel<12, 4, double, true, true>", algo_bytes), "fp64_tflops": flops / mean_s / 1e12, "fp64_frac": flops / mean_s / 78.6e12,
                     "mfma_counters": measured_mfma(w.name, "decode_mfma_kernel<12, 4, double, true, true>")},
        "products": {"kernel": "gemm_f32_mfma_kernel<1, 2, true, 128, 2, true> (64 worker products, s = 8, once per run)",
                     "ms_mean": float(prod_ms.mean()), "ms_min": float(prod_ms.min()),
                     "algorithmic_bytes_per_launch": prod_bytes,
                     "achieved_gbs": prod_bytes / (float(prod_ms.mean()) * 1e-3) / 1e9,
                     "hbm_frac": prod_bytes / (float(prod_ms.mean()) * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "fp64_tflops": prod_flops / (float(prod_ms.mean()) * 1e-3) / 1e12,
                     "traffic": measured_kernel_traffic(w.name, "gemm_f32_mfma_kernel<1, 2, true, 128, 2, true>", prod_bytes)},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_decode(w, A, X, P, sets, out, args.cpu_decodes)
    result["clock_ramp_s"] = CLOCK_RAMP_S     # untimed calls before the timed steps
    return result


def cpu_baseline_decode(w, A, X, P, sets, out_dev, count):
    """The fp64 oracle decoding a sample of the same survivor sets from its own worker products."""
    from oracle import coded as oc

    G = oc.systematic_generator(P)
    Yo = oc.worker_products(oc.encode(G, oc.pad_and_split(A, w.k)), X)
    idx = np.linspace(0, len(sets) - 1, count).astype(int)
    worst = 0.0
    t0 = time.perf_counter()
    refs = [oc.decode_from_all(G, sets[b], Yo, w.q) for b in idx]
    t = time.perf_counter() - t0
    for b, ref in zip(idx, refs):
        got = out_dev[b].cpu().numpy().astype(np.float64)
        den = np.max(np.abs(ref), axis=0)
        worst = max(worst, float(np.max(np.max(np.abs(got - ref), axis=0) / den)))
    return {"value": count / t, "unit": "decodes/s", "cores": blas_threads(), "kind": "oracle",
            "sample": f"{w.name}: {count} of the {len(sets)} survivor sets decoded by the oracle (LU of G_S, "
                      f"solve for all block rows) in {t:.1f} s; encode and worker products not timed",
            "gpu_vs_oracle_max_rel_err": worst}


def gd_workload(args):
    """Coded gradient descent for least squares (Sec. III-E): A 262144 x 4096 fp32
    N(0, 1/4096), y = A w* + N(0, 0.01) noise, (20,16) codes for A and for A^T,
    step 0.5 normalised by q * sigma^2 = 64.  One step = one iteration (two coded
    products, residual and update fused into the decodes)."""
    import torch

    from paper_1512_02673_amd import binding as lib

    w = synth.WORKLOADS[args.workload if args.workload.startswith("gd20x16") else "gd20x16_262144x4096"]
    n, k, q, r, seed = w.n, w.k, w.q, w.r, w.seed
    K, W = args.steps, args.warmup
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A, std=w.a_std)
    wstar = synth.gaussian((r,), seed, synth.STREAM_WSTAR)
    noise = synth.gaussian((q,), seed, synth.STREAM_NOISE)
    PA, PT, planes = synth.gd_codes(w)
    cA = lib.Code.systematic(PA, planes)
    cT = lib.Code.systematic(PT, planes)
    dA = torch.from_numpy(A).cuda()
    # y = A w* + noise, formed once on the device in fp64 as input preparation
    dy = (dA.double() @ torch.from_numpy(wstar).cuda().double() +
          w.extra["noise_std"] * torch.from_numpy(noise).cuda().double()).float()
    eta = w.extra["eta"] / (q * w.a_std ** 2)
    dAT = torch.empty((r, q), dtype=torch.float32, device="cuda")
    lib.coded_transpose(dA, dAT)
    pA, pT = lib.alloc_parity(cA, q, r, torch.float32), lib.alloc_parity(cT, r, q, torch.float32)
    lib.coded_encode(cA, dA, pA)
    lib.coded_encode(cT, dAT, pT)
    x = torch.zeros(r, dtype=torch.float32, device="cuda")
    ws = torch.empty(lib.coded_gd_sizes(cA, cT, q, r), dtype=torch.uint8, device="cuda")
    info = torch.zeros(2, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    for t in range(W):
        lib.coded_gd_step(cA, cT, dA, pA, dAT, pT, dy, x, eta, seed, t, ws, info)
    torch.cuda.synchronize()
    # no per-step events in the timed loop (they add GPU-side markers)
    start = time.perf_counter()
    for i in range(K):
        lib.coded_gd_step(cA, cT, dA, pA, dAT, pT, dy, x, eta, seed, W + i, ws, info)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - start
    if int(info.abs().sum().item()) != 0:
        raise RuntimeError("a decode reported a singular or invalid survivor set")
    step_ms = elapsed * 1e3 / K
    # The two worker GEMV launches of a step, timed alone on the same buffers.
    Y1 = lib.alloc_y(cA, q, 1, torch.float64)
    Y2 = lib.alloc_y(cT, r, 1, torch.float64)
    z = torch.zeros(q, dtype=torch.float32, device="cuda")
    g = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(40)]
    for i in range(20):
        g[2 * i][0].record(stream)
        lib.coded_worker_mm(cA, dA, pA, x, Y1)
        g[2 * i][1].record(stream)
        g[2 * i + 1][0].record(stream)
        lib.coded_worker_mm(cT, dAT, pT, z, Y2)
        g[2 * i + 1][1].record(stream)
    torch.cuda.synchronize()
    tA = float(np.mean([g[2 * i][0].elapsed_time(g[2 * i][1]) for i in range(20)]))
    tT = float(np.mean([g[2 * i + 1][0].elapsed_time(g[2 * i + 1][1]) for i in range(20)]))
    qbA, qbT = cA.qb(q), cT.qb(r)
    bA = 4.0 * q * r + 4.0 * planes * (n - k) * qbA * r + 4.0 * r + 8.0 * n * qbA
    bT = 4.0 * r * q + 4.0 * planes * (n - k) * qbT * q + 4.0 * q + 8.0 * n * qbT
    achieved = (bA + bT) / ((tA + tT) * 1e-3) / 1e9
    result = {
        "metric": METRIC, "value": K / elapsed, "unit": "iterations/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": elapsed * 1e3 / K, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {"workload": w.name, "n": n, "k": k, "q": q, "r": r, "eta_applied": eta,
                   "codes": ("separate (20,16) systematic codes for A and A^T, hi+lo parity" if planes == 2 else
                             "separate certified (20,16) codes for A and A^T (worst decode condition "
                             f"{w.extra['worst_condition']} and {w.extra['worst_condition_T']}), one fp32 parity plane"),
                   "parity_planes": planes},
        "gemv_A_ms": tA, "gemv_AT_ms": tT,
        "roofline": {"bound": "hbm", "kernel": "gemv_wg_kernel (A and A^T launches)", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "algorithmic_bytes_per_launch": [bA, bT],
                     "traffic": [measured_kernel_traffic(w.name, "gemv_wg_kernel<4, 4, 256, false>", bA),
                                 measured_kernel_traffic(w.name, "gemv_wg_kernel<4, 8, 256, false>", bT)],
                     "step_frac": (bA + bT) / (step_ms * 1e-3) / 1e9 / HBM_PEAK_GBS},
    }
    return result


def dense_bf16_workload(args):
    """Dense contraction regime: A 131072 x 16384 bf16 (N(0,1) rounded), (32,24)
    code, X 16384 x 64 bf16 with fp32 accumulation.  One step = one call:
    encode (hi+lo bf16 parity), the 32 worker products on the matrix cores, and
    the decode, with a fresh X and a fresh survivor draw."""
    import torch

    from paper_1512_02673_amd import binding as lib

    w = synth.WORKLOADS["gemm_bf16_32x24_131072x16384x64"]
    n, k, q, r, s, seed = w.n, w.k, w.q, w.r, w.s, w.seed
    K, W = args.steps, args.warmup
    t0 = time.time()
    A = synth.bf16_round(synth.gaussian_rows(q, r, seed, synth.STREAM_A))
    Xs = [synth.bf16_round(synth.gaussian((r, s), seed, synth.STREAM_X, t)) for t in range(K + W)]
    P = synth.parity_matrix(n, k, seed, dtype="bf16")
    print(f"[bench] inputs drawn in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    def to_dev(x):
        return torch.from_numpy(synth.bf16_bits(x).view(np.int16)).cuda().view(torch.bfloat16)

    code = lib.Code.systematic(P, planes=2)
    dA = to_dev(A)
    dX = [to_dev(x) for x in Xs]
    par = lib.alloc_parity(code, q, r, torch.bfloat16)
    ws = lib.matmul_workspace(code, dA, dX[0])
    out = torch.empty((K + W, q, s), dtype=torch.float32, device="cuda")
    info = torch.zeros(K + W, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    for t in range(W):
        lib.coded_matmul(code, dA, par, dX[t], out[t], ws, info[t:t + 1], seed, t, parity_ready=False)
    torch.cuda.synchronize()
    # draws and outputs the timed loop also uses
    ramp_clocks(lambda i: lib.coded_matmul(code, dA, par, dX[i % (K + W)], out[i % (K + W)], ws,
                                           info[i % (K + W):i % (K + W) + 1], seed, i % (K + W), parity_ready=False))
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    start = time.perf_counter()
    for i in range(K):
        t = W + i
        evs[i][0].record(stream)
        lib.coded_matmul(code, dA, par, dX[t], out[t], ws, info[t:t + 1], seed, t, parity_ready=False)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - start
    if int(info.abs().sum().item()) != 0:
        raise RuntimeError("a decode reported a singular or invalid survivor set")
    call_ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    # the single pass (encode + all worker products) alone, then the two-step
    # calls for context, same buffers
    Y = lib.alloc_y(code, q, s, torch.float32)
    wws = lib.worker_workspace(code, dA, dX[0])
    fused = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(10)]
    # one untimed call of each first: Y and the workspace are new allocations
    lib.coded_encode_worker_mm(code, dA, par, dX[W], Y, workspace=wws)
    lib.coded_encode(code, dA, par)
    lib.coded_worker_mm(code, dA, par, dX[W], Y, workspace=wws)
    for i in range(10):
        fused[i][0].record(stream)
        lib.coded_encode_worker_mm(code, dA, par, dX[W], Y, workspace=wws)
        fused[i][1].record(stream)
    ph = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(10)]
    for i in range(10):
        ph[i][0].record(stream)
        lib.coded_encode(code, dA, par)
        ph[i][1].record(stream)
        lib.coded_worker_mm(code, dA, par, dX[W], Y, workspace=wws)
        ph[i][2].record(stream)
    torch.cuda.synchronize()
    fused_ms = float(np.mean([a.elapsed_time(b) for a, b in fused]))
    enc_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ph]))
    wrk_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ph]))
    qb = code.qb(q)
    rows = k * qb + code.planes * (n - k) * qb
    par_bytes = 2.0 * code.planes * (n - k) * qb * r
    # one pass: A read once, the planes written once, X^T, Y written once
    fused_bytes = 2.0 * q * r + par_bytes + 2.0 * r * s + 4.0 * n * qb * s
    wrk_flops = 2.0 * rows * r * s
    enc_flops = 2.0 * (n - k) * k * qb * r
    wrk_bytes = 2.0 * q * r + par_bytes + 2.0 * r * s + 4.0 * n * qb * s
    enc_bytes = 2.0 * q * r + par_bytes
    call_bytes = fused_bytes + 4.0 * k * qb * s + 4.0 * q * s
    result = {
        "metric": METRIC, "value": K / elapsed, "unit": "calls/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": elapsed * 1e3 / K, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "n": n, "k": k, "q": q, "r": r, "s": s, "accumulate": "f32",
                   "parity_planes": code.planes, "per_call": "encode + worker products + decode, fresh X and draw"},
        "call_ms_events": call_ms, "encode_worker_ms": fused_ms,
        "two_step": {"encode_ms": enc_ms, "worker_ms": wrk_ms,
                     "bytes": enc_bytes + wrk_bytes, "note": "coded_encode then coded_worker_mm"},
        "call_hbm_frac": call_bytes / (call_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "roofline": {"bound": "hbm", "kernel": "fused_bf16_kernel (with the X transpose and the Y zero fill)",
                     "achieved": fused_bytes / (fused_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": fused_bytes / (fused_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "algorithmic_bytes_per_launch": fused_bytes,
                     "traffic": measured_traffic(fused_bytes, DENSE_TRAFFIC_FILE, DENSE_SOURCES),
                     "mfma_tflops": (wrk_flops + enc_flops) / (fused_ms * 1e-3) / 1e12,
                     "mfma_frac_of_bf16_dense_peak": (wrk_flops + enc_flops) / (fused_ms * 1e-3) / 2.5e15,
                     "mfma_ceiling_at_hbm_peak": (wrk_flops + enc_flops) / (fused_bytes / 8e12) / 2.5e15,
                     "mfma_counters": measured_mfma(w.name, "fused_bf16_kernel<8, 24, 8, true>")},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_dense(w, A, Xs, P, W, out, code.qb(q), args.cpu_rows)
    result["clock_ramp_s"] = CLOCK_RAMP_S     # untimed calls before the timed steps
    return result


def cpu_baseline_dense(w, A, Xs, P, t, out_dev, qb, rows):
    """The fp64 oracle on a slice of the same call: block rows [0, rows) of every
    block (the coded product is separable over block rows), encode + all 32 worker
    products + survivor draw + LU decode; the rate is scaled to whole calls."""
    from oracle import coded as oc

    n, k, q = w.n, w.k, w.q
    G = oc.systematic_generator(P)
    t0 = time.perf_counter()
    idx = np.concatenate([np.arange(j * qb, min(j * qb + rows, q)) for j in range(k)])
    slice_blocks = np.stack([np.vstack([A[j * qb + i].astype(np.float64) if j * qb + i < q else np.zeros(A.shape[1])
                                        for i in range(rows)]) for j in range(k)])
    coded = oc.encode(G, slice_blocks)
    Yo = oc.worker_products(coded, Xs[t])
    S, _ = oc.draw_survivors(n, k, w.seed, t)
    ref = oc.decode_from_all(G, S, Yo, k * rows)
    el = time.perf_counter() - t0
    got = out_dev[t].cpu().numpy()[idx].astype(np.float64)
    ref = ref[:len(idx)]
    den = np.max(np.abs(ref), axis=0)
    err = float(np.max(np.max(np.abs(got - ref), axis=0) / den))
    frac = rows / qb
    return {"value": frac / el, "unit": "calls/s", "cores": blas_threads(), "kind": "oracle",
            "sample": f"{w.name}: block rows [0, {rows}) of all {k} blocks ({frac:.4f} of a call) through encode, "
                      f"32 worker products, draw and decode in {el:.1f} s; rate scaled to whole calls",
            "gpu_vs_oracle_max_rel_err_on_sample": err}


def runtime_sim_workload(args):
    """Runtime model of Sec. III-C/III-D at the setting of its runtime-distribution
    figure (n = 10, k = 5, shift 1, rate 1): one step simulates 16M draws and
    writes the uncoded, 2-repetition and (10,5) MDS overall runtimes of each."""
    import torch

    from paper_1512_02673_amd import binding as lib

    n, k, seed, draws = 10, 5, 6, 1 << 24
    K, W = args.steps, args.warmup
    out = [torch.empty(draws, dtype=torch.float64, device="cuda") for _ in range(3)]
    stream = torch.cuda.current_stream()
    for t in range(W):
        lib.coded_simulate_runtimes(n, k, seed, t * draws, *out)
    torch.cuda.synchronize()
    ramp_clocks(lambda i: lib.coded_simulate_runtimes(n, k, seed, (i % max(W, 1)) * draws, *out))
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    start = time.perf_counter()
    for i in range(K):
        evs[i][0].record(stream)
        lib.coded_simulate_runtimes(n, k, seed, (W + i) * draws, *out)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - start
    ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    means = [float(t.mean().item()) for t in out]
    valu = measured_valu(draws)
    achieved = valu / (ms * 1e-3) / 1e9 if valu is not None else None
    result = {
        "metric": METRIC, "value": K * draws / elapsed, "unit": "simulated draws/s", "n_gpus": 1, "steps": K,
        "warmup": W, "ms_per_step": elapsed * 1e3 / K, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "runtime_sim_10x5", "n": n, "k": k, "shift": 1.0, "rate": 1.0,
                   "draws_per_step": draws, "schemes": ["uncoded", "repetition", "mds"]},
        "means_last_step": dict(zip(["uncoded", "repetition", "mds"], means)),
        "roofline": {"bound": "alu", "kernel": "runtime_sim_kernel<12>",
                     "note": "vector-issue bound: 64-bit SplitMix64 words and the O(n^2) ranking per draw; "
                             "achieved = executed VALU wave-instructions per launch (SQ_INSTS_VALU) / launch time",
                     "achieved": achieved, "peak": ALU_PEAK_G, "unit": "G wave-instructions/s",
                     "frac": achieved / ALU_PEAK_G if achieved is not None else None,
                     "valu_insts_per_launch": valu, "hbm_write_gbs": 24.0 * draws / (ms * 1e-3) / 1e9,
                     "traffic": None},
    }
    if not args.no_cpu_baseline:
        from oracle import runtime as rt
        chunk, chunks = 1 << 21, 16
        t0 = time.perf_counter()
        for c in range(chunks):
            rt.simulate(n, k, seed, c * chunk, chunk)
        el = time.perf_counter() - t0
        cnt = chunk * chunks
        result["cpu_baseline"] = {"value": cnt / el, "unit": "simulated draws/s", "cores": 1,
                                  "kind": "oracle", "sample": f"{cnt} draws of the same simulation with the NumPy "
                                                              f"oracle, {chunks} calls of {chunk}, in {el:.1f} s"}
    result["clock_ramp_s"] = CLOCK_RAMP_S     # untimed calls before the timed steps
    return result


def harmonic(n: int) -> float:
    return float(sum(1.0 / i for i in range(1, n + 1)))


def straggler_workload(args):
    """Real straggling on the GEMV workload's data: the protocol of Sec. III-A
    against the clock.  Each worker's product is started at its drawn task
    time T_i (Sec. III-C, eq. shifted_exp, shift 1, rate 1) times a time unit;
    the decode starts when the first k products have completed, and workers
    not started by then never run.  The same draws are run with the (16,12)
    code and uncoded (the (16,16) identity code: every one of 16 workers must
    finish).  The runtime model predicts E[T_(12 of 16)] = (1 + H_16 - H_4)/12
    and E[T_(16 of 16)] = (1 + H_16)/16 (eqs. mds_coded, uncoded); the
    measured latency adds the products, the decode and the host's polling.
    One step is one coded and one uncoded product."""
    import torch

    from paper_1512_02673_amd import binding as lib

    w = synth.WORKLOADS["gemv16x12_65536x8192"]
    n, k, q, r, seed = w.n, w.k, w.q, w.r, w.seed
    D, W, unit = args.steps, args.warmup, args.time_unit_us
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    P = synth.parity_matrix(n, k, seed)
    x = synth.gaussian((r,), seed, synth.STREAM_X, 0)
    coded = lib.Code.systematic(P, planes=2)
    uncoded = lib.Code.systematic(np.zeros((0, n)), planes=2)
    dA, dx = torch.from_numpy(A).cuda(), torch.from_numpy(x).cuda()
    par = lib.alloc_parity(coded, q, r, torch.float32)
    lib.coded_encode(coded, dA, par)
    Yc, Yu = lib.alloc_y(coded, q, 1, torch.float64), lib.alloc_y(uncoded, q, 1, torch.float64)
    out = torch.empty(q, dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()

    def run(code, Y, parity, draw):
        surv, tl, lat = lib.coded_straggler_matmul(code, dA, parity, dx, Y, out, info, seed, draw, unit)
        if int(info.item()) != 0:
            raise RuntimeError("a straggler decode reported a singular or invalid survivor set")
        return surv, tl, lat

    for d in range(W):
        run(coded, Yc, par, (1 << 30) + d)
        run(uncoded, Yu, None, (1 << 30) + d)
    lat_c, lat_u, over_c, over_u, started = [], [], [], [], []
    t0 = time.perf_counter()
    for d in range(D):
        surv, tl, lat = run(coded, Yc, par, d)
        lat_c.append(lat)
        over_c.append(lat - np.sort(tl[:, 0])[k - 1])
        started.append(int(np.sum(tl[:, 1] >= 0)))
        surv, tl, lat = run(uncoded, Yu, None, d)
        lat_u.append(lat)
        over_u.append(lat - np.max(tl[:, 0]))
    elapsed = time.perf_counter() - t0
    model_c = (1.0 + harmonic(n) - harmonic(n - k)) / k * unit * 1e-3
    model_u = (1.0 + harmonic(n)) / n * unit * 1e-3
    mc, mu = float(np.mean(lat_c)) * 1e-3, float(np.mean(lat_u)) * 1e-3
    return {
        "metric": METRIC, "value": mc, "unit": "ms per coded product (mean latency under straggling)",
        "n_gpus": 1, "steps": D, "warmup": W, "ms_per_step": elapsed * 1e3 / D, "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "straggler16x12_65536x8192", "n": n, "k": k, "q": q, "r": r,
                   "time_unit_us": unit, "shift": 1.0, "rate": 1.0, "survivors_only": True},
        "uncoded_ms": mu, "speedup_vs_uncoded": mu / mc,
        "model": {"coded_ms": model_c, "uncoded_ms": model_u, "speedup": model_u / model_c},
        "overhead_ms": {"coded_mean": float(np.mean(over_c)) * 1e-3, "uncoded_mean": float(np.mean(over_u)) * 1e-3,
                        "note": "latency minus the draw's own k-th (or last) start time: products, decode, polling"},
        "p95_ms": {"coded": float(np.percentile(lat_c, 95)) * 1e-3, "uncoded": float(np.percentile(lat_u, 95)) * 1e-3},
        "workers_started_mean": float(np.mean(started)),
        "roofline": None,
        "roofline_note": "a latency experiment: the time is set by the injected runtimes, not by a kernel's roofline",
    }


def shuffle_workload(args):
    """Coded shuffling (Sec. IV) with the paper's cache fraction s/q = 0.1
    and n = 16 workers, q = 10^6 rows of 256 fp32 (1 GB): a regime where the
    law-of-large-numbers step of Theorem 1 holds (the number of worker groups
    a row can fall into stays far below q).  One step is one iteration: the host plans Algorithm 1 for a fresh
    random partition, the device encodes the multicast rows and decodes every
    worker's missing rows, and the host applies the cache rule.  Unit: decoded
    rows per second of device time (encode + decode); the host planning time
    and the communication rates (measured vs eqs. r1 and r2) are reported
    beside it."""
    import torch

    from paper_1512_02673_amd import binding as lib

    n, q, r, cache, seed = 16, 1_000_000, 256, 100_000, 8
    K, W = args.steps, args.warmup
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    dA = torch.from_numpy(A).cuda()
    st = lib.Shuffle(n, q, cache, seed)
    stream = torch.cuda.current_stream()
    rec = []
    for it in range(W + K):
        t0 = time.perf_counter()
        coded_rows, terms = st.plan()
        tb = st.tables()
        t_plan = time.perf_counter() - t0
        dev = {k: torch.from_numpy(tb[k]).cuda() for k in ("enc_off", "enc_rows", "term_msg")}
        M = torch.empty((coded_rows, r), dtype=torch.float32, device="cuda")
        out = torch.empty((terms, r), dtype=torch.float32, device="cuda")
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        torch.cuda.synchronize()
        # a short spin ahead of the first event keeps the stream busy while the host
        # launches the encode: the interval then holds the kernel, not the launch latency
        torch.cuda._sleep(1_000_000)
        ev[0].record(stream)
        lib.coded_shuffle_encode(dA, dev["enc_off"], dev["enc_rows"], M)
        ev[1].record(stream)
        lib.coded_shuffle_decode(dA, M, dev["enc_off"], dev["enc_rows"], dev["term_msg"], out)
        ev[2].record(stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        st.commit()
        t_commit = time.perf_counter() - t1
        c = np.diff(tb["enc_off"]).astype(np.float64)            # terms per message row
        enc_bytes = 4.0 * r * (terms + coded_rows)
        dec_bytes = 4.0 * r * (coded_rows + 2.0 * terms)            # each message and data row read once, rows written
        if it >= W:
            rec.append((coded_rows, terms, t_plan, t_commit, ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2]),
                        enc_bytes, dec_bytes))
        del M, out, dev
    a = np.array(rec)
    enc_ms, dec_ms = float(a[:, 4].mean()), float(a[:, 5].mean())
    enc_gbs = float(np.mean(a[:, 6] / (a[:, 4] * 1e-3))) / 1e9
    dec_gbs = float(np.mean(a[:, 7] / (a[:, 5] * 1e-3))) / 1e9
    s_rows = cache

    def harm_rate_coded():
        pp = (s_rows - q / n) / (q - q / n)
        return q / (n * pp) ** 2 * ((1 - pp) ** (n + 1) + (n - 1) * pp * (1 - pp) - (1 - pp) ** 2)
    result = {
        "metric": METRIC, "value": float(np.sum(a[:, 1]) / np.sum((a[:, 4] + a[:, 5]) * 1e-3)),
        "unit": "decoded rows/s (device encode + decode)", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": float(np.mean((a[:, 4] + a[:, 5]))), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "shuffle16_1000000x256", "n": n, "q": q, "r": r, "cache_rows": cache, "seed": seed},
        "rates_rows_per_iteration": {
            "coded_measured": float(a[:, 0].mean()), "uncoded_measured": float(a[:, 1].mean()),
            "coded_theorem_eq_r2": harm_rate_coded(), "uncoded_eq_r1": q * (1 - s_rows / q),
            "reduction_measured": 1 - float(a[:, 0].mean() / a[:, 1].mean())},
        "host_ms": {"plan": float(a[:, 2].mean()) * 1e3, "cache_rule": float(a[:, 3].mean()) * 1e3},
        "encode_ms": enc_ms, "decode_ms": dec_ms,
        "roofline": {"bound": "hbm", "kernel": "shuffle_decode_kernel", "achieved": dec_gbs, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": dec_gbs / HBM_PEAK_GBS,
                     "algorithmic_bytes_per_launch": float(a[:, 7].mean()),
                     "traffic": measured_kernel_traffic("shuffle16_1000000x256", "shuffle_decode_kernel<4>",
                                                        float(a[:, 7].mean())),
                     "encode_achieved_gbs": enc_gbs, "encode_algorithmic_bytes_per_launch": float(a[:, 6].mean())},
    }
    if not args.no_cpu_baseline:
        from oracle import shuffle as sh
        # the oracle on its own plan: the first iteration from the same seed's
        # initial state (its own partition, cache signatures and Algorithm 1)
        t0 = time.perf_counter()
        ost = sh.initial_state(n, q, cache, seed)
        op = sh.plan(ost)
        t_plan = time.perf_counter() - t0
        t0 = time.perf_counter()
        sh.decode(A, sh.encode(A, op), op)
        el = time.perf_counter() - t0
        mcount = op.coded_rows
        result["cpu_baseline"] = {"value": op.uncoded_rows / el, "unit": "decoded rows/s (encode + decode)",
                                  "cores": 1, "kind": "oracle", "plan_s": t_plan,
                                  "sample": f"the oracle's own plan of iteration 1 from the same seed ({mcount} "
                                            f"messages, {op.uncoded_rows} decoded rows; planning {t_plan:.1f} s "
                                            f"not in value), oracle encode + decode in {el:.1f} s"}
    return result


def calibrate_copy(nbytes: int, reps: int):
    """A plain device copy of known size, for scaling rocprofv3 FETCH_SIZE/WRITE_SIZE counters."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "reps": reps}))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="gemv16x12_65536x8192",
                    choices=["gemv16x12_65536x8192", "gemv16x12_conditioned_65536x8192",
                             "gemv16x12_bf16lo_65536x8192", "mds4x2_2048x512",
                             "decode64x48_16384x4096x8", "gd20x16_262144x4096", "gd20x16_conditioned_262144x4096",
                             "gemm_bf16_32x24_131072x16384x64", "runtime_sim_10x5",
                             "straggler16x12_65536x8192", "shuffle16_1000000x256"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--exact-parity", type=int, default=None, metavar="M",
                    help="decode workload: survivor sets with exactly M parity survivors instead of the drawn sets")
    ap.add_argument("--no-lo-plane", action="store_true",
                    help="default workload: skip the sub-record of the same products with a bfloat16 lo plane")
    ap.add_argument("--no-dense", action="store_true",
                    help="default workload: skip the dense bf16 sub-record (the GEMM half of the metric)")
    ap.add_argument("--cpu-products", type=int, default=700)
    ap.add_argument("--cpu-decodes", type=int, default=1000)
    ap.add_argument("--cpu-rows", type=int, default=3072)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES")
    ap.add_argument("--calibrate", action="store_true",
                    help="measure the device ceilings (read/write bandwidth, row-window reads, matrix rates) and exit")
    ap.add_argument("--time-unit-us", type=float, default=10000.0,
                    help="straggler workload: microseconds per unit of the runtime model")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the coded product is simulated on a single device); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy, 5)
        return
    if args.calibrate:
        from paper_1512_02673_amd import build as _build, calib
        if not os.path.exists(_build.CALIB_PATH):
            _build.build_calib()
        print(json.dumps(calib.ceilings()), flush=True)
        return
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    from paper_1512_02673_amd import build as _build
    if not os.path.exists(_build.LIB_PATH):
        _build.build()
    if args.workload == "mds4x2_2048x512":
        result = mds_small_workload(args)
    elif args.workload == "decode64x48_16384x4096x8":
        if "--steps" not in sys.argv:
            args.steps = 30
        if "--warmup" not in sys.argv:
            args.warmup = 10
        result = decode_workload(args)
    elif args.workload == "gemm_bf16_32x24_131072x16384x64":
        if "--steps" not in sys.argv:
            args.steps = 20
        if "--warmup" not in sys.argv:
            args.warmup = 3
        result = dense_bf16_workload(args)
    elif args.workload == "runtime_sim_10x5":
        if "--steps" not in sys.argv:
            args.steps = 20
        if "--warmup" not in sys.argv:
            args.warmup = 2
        result = runtime_sim_workload(args)
    elif args.workload == "shuffle16_1000000x256":
        if "--steps" not in sys.argv:
            args.steps = 5
        if "--warmup" not in sys.argv:
            args.warmup = 1
        result = shuffle_workload(args)
    elif args.workload == "straggler16x12_65536x8192":
        if "--steps" not in sys.argv:
            args.steps = 100
        if "--warmup" not in sys.argv:
            args.warmup = 3
        result = straggler_workload(args)
    elif args.workload.startswith("gd20x16"):
        if "--steps" not in sys.argv:
            args.steps = 200
        if "--warmup" not in sys.argv:
            args.warmup = 5
        result = gd_workload(args)
    else:
        result = gemv_workload(args)
        if args.workload == "gemv16x12_65536x8192" and not args.no_lo_plane:
            # The same products with a bfloat16 lo parity plane (6-byte parity elements).
            import copy
            largs = copy.copy(args)
            largs.workload, largs.no_cpu_baseline = "gemv16x12_bf16lo_65536x8192", True
            torch.cuda.empty_cache()
            lo = gemv_workload(largs)
            result["bf16_lo_plane"] = {key: lo[key] for key in ("value", "unit", "steps", "warmup", "ms_per_step",
                                                                "config", "gemv_ms_mean", "decode_ms_mean",
                                                                "roofline")}
        if args.workload == "gemv16x12_65536x8192" and not args.no_dense:
            # The metric's GEMM half: the dense bf16 workload in the same run, 20 timed calls.
            import copy
            dargs = copy.copy(args)
            dargs.steps, dargs.warmup = 20, 3
            torch.cuda.empty_cache()
            d = dense_bf16_workload(dargs)
            if isinstance(d.get("cpu_baseline"), dict):
                d["cpu_baseline"].update(host_info())
            result["dense_gemm"] = {key: d[key] for key in ("value", "unit", "steps", "warmup", "ms_per_step",
                                                            "dtype", "config", "call_ms_events", "encode_worker_ms",
                                                            "call_hbm_frac", "roofline", "cpu_baseline", "clock_ramp_s")
                                   if key in d}
    if isinstance(result.get("cpu_baseline"), dict):
        result["cpu_baseline"].update(host_info())
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
