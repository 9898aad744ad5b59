"""GPU parity at the workloads' full sizes, in the launch configurations bench.py times.

Every decoded output is checked against the oracle's fp64 product A X (a
property that holds for every survivor set), sampled ones also against the
oracle's own coded pipeline, and every survivor set bit for bit against the
oracle's draw.
"""
import numpy as np
import pytest

import synth
from oracle import coded as oc
from tests.gpu_helpers import torch_mod

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def per_set_errors(torch, out, ref):
    """Normwise relative error of each decoded set (batch, q, s) against ref (q, s), on the GPU."""
    den = ref.abs().amax(dim=0)
    errs = []
    for b0 in range(0, out.shape[0], 500):
        d = (out[b0:b0 + 500].double() - ref.unsqueeze(0)).abs().amax(dim=1) / den
        errs.append(d.amax(dim=1))
    return torch.cat(errs).cpu().numpy()


def test_gemv_workload_full_size(lib, torch):
    """(16,12) code, A 65536 x 8192 fp32: coded_matmul for several draws with fresh x."""
    w = synth.WORKLOADS["gemv16x12_65536x8192"]
    n, k, q, r, seed = w.n, w.k, w.q, w.r, w.seed
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    P = synth.parity_matrix(n, k, seed)
    code = lib.Code.systematic(P, 2)
    dA = torch.from_numpy(A).cuda()
    par = lib.alloc_parity(code, q, r, torch.float32)
    ws = lib.alloc_y(code, q, 1, torch.float64)
    out = torch.empty(q, dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    A64 = A.astype(np.float64)
    for t in range(4):
        x = synth.gaussian((r,), seed, synth.STREAM_X, t)
        surv, T = lib.coded_matmul(code, dA, par, torch.from_numpy(x).cuda(), out, ws, info, seed, t,
                                   parity_ready=t > 0)
        torch.cuda.synchronize()
        S, T_ref = oc.draw_survivors(n, k, seed, t)
        assert np.array_equal(surv, S) and int(info.item()) == 0
        ref = oc.plain_product(A64, x)[:, 0]
        err = float(np.max(np.abs(out.cpu().numpy() - ref)) / np.max(np.abs(ref)))
        assert err <= TOL_F32, (t, err)


def test_decode_heavy_workload_full_size(lib, torch):
    """(64,48) code, A 16384 x 4096 fp32, X 4096 x 8: all 10000 distinct survivor sets
    (>= 8 parity survivors each) decoded in one batched launch."""
    w = synth.WORKLOADS["decode64x48_16384x4096x8"]
    n, k, q, r, s, seed, B = w.n, w.k, w.q, w.r, w.s, w.seed, w.units
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    X = synth.gaussian((r, s), seed, synth.STREAM_X)
    P = synth.parity_matrix(n, k, seed)
    code = lib.Code.systematic(P, 2)
    dA, dX = torch.from_numpy(A).cuda(), torch.from_numpy(X).cuda()
    par = lib.alloc_parity(code, q, r, torch.float32)
    Y = lib.alloc_y(code, q, s, torch.float64)
    lib.coded_encode(code, dA, par)
    lib.coded_worker_mm(code, dA, par, dX, Y)
    sets, nxt = lib.coded_draw_survivor_sets(n, k, seed, B, min_parity=w.extra["min_parity"])
    sets_ref, nxt_ref = oc.draw_survivor_sets(n, k, seed, B, min_parity=w.extra["min_parity"])
    assert np.array_equal(sets, sets_ref) and nxt == nxt_ref
    out = torch.full((B, q, s), float("nan"), dtype=torch.float32, device="cuda")
    info = torch.full((B,), 7, dtype=torch.int32, device="cuda")
    lib.coded_decode_batched(code, torch.from_numpy(sets).cuda(), Y, q, out, info)
    torch.cuda.synchronize()
    assert int((info != 0).sum().item()) == 0
    ref = torch.from_numpy(oc.plain_product(A, X)).cuda()
    errs = per_set_errors(torch, out, ref)
    assert np.all(np.isfinite(errs)) and float(errs.max()) <= TOL_F32, float(errs.max())
    # sampled sets against the oracle's own encode / worker products / LU decode
    G = oc.systematic_generator(P)
    Yo = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    for b in np.linspace(0, B - 1, 12).astype(int):
        ref_b = oc.decode_from_all(G, sets[b], Yo, q)
        got = out[b].cpu().numpy().astype(np.float64)
        den = np.max(np.abs(ref_b), axis=0)
        assert float(np.max(np.max(np.abs(got - ref_b), axis=0) / den)) <= TOL_F32


@pytest.mark.parametrize("name", ["gd20x16_262144x4096", "gd20x16_conditioned_262144x4096"])
def test_gd_workload_full_size(lib, torch, name):
    """(20,16) codes for A (262144 x 4096, N(0, 1/4096)) and A^T: sampled iterations against the plain
    fp64 update of the same iterate, survivors against the oracle, and first-order optimality after
    the 200 iterations of the workload.  The configured recipe (plain draws, two planes) and the
    certified generators with one parity plane."""
    w = synth.WORKLOADS[name]
    n, k, q, r, seed = w.n, w.k, w.q, w.r, w.seed
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A, std=w.a_std)
    wstar = synth.gaussian((r,), seed, synth.STREAM_WSTAR)
    A64 = A.astype(np.float64)
    y = (A64 @ wstar.astype(np.float64) + w.extra["noise_std"] * synth.gaussian((q,), seed, synth.STREAM_NOISE)
         ).astype(np.float32)
    eta = w.extra["eta"] / (q * w.a_std ** 2)
    PA, PT, planes = synth.gd_codes(w)
    cA = lib.Code.systematic(PA, planes)
    cT = lib.Code.systematic(PT, planes)
    dA = torch.from_numpy(A).cuda()
    dAT = torch.empty((r, q), dtype=torch.float32, device="cuda")
    lib.coded_transpose(dA, dAT)
    pA, pT = lib.alloc_parity(cA, q, r, torch.float32), lib.alloc_parity(cT, r, q, torch.float32)
    lib.coded_encode(cA, dA, pA)
    lib.coded_encode(cT, dAT, pT)
    dy = torch.from_numpy(y).cuda()
    x = torch.zeros(r, dtype=torch.float32, device="cuda")
    ws = torch.empty(lib.coded_gd_sizes(cA, cT, q, r), dtype=torch.uint8, device="cuda")
    info = torch.zeros(2, dtype=torch.int32, device="cuda")
    y64 = y.astype(np.float64)
    for t in range(w.units):
        before = x.cpu().numpy().astype(np.float64) if t in (0, 1, 7, 199) else None
        S1, S2 = lib.coded_gd_step(cA, cT, dA, pA, dAT, pT, dy, x, eta, seed, t, ws, info)
        if before is not None:
            torch.cuda.synchronize()
            assert np.array_equal(S1, oc.draw_survivors(n, k, seed, 2 * t)[0])
            assert np.array_equal(S2, oc.draw_survivors(n, k, seed, 2 * t + 1)[0])
            assert np.all(info.cpu().numpy() == 0)
            want = before - eta * (A64.T @ (A64 @ before - y64))
            got = x.cpu().numpy().astype(np.float64)
            assert np.max(np.abs(got - want)) <= 1e-4 * np.max(np.abs(want)), t
    torch.cuda.synchronize()
    xf = x.cpu().numpy().astype(np.float64)
    grad = A64.T @ (A64 @ xf - y64)
    assert np.linalg.norm(grad) <= 1e-4 * np.linalg.norm(A64.T @ y64)


def test_dense_bf16_workload_full_size(lib, torch):
    """(32,24) code, A 131072 x 16384 bf16, X 16384 x 64 bf16, fp32 accumulation: the first five
    calls as bench.py makes them (encode + matrix-core worker products + decode, fresh X and draw
    each); every output row of every call against the oracle's fp64 product (normwise per column,
    2e-2), survivors against the oracle's draw."""
    w = synth.WORKLOADS["gemm_bf16_32x24_131072x16384x64"]
    n, k, q, r, s, seed = w.n, w.k, w.q, w.r, w.s, w.seed
    calls = 5
    A = synth.bf16_round(synth.gaussian_rows(q, r, seed, synth.STREAM_A))
    P = synth.parity_matrix(n, k, seed, dtype="bf16")
    code = lib.Code.systematic(P, 2)
    dA = torch.from_numpy(synth.bf16_bits(A).view(np.int16)).cuda().view(torch.bfloat16)
    par = lib.alloc_parity(code, q, r, torch.bfloat16)
    outs = torch.empty((calls, q, s), dtype=torch.float32, device="cuda")
    info = torch.full((calls,), -7, dtype=torch.int32, device="cuda")
    Xs = []
    for t in range(calls):
        X = synth.bf16_round(synth.gaussian((r, s), seed, synth.STREAM_X, t))
        Xs.append(X)
        dX = torch.from_numpy(synth.bf16_bits(X).view(np.int16)).cuda().view(torch.bfloat16)
        ws = lib.matmul_workspace(code, dA, dX)
        surv, _ = lib.coded_matmul(code, dA, par, dX, outs[t], ws, info[t:t + 1], seed, t, parity_ready=False)
        assert np.array_equal(surv, oc.draw_survivors(n, k, seed, t)[0])
    torch.cuda.synchronize()
    assert np.all(info.cpu().numpy() == 0)
    del dA, par
    got = outs.cpu().numpy()                                   # (calls, q, s)
    Xall = np.concatenate(Xs, axis=1)                          # (r, calls * s): one fp64 product per row block
    max_diff = np.zeros(calls * s)
    max_ref = np.zeros(calls * s)
    for r0 in range(0, q, 4096):
        ref = oc.plain_product(A[r0:r0 + 4096], Xall)          # fp64
        g = got[:, r0:r0 + 4096, :].transpose(1, 0, 2).reshape(ref.shape[0], calls * s)
        max_diff = np.maximum(max_diff, np.max(np.abs(g - ref), axis=0))
        max_ref = np.maximum(max_ref, np.max(np.abs(ref), axis=0))
    err = float(np.max(max_diff / max_ref))
    print(f"dense full size: {calls} calls x {q} rows x {s} columns, max normwise error {err:.3e}")
    assert err <= 2e-2, err


def test_conditioned_gemv_workload_full_size(lib, torch):
    """The certified (16,12) generator with one fp32 parity plane, A 65536 x 8192
    fp32: coded_matmul for several draws with fresh x, as bench.py runs it."""
    w = synth.WORKLOADS["gemv16x12_conditioned_65536x8192"]
    n, k, q, r, seed = w.n, w.k, w.q, w.r, w.seed
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    P = synth.conditioned_parity_matrix(n, k, seed, w.extra["candidates"], pick=w.extra["parity_candidate"])[0]
    code = lib.Code.systematic(P, w.extra["planes"])
    assert code.planes == 1
    dA = torch.from_numpy(A).cuda()
    par = lib.alloc_parity(code, q, r, torch.float32)
    ws = lib.alloc_y(code, q, 1, torch.float64)
    out = torch.empty(q, dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    A64 = A.astype(np.float64)
    for t in range(3):
        x = synth.gaussian((r,), seed, synth.STREAM_X, t)
        surv, _ = lib.coded_matmul(code, dA, par, torch.from_numpy(x).cuda(), out, ws, info, seed, t,
                                   parity_ready=t > 0)
        torch.cuda.synchronize()
        S, _ = oc.draw_survivors(n, k, seed, t)
        assert np.array_equal(surv, S) and int(info.item()) == 0
        ref = oc.plain_product(A64, x)[:, 0]
        err = float(np.max(np.abs(out.cpu().numpy() - ref)) / np.max(np.abs(ref)))
        assert err <= TOL_F32, (t, err)


def test_straggler_workload_full_size(lib, torch):
    """Real straggling at the GEMV workload's size ((16,12), A 65536 x 8192 fp32),
    survivors only, as bench.py runs it, coded and uncoded ((16,16) identity
    code): each product against the oracle's fp64 A x, the survivors consistent
    with the timeline, and the start times the runtime model's draws."""
    from tests.test_gpu_straggler import check_timeline
    w = synth.WORKLOADS["gemv16x12_65536x8192"]
    n, k, q, r, seed = w.n, w.k, w.q, w.r, w.seed
    unit = 2000.0                                  # microseconds per unit of the runtime model
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    x = synth.gaussian((r,), seed, synth.STREAM_X, 0)
    ref = oc.plain_product(A.astype(np.float64), x)[:, 0]
    coded = lib.Code.systematic(synth.parity_matrix(n, k, seed), planes=2)
    uncoded = lib.Code.systematic(np.zeros((0, n)), planes=2)
    dA, dx = torch.from_numpy(A).cuda(), torch.from_numpy(x).cuda()
    par = lib.alloc_parity(coded, q, r, torch.float32)
    lib.coded_encode(coded, dA, par)
    out = torch.empty(q, dtype=torch.float32, device="cuda")
    info = torch.full((1,), 9, dtype=torch.int32, device="cuda")
    for code, parity, kk in ((coded, par, k), (uncoded, None, n)):
        Y = lib.alloc_y(code, q, 1, torch.float64)
        for draw in range(2):
            out.fill_(float("nan"))
            surv, tl, lat = lib.coded_straggler_matmul(code, dA, parity, dx, Y, out, info, seed, draw, unit)
            torch.cuda.synchronize()
            assert int(info.item()) == 0
            err = float(np.max(np.abs(out.cpu().numpy() - ref)) / np.max(np.abs(ref)))
            assert err <= TOL_F32, (kk, draw, err)
            check_timeline(n, kk, surv, tl, lat, False)
            assert np.allclose(tl[:, 0], oc.worker_runtimes(n, kk, seed, draw) * unit, rtol=1e-12)


def test_shuffle_workload_full_size(lib, torch):
    """Coded shuffling at the size bench.py measures (n = 16 workers, 10^6 rows of
    256 fp32, caches of 10^5 rows), two iterations.  The planner's tables equal
    the oracle's plan; three runs of 1000 messages (first, middle, last) of the
    coded rows, and the rows decoded from them, equal the oracle's encode and
    decode bit for bit; and every decoded row is the row of A it stands for,
    within the rounding of its message's fp32 sums (checked on the GPU)."""
    from oracle import shuffle as sh
    n, q, r, cache, seed = 16, 1_000_000, 256, 100_000, 8
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    dA = torch.from_numpy(A).cuda()
    st = lib.Shuffle(n, q, cache, seed)
    ref = sh.initial_state(n, q, cache, seed)
    for _ in range(2):
        coded_rows, terms = st.plan()
        tb = st.tables()
        p = sh.plan(ref)
        for key in ("enc_off", "enc_rows", "term_worker", "term_msg"):
            assert np.array_equal(tb[key], getattr(p, key)), key
        assert np.array_equal(tb["next_assign"], p.new_assign)
        assert (coded_rows, terms) == (p.coded_rows, p.uncoded_rows)
        dev = {key: torch.from_numpy(tb[key]).cuda() for key in ("enc_off", "enc_rows", "term_msg")}
        M = torch.full((coded_rows, r), float("nan"), dtype=torch.float32, device="cuda")
        out = torch.full((terms, r), float("nan"), dtype=torch.float32, device="cuda")
        lib.coded_shuffle_encode(dA, dev["enc_off"], dev["enc_rows"], M)
        lib.coded_shuffle_decode(dA, M, dev["enc_off"], dev["enc_rows"], dev["term_msg"], out)
        torch.cuda.synchronize()
        off = tb["enc_off"]
        for m0 in (0, coded_rows // 2, coded_rows - 1000):
            m1 = m0 + 1000
            a, b = int(off[m0]), int(off[m1])
            sub = sh.Plan(p.new_assign, [], off[m0:m1 + 1] - a, tb["enc_rows"][a:b], tb["term_worker"][a:b],
                          tb["term_msg"][a:b] - m0, m1 - m0, b - a)
            M_ref = sh.encode(A, sub)
            assert np.array_equal(M[m0:m1].cpu().numpy(), M_ref), m0
            assert np.array_equal(out[a:b].cpu().numpy(), sh.decode(A, M_ref, sub)), m0
        # all rows: |decoded - A[row]| <= 2 c 2^-24 (sum of the message's |rows|), c its term count
        rows = dev["enc_rows"].long()
        msg = dev["term_msg"].long()
        cnt = (dev["enc_off"][1:] - dev["enc_off"][:-1]).to(torch.float32)
        absum = torch.zeros((coded_rows, r), dtype=torch.float32, device="cuda")
        step = 100_000
        for c0 in range(0, terms, step):
            absum.index_add_(0, msg[c0:c0 + step], dA[rows[c0:c0 + step]].abs())
        for c0 in range(0, terms, step):
            mm = msg[c0:c0 + step]
            err = (out[c0:c0 + step] - dA[rows[c0:c0 + step]]).abs()
            bound = 2.0 * cnt[mm].unsqueeze(1) * 2.0 ** -24 * absum[mm]
            assert bool((err <= bound).all()), c0
        del M, out, absum
        st.commit()
        ref = sh.commit(ref, p)
