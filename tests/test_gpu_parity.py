"""GPU parity: the HIP library, called through the C ABI, against the fp64 oracle.

Tolerances: max normwise relative error 1e-4 for fp32 inputs and 2e-2 for
bf16 inputs (fp32 accumulation) against the fp64 product of the same input
values; integer-valued inputs are exact in every precision used on the
device, so those cases compare bit for bit; survivor sets always compare
bit for bit.
"""
import itertools

import numpy as np
import pytest

import synth
from oracle import coded as oc
from tests.gpu_helpers import device_tensor, make_inputs, normwise_rel_err, torch_mod

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def to_np(t):
    torch = torch_mod()
    if t.dtype == torch.bfloat16:
        return synth.bf16_from_bits(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


def info_tensor(torch, batch=1):
    return torch.full((batch,), 12345, dtype=torch.int32, device="cuda")


def vandermonde_parity(n, k):
    return np.array([[float((j + 1) ** i) for j in range(k)] for i in range(n - k)])


# ---------------------------------------------------------------- encode

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("planes", [1, 2])
@pytest.mark.parametrize("n,k,q,r", [(16, 12, 1000, 520), (5, 3, 31, 7), (64, 48, 700, 256), (4, 2, 1, 8)])
def test_encode_integer_inputs_bit_exact(lib, torch, dtype, planes, n, k, q, r):
    P, A, _ = make_inputs(n, k, q, r, 1, 3, dtype, integer=True)
    code = lib.Code.systematic(P, planes)
    dA = device_tensor(A, dtype)
    par = lib.alloc_parity(code, q, r, dA.dtype)
    par.fill_(7)
    lib.coded_encode(code, dA, par)
    torch.cuda.synchronize()
    ref = oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k))[k:]
    got = to_np(par).astype(np.float64)
    assert np.array_equal(got[0], ref)
    if planes == 2:
        assert np.all(got[1] == 0)


@pytest.mark.parametrize("n,k,q,r", [(16, 12, 2000, 1030), (64, 48, 400, 100)])
def test_encode_gaussian_split_planes(lib, torch, n, k, q, r):
    P, A, _ = make_inputs(n, k, q, r, 1, 4)
    code = lib.Code.systematic(P, 2)
    dA = device_tensor(A)
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    torch.cuda.synchronize()
    blocks = oc.pad_and_split(A, k)
    ref = oc.encode(oc.systematic_generator(P), blocks)[k:]
    scale = np.abs(oc.encode(oc.systematic_generator(np.abs(P)), np.abs(blocks))[k:])
    got = to_np(par).astype(np.float64)
    # fp64 sums on both sides (k roundings each) plus the hi/lo split
    assert np.all(np.abs(got[0] + got[1] - ref) <= (2.0 ** -46 + 4 * k * 2.0 ** -53) * scale)
    assert np.all(np.abs(got[0] - ref) <= 2.0 ** -24 * np.abs(ref) + 1e-300)


def test_encode_bf16_gaussian(lib, torch):
    n, k, q, r = 32, 24, 480, 136
    P, A, _ = make_inputs(n, k, q, r, 1, 5, "bf16")
    code = lib.Code.systematic(P, 2)
    dA = device_tensor(A, "bf16")
    par = lib.alloc_parity(code, q, r, torch.bfloat16)
    lib.coded_encode(code, dA, par)
    torch.cuda.synchronize()
    blocks = oc.pad_and_split(A, k)
    ref = oc.encode(oc.systematic_generator(P), blocks)[k:]
    scale = np.abs(oc.encode(oc.systematic_generator(np.abs(P)), np.abs(blocks))[k:])
    got = to_np(par).astype(np.float64)
    assert np.all(np.abs(got[0] + got[1] - ref) <= k * 2.0 ** -23 * scale + 2.0 ** -16 * np.abs(ref))


def test_encode_rejects_non_bf16_coefficients(lib, torch):
    P = synth.parity_matrix(6, 4, 1, dtype="f32")
    code = lib.Code.systematic(P, 2)
    A = device_tensor(synth.bf16_round(synth.gaussian((8, 8), 1, 1)), "bf16")
    par = lib.alloc_parity(code, 8, 8, torch.bfloat16)
    with pytest.raises(lib.CodedError):
        lib.coded_encode(code, A, par)


# ---------------------------------------------------------------- worker products

WORKER_CASES = [(16, 12, 3000, 2100, 1), (16, 12, 1000, 1024, 1), (4, 2, 2048, 512, 1), (5, 3, 31, 7, 1),
                (64, 48, 700, 256, 8), (6, 4, 50, 33, 5), (20, 16, 100, 4096, 1), (3, 1, 9, 12, 1),
                (4, 4, 17, 20, 1)]


@pytest.mark.parametrize("n,k,q,r,s", WORKER_CASES)
def test_worker_products_integer_bit_exact(lib, torch, n, k, q, r, s):
    P, A, X = make_inputs(n, k, q, r, s, 6, integer=True)
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A), device_tensor(X[:, 0] if s == 1 else X)
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    Y = lib.alloc_y(code, q, s, torch.float64)
    Y.fill_(float("nan"))
    lib.coded_worker_mm(code, dA, par, dX, Y)
    torch.cuda.synchronize()
    ref = oc.worker_products(oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k)), X)
    assert np.array_equal(Y.cpu().numpy(), ref)


@pytest.mark.parametrize("n,k,q,r,s", WORKER_CASES)
@pytest.mark.parametrize("planes", [1, 2])
def test_worker_products_gaussian(lib, torch, n, k, q, r, s, planes):
    P, A, X = make_inputs(n, k, q, r, s, 7)
    code = lib.Code.systematic(P, planes)
    dA, dX = device_tensor(A), device_tensor(X[:, 0] if s == 1 else X)
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    Y = lib.alloc_y(code, q, s, torch.float64)
    lib.coded_worker_mm(code, dA, par, dX, Y)
    torch.cuda.synchronize()
    G = oc.systematic_generator(P)
    coded = oc.encode(G, oc.pad_and_split(A, k))
    ref = oc.worker_products(coded, X)
    bound = oc.worker_products(np.abs(coded), np.abs(X))
    # fp64 accumulation; the parity blocks carry the hi/lo (or hi-only) rounding
    parity_u = 2.0 ** -46 if planes == 2 else 2.0 ** -24
    err = np.abs(Y.cpu().numpy() - ref)
    assert np.all(err[:k] <= 1e-12 * bound[:k])
    assert np.all(err[k:] <= (1e-12 + parity_u) * bound[k:])


@pytest.mark.parametrize("n,k,q,r,s", [(32, 24, 1000, 512, 64), (32, 24, 333, 136, 40), (6, 4, 70, 256, 16),
                                       (5, 3, 31, 64, 7), (8, 5, 90, 128, 100), (4, 2, 10, 8, 1), (5, 3, 20, 12, 3)])
@pytest.mark.parametrize("planes", [1, 2])
def test_worker_products_bf16_integer_bit_exact(lib, torch, n, k, q, r, s, planes):
    """bf16 blocks and X on the matrix cores (and the vector kernel without a workspace):
    integer-valued inputs make every fp32 sum exact, so Y must equal the oracle's exactly."""
    P, A, X = make_inputs(n, k, q, r, s, 19, "bf16", integer=True)
    code = lib.Code.systematic(P, planes)
    dA, dX = device_tensor(A, "bf16"), device_tensor(X[:, 0] if s == 1 else X, "bf16")
    par = lib.alloc_parity(code, q, r, torch.bfloat16)
    lib.coded_encode(code, dA, par)
    ref = oc.worker_products(oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k)), X)
    for ws in ("auto", None):
        Y = lib.alloc_y(code, q, s, torch.float32)
        Y.fill_(float("nan"))
        lib.coded_worker_mm(code, dA, par, dX, Y, workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(Y.cpu().numpy().astype(np.float64), ref), ws


def test_worker_mask_leaves_other_rows_untouched(lib, torch):
    n, k, q, r = 16, 12, 500, 640
    P, A, X = make_inputs(n, k, q, r, 1, 8, integer=True)
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A), device_tensor(X[:, 0])
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    mask = np.zeros(n, dtype=np.uint8)
    mask[[0, 5, 12, 15]] = 1
    Y = lib.alloc_y(code, q, 1, torch.float64)
    Y.fill_(-1.0)
    lib.coded_worker_mm(code, dA, par, dX, Y, worker_mask=mask)
    torch.cuda.synchronize()
    ref = oc.worker_products(oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k)), X)
    got = Y.cpu().numpy()
    for i in range(n):
        if mask[i]:
            assert np.array_equal(got[i], ref[i])
        else:
            assert np.all(got[i] == -1.0)


# ---------------------------------------------------------------- decode

@pytest.mark.parametrize("n,k", [(3, 2), (4, 2), (5, 3), (6, 4), (7, 4), (6, 3)])
def test_decode_every_subset_integer_inputs(lib, torch, n, k):
    q, r, s = 4 * k - 1, 6, 3
    P = vandermonde_parity(n, k)
    A = synth.integers((q, r), 9, synth.STREAM_A)
    X = synth.integers((r, s), 9, synth.STREAM_X)
    G = oc.systematic_generator(P)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    code = lib.Code(n, k, G, 2)
    dY = torch.from_numpy(Y).to("cuda")
    expect = A.astype(np.float64) @ X
    info = info_tensor(torch)
    for S in itertools.combinations(range(n), k):
        out = torch.full((q, s), float("nan"), dtype=torch.float32, device="cuda")
        lib.coded_decode(code, list(S), dY, q, out, info)
        torch.cuda.synchronize()
        assert int(info.item()) == 0
        # fp64 elimination leaves rounding of order 1e-15 of the largest term,
        # which fp32 output rounding does not remove near zero
        err = float(np.max(np.abs(out.cpu().numpy().astype(np.float64) - expect)))
        assert err <= 1e-12 * max(1.0, float(np.max(np.abs(expect)))), (S, err)


@pytest.mark.parametrize("n,k,q,s", [(16, 12, 4001, 1), (64, 48, 700, 8), (20, 16, 333, 2), (32, 24, 200, 4)])
def test_decode_gaussian_matches_oracle(lib, torch, n, k, q, s):
    r = 40
    P, A, X = make_inputs(n, k, q, r, s, 10)
    G = oc.systematic_generator(P)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    code = lib.Code(n, k, G, 2)
    dY = torch.from_numpy(Y).to("cuda")
    info = info_tensor(torch)
    rng = np.random.default_rng(0)
    for trial in range(25):
        S = sorted(rng.choice(n, size=k, replace=False).tolist())
        out = torch.empty((q, s), dtype=torch.float32, device="cuda")
        lib.coded_decode(code, S, dY, q, out, info)
        torch.cuda.synchronize()
        assert int(info.item()) == 0
        ref = oc.decode_from_all(G, S, Y, q)
        kappa = np.linalg.cond(G[S])
        assert normwise_rel_err(out.cpu().numpy(), ref) <= 2.0 ** -23 + 1e-14 * kappa * k


def test_decode_order_and_extra_survivors(lib, torch):
    n, k, q, s = 16, 12, 1000, 1
    P, A, X = make_inputs(n, k, q, 30, s, 11)
    G = oc.systematic_generator(P)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    code = lib.Code(n, k, G, 2)
    dY = torch.from_numpy(Y).to("cuda")
    info = info_tensor(torch)
    base = [0, 2, 3, 4, 5, 6, 8, 9, 12, 13, 14, 15]
    outs = []
    for order in (base, base[::-1], [13, 0, 15, 2, 12, 3, 14, 4, 9, 5, 8, 6] + [1, 7, 10]):
        out = torch.empty((q, s), dtype=torch.float32, device="cuda")
        lib.coded_decode(code, order, dY, q, out, info)
        outs.append(out.cpu().numpy())
    assert all(np.array_equal(outs[0], o) for o in outs[1:])
    # results of workers outside the set never matter
    Yp = Y.copy()
    Yp[[1, 7, 10, 11]] = np.nan
    out = torch.empty((q, s), dtype=torch.float32, device="cuda")
    lib.coded_decode(code, base, torch.from_numpy(Yp).to("cuda"), q, out, info)
    assert np.array_equal(out.cpu().numpy(), outs[0])


def test_decode_errors(lib, torch):
    n, k, q = 6, 4, 20
    code = lib.Code.systematic(vandermonde_parity(n, k), 2)
    Y = torch.zeros((n, code.qb(q), 1), dtype=torch.float64, device="cuda")
    out = torch.zeros((q, 1), dtype=torch.float32, device="cuda")
    info = info_tensor(torch)
    with pytest.raises(lib.CodedError) as e:
        lib.coded_decode(code, [0, 1, 2], Y, q, out, info)
    assert e.value.status == lib.CODED_ERR_TOO_FEW
    with pytest.raises(lib.CodedError) as e:
        lib.coded_decode(code, [0, 1, 2, 2], Y, q, out, info)
    assert e.value.status == lib.CODED_ERR_ARG
    with pytest.raises(lib.CodedError) as e:
        lib.coded_decode(code, [0, 1, 2, 6], Y, q, out, info)
    assert e.value.status == lib.CODED_ERR_ARG
    # a code with two equal parity rows is not MDS: that survivor set is singular
    Pbad = np.array([[1.0, 2.0, 3.0, 4.0], [1.0, 2.0, 3.0, 4.0]])
    bad = lib.Code.systematic(Pbad, 2)
    out.fill_(5.0)
    lib.coded_decode(bad, [0, 1, 4, 5], Y, q, out, info)
    torch.cuda.synchronize()
    assert int(info.item()) > 0
    assert np.all(out.cpu().numpy() == 5.0)          # nothing written
    with pytest.raises(oc.DecodeError):
        oc.decode(oc.systematic_generator(Pbad), [0, 1, 4, 5], [np.zeros((5, 1))] * 4, q)


def test_decode_batched_zero_sets(lib, torch):
    """An empty batch of survivor sets: nothing is enqueued, out and info untouched."""
    n, k, q, r, s = 8, 6, 60, 32, 1
    P, A, X = make_inputs(n, k, q, r, s, 61)
    code = lib.Code.systematic(P, 2)
    Y = lib.alloc_y(code, q, s, torch.float64)
    sets = torch.zeros((0, k), dtype=torch.int32, device="cuda")
    out = torch.zeros((0, q, s), dtype=torch.float32, device="cuda")
    info = torch.zeros(0, dtype=torch.int32, device="cuda")
    lib.coded_decode_batched(code, sets, Y, q, out, info)
    torch.cuda.synchronize()


def test_decode_batched_matches_single(lib, torch):
    n, k, q, s = 64, 48, 1000, 8
    P, A, X = make_inputs(n, k, q, 24, s, 12)
    G = oc.systematic_generator(P)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    code = lib.Code(n, k, G, 2)
    dY = torch.from_numpy(Y).to("cuda")
    sets, _ = lib.coded_draw_survivor_sets(n, k, 4, 40, min_parity=8)
    sets_ref, _ = oc.draw_survivor_sets(n, k, 4, 40, min_parity=8)
    assert np.array_equal(sets, sets_ref)
    # shuffle the order inside each row: decoding must not care
    rng = np.random.default_rng(1)
    shuffled = np.array([rng.permutation(row) for row in sets], dtype=np.int32)
    bad = shuffled.copy()
    bad[3, 5] = bad[3, 6]                           # repeated index
    bad[7, 0] = 64                                  # out of range
    dsets = torch.from_numpy(bad).to("cuda")
    out = torch.full((len(sets), q, s), float("nan"), dtype=torch.float32, device="cuda")
    info = info_tensor(torch, len(sets))
    lib.coded_decode_batched(code, dsets, dY, q, out, info)
    torch.cuda.synchronize()
    got, inf = out.cpu().numpy(), info.cpu().numpy()
    for b in range(len(sets)):
        if b in (3, 7):
            assert inf[b] == -1 and np.all(np.isnan(got[b]))
            continue
        assert inf[b] == 0
        ref = oc.decode_from_all(G, sets[b], Y, q)
        assert normwise_rel_err(got[b], ref) <= 2.0 ** -23 + 1e-14 * np.linalg.cond(G[sets[b]]) * k
        single = torch.empty((q, s), dtype=torch.float32, device="cuda")
        one = info_tensor(torch)
        lib.coded_decode(code, sets[b], dY, q, single, one)
        assert np.array_equal(single.cpu().numpy(), got[b])


# ---------------------------------------------------------------- end to end

def run_matmul(lib, torch, code, dA, par, dX, q, s, seed, draw, parity_ready):
    out = torch.empty((q, s) if s > 1 else (q,), dtype=torch.float32, device="cuda")
    ws = lib.matmul_workspace(code, dA, dX)
    info = info_tensor(torch)
    surv, t = lib.coded_matmul(code, dA, par, dX, out, ws, info, seed, draw, parity_ready=parity_ready)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    return out.cpu().numpy(), surv, t


def test_matmul_mds4x2_100_seeds(lib, torch):
    """The (4,2) workload: A 2048x512, x 512x1, fresh code and inputs per seed, seeds 0..99."""
    n, k, q, r = 4, 2, 2048, 512
    worst = 0.0
    for seed in range(100):
        P, A, X = make_inputs(n, k, q, r, 1, seed)
        code = lib.Code.systematic(P, 2)
        dA, dX = device_tensor(A), device_tensor(X[:, 0])
        par = lib.alloc_parity(code, q, r, torch.float32)
        out, surv, t = run_matmul(lib, torch, code, dA, par, dX, q, 1, seed, 0, parity_ready=False)
        S, T = oc.draw_survivors(n, k, seed, 0)
        assert np.array_equal(surv, S)
        assert t == pytest.approx(T, rel=1e-15)
        err = normwise_rel_err(out, oc.plain_product(A, X))
        worst = max(worst, err)
    assert worst <= TOL_F32, worst


@pytest.mark.parametrize("n,k,q,r,s", [(16, 12, 5000, 1500, 1), (64, 48, 1500, 512, 8), (20, 16, 3001, 257, 1),
                                       (5, 5, 10, 8, 1), (7, 1, 13, 9, 2), (16, 12, 11, 64, 1)])
def test_matmul_small_shapes_match_oracle(lib, torch, n, k, q, r, s):
    P, A, X = make_inputs(n, k, q, r, s, 13)
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A), device_tensor(X[:, 0] if s == 1 else X)
    par = lib.alloc_parity(code, q, r, torch.float32)
    ref = oc.plain_product(A, X)
    G = oc.systematic_generator(P)
    for draw in range(6):
        out, surv, _ = run_matmul(lib, torch, code, dA, par, dX, q, s, 13, draw, parity_ready=draw > 0)
        S, _ = oc.draw_survivors(n, k, 13, draw)
        assert np.array_equal(surv, S)
        assert normwise_rel_err(out.reshape(q, s), ref) <= TOL_F32
        # and against the oracle's own coded pipeline on the same survivors
        y_or = oc.decode_from_all(G, S, oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X), q)
        assert normwise_rel_err(out.reshape(q, s), y_or) <= TOL_F32


def test_matmul_bf16_dense_regime_small(lib, torch):
    """bf16 A and X, (32,24) code, 64 columns, fp32 accumulation: within 2e-2 of the fp64 product."""
    n, k, q, r, s = 32, 24, 2400, 384, 64
    P, A, X = make_inputs(n, k, q, r, s, 14, "bf16")
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A, "bf16"), device_tensor(X, "bf16")
    par = lib.alloc_parity(code, q, r, torch.bfloat16)
    ref = oc.plain_product(A, X)
    for draw in range(4):
        out, surv, _ = run_matmul(lib, torch, code, dA, par, dX, q, s, 14, draw, parity_ready=False)
        assert np.array_equal(surv, oc.draw_survivors(n, k, 14, draw)[0])
        assert normwise_rel_err(out, ref) <= TOL_BF16


def test_matmul_deterministic(lib, torch):
    n, k, q, r = 16, 12, 6000, 2048
    P, A, X = make_inputs(n, k, q, r, 1, 15)
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A), device_tensor(X[:, 0])
    par = lib.alloc_parity(code, q, r, torch.float32)
    a, _, _ = run_matmul(lib, torch, code, dA, par, dX, q, 1, 15, 3, parity_ready=False)
    b, _, _ = run_matmul(lib, torch, code, dA, par, dX, q, 1, 15, 3, parity_ready=False)
    assert np.array_equal(a, b)


def test_matmul_empty_and_argument_errors(lib, torch):
    code = lib.Code.systematic(synth.parity_matrix(6, 4, 1), 2)
    A = torch.zeros((0, 8), dtype=torch.float32, device="cuda")
    X = torch.zeros(8, dtype=torch.float32, device="cuda")
    out = torch.zeros(0, dtype=torch.float32, device="cuda")
    ws = torch.zeros(1, dtype=torch.float64, device="cuda")
    par = torch.zeros(1, dtype=torch.float32, device="cuda")
    info = info_tensor(torch)
    surv, _ = lib.coded_matmul(code, A, par, X, out, ws, info, 1, 0, parity_ready=False)
    torch.cuda.synchronize()
    assert len(surv) == 4 and int(info.item()) == 0
    with pytest.raises(ValueError):
        lib.coded_matmul(code, torch.zeros((4, 8), device="cuda"), par, torch.zeros(7, device="cuda"), out, ws, info,
                         1, 0)


@pytest.mark.parametrize("s,pad", [(8, 4), (8, 1), (4, 0), (3, 0), (12, 4)])
def test_decode_many_missing_blocks_and_strided_out(lib, torch, s, pad):
    """Sets with up to 20 parity survivors (several register passes), outputs with
    row stride ldo = s + pad, fp64 and fp32 worker results."""
    n, k, q, r = 48, 24, 500, 16
    P, A, X = make_inputs(n, k, q, r, s, 16)
    G = oc.systematic_generator(P)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    code = lib.Code(n, k, G, 2)
    rng = np.random.default_rng(3)
    sets = []
    for mm in (0, 1, 7, 8, 9, 15, 16, 17, 20, 24):
        par = rng.choice(np.arange(k, n), size=mm, replace=False)
        sysw = rng.choice(np.arange(k), size=k - mm, replace=False)
        sets.append(np.sort(np.concatenate([sysw, par])).astype(np.int32))
    for ydt in (torch.float64, torch.float32):
        dY = torch.from_numpy(Y).to("cuda").to(ydt)
        base = torch.full((len(sets), q, s + pad), float("nan"), dtype=torch.float32, device="cuda")
        out = base[:, :, :s]
        info = info_tensor(torch, len(sets))
        lib.coded_decode_batched(code, torch.from_numpy(np.stack(sets)).cuda(), dY, q, out, info)
        torch.cuda.synchronize()
        assert np.all(info.cpu().numpy() == 0)
        got_all = base.cpu().numpy()
        for bi, S in enumerate(sets):
            ref = oc.decode_from_all(G, S, Y, q)
            tol = (2.0 ** -23 if ydt == torch.float64 else 2.0 ** -20) + 1e-14 * np.linalg.cond(G[S]) * k
            if ydt == torch.float32:
                tol += 2.0 ** -23 * np.linalg.cond(G[S]) * k
            assert normwise_rel_err(got_all[bi, :, :s], ref) <= tol, (bi, ydt)
            assert np.all(np.isnan(got_all[bi, :, s:]))          # the row padding is never written
            single = torch.full((q, s + pad), float("nan"), dtype=torch.float32, device="cuda")
            lib.coded_decode(code, S, dY, q, single[:, :s], info[:1])
            torch.cuda.synchronize()
            assert np.array_equal(single.cpu().numpy()[:, :s], got_all[bi, :, :s])


@pytest.mark.parametrize("q,r", [(1, 1), (63, 65), (128, 64), (300, 17)])
def test_transpose_exact(lib, torch, q, r):
    A = synth.gaussian((q, r), 17, synth.STREAM_A)
    dA = torch.from_numpy(A).cuda()
    AT = torch.full((r, q), float("nan"), dtype=torch.float32, device="cuda")
    lib.coded_transpose(dA, AT)
    torch.cuda.synchronize()
    assert np.array_equal(AT.cpu().numpy(), A.T)


@pytest.mark.parametrize("q,r,n1,k1,n2,k2", [(4001, 96, 20, 16, 20, 16), (700, 50, 6, 4, 7, 5)])
def test_coded_gd_matches_oracle_iterates(lib, torch, q, r, n1, k1, n2, k2):
    """Coded gradient descent (Sec. III-E): every iterate against the oracle's coded_gd."""
    seed = 18
    A = synth.gaussian((q, r), seed, synth.STREAM_A, std=1.0 / np.sqrt(r))
    w = synth.gaussian((r,), seed, synth.STREAM_WSTAR)
    y = (oc.plain_product(A, w)[:, 0] + 0.1 * synth.gaussian((q,), seed, synth.STREAM_NOISE)).astype(np.float32)
    P1 = synth.parity_matrix(n1, k1, seed)
    P2 = synth.parity_matrix(n2, k2, seed, synth.STREAM_PT)
    eta = 0.5 * r / q                      # step normalised by the mean Hessian scale q * sigma^2
    iters = 25
    rec = []
    oc.coded_gd(A, y, np.zeros(r), oc.systematic_generator(P1), oc.systematic_generator(P2), eta, iters, seed,
                record=rec)
    cA, cT = lib.Code.systematic(P1, 2), lib.Code.systematic(P2, 2)
    dA = torch.from_numpy(A).cuda()
    dAT = torch.empty((r, q), dtype=torch.float32, device="cuda")
    lib.coded_transpose(dA, dAT)
    pA, pT = lib.alloc_parity(cA, q, r, torch.float32), lib.alloc_parity(cT, r, q, torch.float32)
    lib.coded_encode(cA, dA, pA)
    lib.coded_encode(cT, dAT, pT)
    dy = torch.from_numpy(y).cuda()
    x = torch.zeros(r, dtype=torch.float32, device="cuda")
    ws = torch.empty(lib.coded_gd_sizes(cA, cT, q, r), dtype=torch.uint8, device="cuda")
    info = torch.full((2,), 9, dtype=torch.int32, device="cuda")
    for t in range(iters):
        S1, S2 = lib.coded_gd_step(cA, cT, dA, pA, dAT, pT, dy, x, eta, seed, t, ws, info)
        assert np.array_equal(S1, oc.draw_survivors(n1, k1, seed, 2 * t)[0])
        assert np.array_equal(S2, oc.draw_survivors(n2, k2, seed, 2 * t + 1)[0])
        torch.cuda.synchronize()
        assert np.all(info.cpu().numpy() == 0)
        xt = x.cpu().numpy().astype(np.float64)
        assert np.max(np.abs(xt - rec[t])) <= 1e-4 * np.max(np.abs(rec[t])), t


def test_conditioned_generator_single_plane_every_survivor_set(lib, torch):
    """One fp32 parity plane (no lo plane) with the certified (16,12) generator
    of the GEMV regime: every one of the C(16,12) = 1820 survivor sets decodes
    within the fp32 tolerance.  The plain seed-2 draw, whose worst decode
    system is 6.8 times worse conditioned, does worse on its worst set."""
    w = synth.WORKLOADS["gemv16x12_conditioned_65536x8192"]
    n, k, q, r = w.n, w.k, 12000, 8192
    Pc, _, _ = synth.conditioned_parity_matrix(n, k, w.seed, w.extra["candidates"], pick=w.extra["parity_candidate"])
    A = synth.gaussian((q, r), 41, synth.STREAM_A)
    x = synth.gaussian((r,), 41, synth.STREAM_X)
    ref = oc.plain_product(A, x[:, None])[:, 0]
    sets = np.array(list(itertools.combinations(range(n), k)), dtype=np.int32)
    dA, dx, dsets = torch.from_numpy(A).cuda(), torch.from_numpy(x).cuda(), torch.from_numpy(sets).cuda()
    worst = {}
    for name, P in (("conditioned", Pc), ("plain", synth.parity_matrix(n, k, w.seed))):
        code = lib.Code.systematic(P, 1)
        par = lib.alloc_parity(code, q, r, torch.float32)
        lib.coded_encode(code, dA, par)
        Y = lib.alloc_y(code, q, 1, torch.float64)
        lib.coded_worker_mm(code, dA, par, dx, Y)
        out = torch.empty((len(sets), q), dtype=torch.float32, device="cuda")
        info = info_tensor(torch, len(sets))
        lib.coded_decode_batched(code, dsets, Y, q, out, info)
        torch.cuda.synchronize()
        assert np.all(info.cpu().numpy() == 0)
        got = out.cpu().numpy()
        worst[name] = float(np.max(np.max(np.abs(got - ref[None, :]), axis=1)) / np.max(np.abs(ref)))
    assert worst["conditioned"] <= TOL_F32, worst
    assert worst["plain"] > worst["conditioned"], worst


@pytest.mark.parametrize("which", ["A", "T"])
def test_conditioned_gd_codes_single_plane_every_survivor_set(lib, torch, which):
    """The coded gradient-descent codes' certified (20,16) generators with one fp32
    parity plane: every one of the C(20,16) = 4845 survivor sets decodes A x
    within the fp32 tolerance (code of A and code of A^T, each on its own
    matrix).  The plain draw of the code of A (worst decode system 62 times worse
    conditioned) misses the tolerance on its worst set."""
    w = synth.WORKLOADS["gd20x16_conditioned_262144x4096"]
    n, k, q, r = w.n, w.k, 16000, 2048
    PA, PT, planes = synth.gd_codes(w)
    Pc = PA if which == "A" else PT
    A = synth.gaussian((q, r), 43, synth.STREAM_A)
    x = synth.gaussian((r,), 43, synth.STREAM_X)
    ref = oc.plain_product(A, x[:, None])[:, 0]
    sets = np.array(list(itertools.combinations(range(n), k)), dtype=np.int32)
    dA, dx, dsets = torch.from_numpy(A).cuda(), torch.from_numpy(x).cuda(), torch.from_numpy(sets).cuda()
    cands = [("conditioned", Pc)]
    if which == "A":
        cands.append(("plain", synth.parity_matrix(n, k, w.seed)))
    worst = {}
    for name, P in cands:
        code = lib.Code.systematic(P, planes)
        par = lib.alloc_parity(code, q, r, torch.float32)
        lib.coded_encode(code, dA, par)
        Y = lib.alloc_y(code, q, 1, torch.float64)
        lib.coded_worker_mm(code, dA, par, dx, Y)
        out = torch.empty((len(sets), q), dtype=torch.float32, device="cuda")
        info = info_tensor(torch, len(sets))
        lib.coded_decode_batched(code, dsets, Y, q, out, info)
        torch.cuda.synchronize()
        assert np.all(info.cpu().numpy() == 0)
        got = out.cpu().numpy()
        worst[name] = float(np.max(np.max(np.abs(got - ref[None, :]), axis=1)) / np.max(np.abs(ref)))
    print(f"one plane, every survivor set of the code of {which}: worst normwise error {worst}")
    assert worst["conditioned"] <= TOL_F32, worst
    if "plain" in worst:
        assert worst["plain"] > TOL_F32, worst


@pytest.mark.parametrize("n,k", [(64, 48), (20, 13)])
@pytest.mark.parametrize("s,pad", [(8, 0), (8, 4), (4, 2), (12, 0)])
def test_decode_matrix_core_path_roles_and_strided_out(lib, torch, n, k, s, pad):
    """The matrix-core decode with four-element vectors (s a multiple of 4): the
    copying wave and the three combining waves, dense rows (ldo == s) and padded
    rows, k a multiple of 4 (no padding steps) or not, sets with 0 to min(k, n-k)
    missing blocks; against the oracle and bit for bit against single decodes."""
    q, r = 1000, 24
    P, A, X = make_inputs(n, k, q, r, s, 21)
    G = oc.systematic_generator(P)
    Y = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    code = lib.Code(n, k, G, 2)
    dY = torch.from_numpy(Y).to("cuda")
    mmax = min(k, n - k)
    sets = np.concatenate([synth.exact_parity_sets(n, k, m, 2, 5) for m in sorted({0, 1, 3, mmax // 2, mmax})])
    base = torch.full((len(sets), q, s + pad), float("nan"), dtype=torch.float32, device="cuda")
    out = base[:, :, :s]
    info = info_tensor(torch, len(sets))
    lib.coded_decode_batched(code, torch.from_numpy(sets).cuda(), dY, q, out, info)
    torch.cuda.synchronize()
    assert np.all(info.cpu().numpy() == 0)
    got_all = base.cpu().numpy()
    for bi, S in enumerate(sets):
        ref = oc.decode_from_all(G, S, Y, q)
        tol = 2.0 ** -23 + 1e-14 * np.linalg.cond(G[np.sort(S)]) * k
        assert normwise_rel_err(got_all[bi, :, :s], ref) <= tol, bi
        if pad:
            assert np.all(np.isnan(got_all[bi, :, s:]))
        single = torch.full((q, s + pad), float("nan"), dtype=torch.float32, device="cuda")
        lib.coded_decode(code, S, dY, q, single[:, :s], info[:1])
        torch.cuda.synchronize()
        assert np.array_equal(single.cpu().numpy()[:, :s], got_all[bi, :, :s]), bi
