"""fp32 codes whose lo parity plane is stored in bfloat16 (CODED_PLANES_LO_BF16),
through the C ABI against the fp64 oracle.

A parity block (Sec. III-A: the coded block a parity worker stores) is kept as
hi = fp32(sum) and lo = bf16(fp32(sum - hi)), 6 bytes per element instead of
8.  hi + lo is within (2^-33 + 2^-48)|sum| of the exact fp64 sum: the fp32
remainder carries at most 2^-24 of |sum| and bfloat16 keeps 8 significand
bits of it.  Integer-valued inputs have a zero remainder, so those cases
compare bit for bit.  Every survivor set of the (16,12) code decodes within
the fp32 tolerance.
"""
import itertools

import numpy as np
import pytest

import synth
from oracle import coded as oc
from tests.gpu_helpers import device_tensor, make_inputs, normwise_rel_err, torch_mod

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4
LO_BF16_U = 2.0 ** -33 + 2.0 ** -48      # relative error of hi + lo against the exact sum


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def _planes_np(lib, torch, code, par, q, r):
    hi, lo = lib.parity_planes(code, par, q, r)
    return hi.cpu().numpy().astype(np.float64), lo.float().cpu().numpy().astype(np.float64)


def _encode(lib, torch, P, A, planes):
    q, r = A.shape
    code = lib.Code.systematic(P, planes)
    dA = device_tensor(A)
    par = lib.alloc_parity(code, q, r, torch.float32)
    par.fill_(0x7F)
    lib.coded_encode(code, dA, par)
    torch.cuda.synchronize()
    return code, dA, par


def test_lo_bf16_parity_sizes(lib, torch):
    P, _, _ = make_inputs(16, 12, 10, 8, 1, 1)
    code = lib.Code.systematic(P, lib.CODED_PLANES_LO_BF16)
    q, r = 1000, 520
    qb = -(-q // 12)
    assert lib.coded_sizes(code, lib.CODED_F32, lib.CODED_F64, q, r, 1)[0] == 6 * 4 * qb * r
    # bf16 inputs: the mode is for fp32 codes; bf16 parity stays two bf16 planes
    assert lib.coded_sizes(code, lib.CODED_BF16, lib.CODED_F32, q, r, 1)[0] == 2 * 2 * 4 * qb * r
    assert lib.alloc_parity(code, q, r, torch.float32).numel() == 6 * 4 * qb * r


@pytest.mark.parametrize("n,k,q,r", [(16, 12, 1000, 520), (5, 3, 31, 7), (64, 48, 700, 256)])
def test_encode_lo_bf16_integer_bit_exact(lib, torch, n, k, q, r):
    P, A, _ = make_inputs(n, k, q, r, 1, 3, integer=True)
    code, _, par = _encode(lib, torch, P, A, lib.CODED_PLANES_LO_BF16)
    hi, lo = _planes_np(lib, torch, code, par, q, r)
    ref = oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k))[k:]
    assert np.array_equal(hi, ref)
    assert np.all(lo == 0)


@pytest.mark.parametrize("n,k,q,r", [(16, 12, 2000, 1030), (16, 12, 1500, 1024), (64, 48, 400, 100)])
def test_encode_lo_bf16_gaussian(lib, torch, n, k, q, r):
    """hi + lo against the fp64 oracle within the split's bound (plus the two
    fp64 sums' rounding); the hi plane is the two-plane code's hi plane."""
    P, A, _ = make_inputs(n, k, q, r, 1, 4)
    code, _, par = _encode(lib, torch, P, A, lib.CODED_PLANES_LO_BF16)
    hi, lo = _planes_np(lib, torch, code, par, q, r)
    blocks = oc.pad_and_split(A, k)
    ref = oc.encode(oc.systematic_generator(P), blocks)[k:]
    scale = np.abs(oc.encode(oc.systematic_generator(np.abs(P)), np.abs(blocks))[k:])
    assert np.all(np.abs(hi + lo - ref) <= (LO_BF16_U + 4 * k * 2.0 ** -53) * scale)
    # the remainder is not dropped: a plain fp32 plane misses this bound on Gaussian data
    assert np.max(np.abs(hi - ref) / np.maximum(scale, 1e-300)) > 2.0 ** -30
    _, _, par2 = _encode(lib, torch, P, A, 2)
    assert np.array_equal(par2[0].cpu().numpy().astype(np.float64), hi)


@pytest.mark.parametrize("n,k,q,r", [(16, 12, 1000, 8192), (16, 12, 777, 2052), (64, 48, 700, 256), (5, 3, 31, 7)])
def test_worker_products_lo_bf16_integer_bit_exact(lib, torch, n, k, q, r):
    """GEMV (r a multiple of 4: the vector kernel) and general-shape products."""
    P, A, X = make_inputs(n, k, q, r, 1, 6, integer=True)
    code, dA, par = _encode(lib, torch, P, A, lib.CODED_PLANES_LO_BF16)
    Y = lib.alloc_y(code, q, 1, torch.float64)
    Y.fill_(float("nan"))
    lib.coded_worker_mm(code, dA, par, device_tensor(X[:, 0]), Y)
    torch.cuda.synchronize()
    ref = oc.worker_products(oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k)), X)
    assert np.array_equal(Y.cpu().numpy(), ref)


@pytest.mark.parametrize("n,k,q,r,s", [(16, 12, 3000, 8192, 1), (16, 12, 999, 1028, 1), (16, 12, 500, 260, 3),
                                       (5, 3, 40, 9, 2)])
def test_worker_products_lo_bf16_gaussian(lib, torch, n, k, q, r, s):
    """fp64 sums of exact products: systematic rows within 1e-12 of the oracle
    relative to sum |a||x|, parity rows also within the planes' 2^-33 split."""
    P, A, X = make_inputs(n, k, q, r, s, 7)
    code, dA, par = _encode(lib, torch, P, A, lib.CODED_PLANES_LO_BF16)
    Y = lib.alloc_y(code, q, s, torch.float64)
    lib.coded_worker_mm(code, dA, par, device_tensor(X[:, 0] if s == 1 else X), Y)
    torch.cuda.synchronize()
    coded = oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k))
    ref = oc.worker_products(coded, X)
    bound = oc.worker_products(np.abs(coded), np.abs(X))
    err = np.abs(Y.cpu().numpy() - ref)
    assert np.all(err[:k] <= 1e-12 * bound[:k])
    assert np.all(err[k:] <= (1e-12 + LO_BF16_U) * bound[k:])


def test_lo_bf16_every_survivor_set(lib, torch):
    """The (16,12) Gaussian code of the GEMV workload (the generator the two-plane
    code uses): every one of the C(16,12) = 1820 survivor sets decodes A x
    within the fp32 tolerance with the 6-byte parity planes."""
    w = synth.WORKLOADS["gemv16x12_65536x8192"]
    n, k, q, r = w.n, w.k, 12000, 8192
    P = synth.parity_matrix(n, k, w.seed)
    A = synth.gaussian((q, r), 47, synth.STREAM_A)
    x = synth.gaussian((r,), 47, synth.STREAM_X)
    ref = oc.plain_product(A, x[:, None])[:, 0]
    sets = np.array(list(itertools.combinations(range(n), k)), dtype=np.int32)
    code = lib.Code.systematic(P, lib.CODED_PLANES_LO_BF16)
    dA, dx, dsets = torch.from_numpy(A).cuda(), torch.from_numpy(x).cuda(), torch.from_numpy(sets).cuda()
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    Y = lib.alloc_y(code, q, 1, torch.float64)
    lib.coded_worker_mm(code, dA, par, dx, Y)
    out = torch.empty((len(sets), q), dtype=torch.float32, device="cuda")
    info = torch.full((len(sets),), 12345, dtype=torch.int32, device="cuda")
    lib.coded_decode_batched(code, dsets, Y, q, out, info)
    torch.cuda.synchronize()
    assert np.all(info.cpu().numpy() == 0)
    got = out.cpu().numpy()
    worst = float(np.max(np.max(np.abs(got - ref[None, :]), axis=1)) / np.max(np.abs(ref)))
    print(f"bf16 lo plane, every survivor set: worst normwise error {worst:.3e}")
    assert worst <= TOL_F32


def test_lo_bf16_coded_matmul_full_size(lib, torch):
    """The GEMV workload at full size (65536 x 8192, (16,12)) through coded_matmul
    with 6-byte parity: four draws, each survivor set bit for bit and the
    decoded product within the fp32 tolerance of the oracle's fp64 product."""
    w = synth.WORKLOADS["gemv16x12_65536x8192"]
    n, k, q, r, seed = w.n, w.k, w.q, w.r, w.seed
    A = synth.gaussian_rows(q, r, seed, synth.STREAM_A)
    P = synth.parity_matrix(n, k, seed)
    code = lib.Code.systematic(P, lib.CODED_PLANES_LO_BF16)
    dA = torch.from_numpy(A).cuda()
    par = lib.alloc_parity(code, q, r, torch.float32)
    ws = lib.alloc_y(code, q, 1, torch.float64)
    out = torch.empty(q, dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    A64 = A.astype(np.float64)
    for t in range(4):
        x = synth.gaussian((r,), seed, synth.STREAM_X, t)
        surv, _ = lib.coded_matmul(code, dA, par, torch.from_numpy(x).cuda(), out, ws, info, seed, t,
                                   parity_ready=t > 0)
        torch.cuda.synchronize()
        assert np.array_equal(surv, oc.draw_survivors(n, k, seed, t)[0]) and int(info.item()) == 0
        ref = oc.plain_product(A64, x)[:, 0]
        err = float(np.max(np.abs(out.cpu().numpy() - ref)) / np.max(np.abs(ref)))
        assert err <= TOL_F32, (t, err)
