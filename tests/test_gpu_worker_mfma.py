"""Multi-column fp32 worker products on the fp64 matrix cores (Sec. III-A: every
worker multiplies its stored coded block by the multicast input X, here with
s > 1 columns), through the C ABI against the oracle.

Integer-valued inputs make every product and partial sum exact in fp64, so Y
must equal the oracle's bit for bit whatever the summation order; Gaussian
inputs are held to a rounding bound.  The shapes cover every column variant
(4-column tiles for s <= 8, 16-column tiles above, launches of at most 64
columns), several row tiles with a ragged last one, zero-padded rows (q not a
multiple of k), K tails (r not a multiple of the K chunk) and both plane
counts."""
import numpy as np
import pytest

from oracle import coded as oc
from tests.gpu_helpers import device_tensor, make_inputs, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t

S_CASES = [2, 3, 4, 5, 8, 9, 16, 17, 32, 33, 64, 65, 100]


def _run(lib, torch, P, A, X, planes, mask=None, ldx_pad=0):
    n, k = P.shape[0] + P.shape[1], P.shape[1]
    q, r = A.shape
    s = X.shape[1]
    code = lib.Code.systematic(P, planes)
    dA = device_tensor(A)
    if ldx_pad:
        Xp = np.zeros((r, s + ldx_pad), dtype=np.float32)
        Xp[:, :s] = X
        dX = device_tensor(Xp)[:, :s]
    else:
        dX = device_tensor(X)
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    Y = lib.alloc_y(code, q, s, torch.float64)
    Y.fill_(float("nan"))
    lib.coded_worker_mm(code, dA, par, dX, Y, worker_mask=mask)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


@pytest.mark.parametrize("s", S_CASES)
@pytest.mark.parametrize("planes", [1, 2])
def test_multicolumn_products_integer_bit_exact(lib, torch, s, planes):
    n, k, q, r = 20, 16, 1999, 520          # qb = 125: four 32-row tiles, the last ragged; 8 padding rows
    P, A, X = make_inputs(n, k, q, r, s, 40 + s, integer=True)
    got = _run(lib, torch, P, A, X, planes)
    ref = oc.worker_products(oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k)), X)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("n,k,q,r,s", [(64, 48, 700, 256, 8), (4, 2, 66, 4, 2), (5, 3, 31, 4100, 6),
                                       (3, 1, 40, 128, 12), (4, 4, 33, 132, 7), (64, 48, 16384, 4096, 8)])
def test_multicolumn_products_shapes_integer_bit_exact(lib, torch, n, k, q, r, s):
    """r of one 16-byte piece, a K tail of 4 elements, k = 1, n = k (no parity),
    and the decode-heavy shape at full size."""
    P, A, X = make_inputs(n, k, q, r, s, 9, integer=True)
    got = _run(lib, torch, P, A, X, 2)
    ref = oc.worker_products(oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k)), X)
    assert np.array_equal(got, ref)


def test_multicolumn_products_mask_and_strided_x(lib, torch):
    n, k, q, r, s = 16, 12, 900, 264, 10
    P, A, X = make_inputs(n, k, q, r, s, 12, integer=True)
    mask = np.zeros(n, dtype=np.uint8)
    mask[[1, 11, 12, 15]] = 1
    code = lib.Code.systematic(P, 2)
    dA = device_tensor(A)
    Xp = np.zeros((r, s + 3), dtype=np.float32)
    Xp[:, :s] = X
    dX = device_tensor(Xp)[:, :s]                      # row stride s + 3
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    Y = lib.alloc_y(code, q, s, torch.float64)
    Y.fill_(-7.0)
    lib.coded_worker_mm(code, dA, par, dX, Y, worker_mask=mask)
    torch.cuda.synchronize()
    got = Y.cpu().numpy()
    ref = oc.worker_products(oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, k)), X)
    for i in range(n):
        if mask[i]:
            assert np.array_equal(got[i], ref[i]), i
        else:
            assert np.all(got[i] == -7.0), i


@pytest.mark.parametrize("s", [2, 3, 8, 16, 64])
@pytest.mark.parametrize("planes", [1, 2])
def test_multicolumn_products_gaussian(lib, torch, s, planes):
    """fp64 sums of exact fp32 products: within 1e-12 of the fp64 oracle relative to
    sum |a||x| on systematic rows; parity rows also carry their planes' rounding."""
    n, k, q, r = 64, 48, 3000, 1024
    P, A, X = make_inputs(n, k, q, r, s, 70 + s)
    got = _run(lib, torch, P, A, X, planes)
    G = oc.systematic_generator(P)
    coded = oc.encode(G, oc.pad_and_split(A, k))
    ref = oc.worker_products(coded, X)
    bound = oc.worker_products(np.abs(coded), np.abs(X))
    parity_u = 2.0 ** -46 if planes == 2 else 2.0 ** -24
    err = np.abs(got - ref)
    assert np.all(err[:k] <= 1e-12 * bound[:k])
    assert np.all(err[k:] <= (1e-12 + parity_u) * bound[k:])


def test_multicolumn_products_match_single_columns(lib, torch):
    """Column c of a multi-column product equals the GEMV kernel's product with X[:, c]
    to fp64 rounding (different summation orders)."""
    n, k, q, r, s = 16, 12, 2400, 2048, 5
    P, A, X = make_inputs(n, k, q, r, s, 5)
    code = lib.Code.systematic(P, 2)
    dA = device_tensor(A)
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    Y = lib.alloc_y(code, q, s, torch.float64)
    lib.coded_worker_mm(code, dA, par, device_tensor(X), Y)
    y1 = lib.alloc_y(code, q, 1, torch.float64)
    torch.cuda.synchronize()
    multi = Y.cpu().numpy()
    for c in range(s):
        lib.coded_worker_mm(code, dA, par, device_tensor(np.ascontiguousarray(X[:, c])), y1)
        torch.cuda.synchronize()
        single = y1.cpu().numpy()[:, :, 0]
        scale = np.max(np.abs(single))
        assert np.max(np.abs(multi[:, :, c] - single)) <= 1e-13 * scale
