"""coded_matmul on small fp32 problems with one column runs as one launch
(encode unless the planes are ready, all n worker products, decode).  Its
planes must equal coded_encode's bit for bit, its worker results and output
must equal the separate steps' (coded_encode, coded_worker_mm, coded_decode)
up to fp64 summation order, and the output must match the fp64 oracle."""
import ctypes

import numpy as np
import pytest

from oracle import coded as oc
from tests.gpu_helpers import device_tensor, make_inputs, normwise_rel_err, torch_mod

pytestmark = pytest.mark.gpu

# (n, k, q, r): the configured (4,2) shape; padding rows (q % k != 0) with the
# 64-thread variant; 260 columns (a partial chunk) with 128 threads; the
# 256-thread variant over several column chunks; a single block row; the
# widest code served; three and two workers (the n <= 4 sums with absent
# values)
SHAPES = [(4, 2, 2048, 512), (5, 3, 31, 8), (6, 4, 1001, 260), (16, 12, 700, 1024), (7, 4, 3, 4),
          (16, 8, 2000, 2048), (3, 2, 999, 132), (2, 1, 65, 64)]


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def one_pass(lib, torch, code, dA, par, dx, q, seed, draw, parity_ready):
    """coded_matmul; returns (out, survivors, Y as n x qb, info)."""
    out = torch.full((q,), float("nan"), dtype=torch.float32, device="cuda")
    ws = lib.matmul_workspace(code, dA, dx)
    info = torch.full((1,), 12345, dtype=torch.int32, device="cuda")
    surv, _ = lib.coded_matmul(code, dA, par, dx, out, ws, info, seed, draw, parity_ready=parity_ready)
    torch.cuda.synchronize()
    qb = code.qb(q)
    Y = ws[: 8 * code.n * qb].view(torch.float64).view(code.n, qb).cpu().numpy()
    return out.cpu().numpy(), surv, Y, int(info.item())


def three_steps(lib, torch, code, dA, dx, q, r, survivors):
    """The same product through the separate entry points."""
    par = lib.alloc_parity(code, q, r, torch.float32)
    lib.coded_encode(code, dA, par)
    Y = lib.alloc_y(code, q, 1, torch.float64)
    lib.coded_worker_mm(code, dA, par, dx, Y)
    out = torch.full((q,), float("nan"), dtype=torch.float32, device="cuda")
    info = torch.full((1,), 12345, dtype=torch.int32, device="cuda")
    lib.coded_decode(code, survivors, Y, q, out, info)
    torch.cuda.synchronize()
    return par, Y.view(code.n, code.qb(q)).cpu().numpy(), out.cpu().numpy(), int(info.item())


@pytest.mark.parametrize("n,k,q,r", SHAPES)
@pytest.mark.parametrize("planes", [1, 2])
def test_one_pass_matches_steps_and_oracle(lib, torch, n, k, q, r, planes):
    P, A, X = make_inputs(n, k, q, r, 1, 41)
    code = lib.Code.systematic(P, planes)
    dA, dx = device_tensor(A), device_tensor(X[:, 0])
    par = lib.alloc_parity(code, q, r, torch.float32)
    par.fill_(123.0)
    ref = oc.plain_product(A, X)
    for draw in range(4):
        out, surv, Y1, info = one_pass(lib, torch, code, dA, par, dx, q, 41, draw, parity_ready=False)
        assert info == 0
        assert np.array_equal(surv, oc.draw_survivors(n, k, 41, draw)[0])
        p3, Y3, out3, info3 = three_steps(lib, torch, code, dA, dx, q, r, surv)
        assert info3 == 0
        # the planes, bit for bit
        assert torch.equal(par, p3)
        # every worker's result: fp64 sums of exact products, in another order
        planes_np = np.abs(p3.cpu().numpy().astype(np.float64)).sum(axis=0)
        mag = oc.worker_products(np.concatenate([np.abs(oc.pad_and_split(A, k)), planes_np]), np.abs(X))[..., 0]
        assert np.all(np.abs(Y1 - Y3) <= 2 * r * 2.0 ** -52 * mag)
        # the decoded product
        assert normwise_rel_err(out, out3) <= 1e-6
        assert normwise_rel_err(out, ref) <= 1e-4
        # with the planes ready the stored planes are read: same result
        out2, surv2, Y2, info2 = one_pass(lib, torch, code, dA, par, dx, q, 41, draw, parity_ready=True)
        assert info2 == 0 and np.array_equal(surv2, surv)
        assert np.array_equal(out2, out) and np.array_equal(Y2, Y1)


def test_one_pass_integer_bit_exact(lib, torch):
    """Integer-valued inputs make every worker sum exact: the one-pass worker
    results equal the separate steps' bit for bit.  The parity rows are
    Vandermonde with nodes 1..k (every square sub-block is nonsingular), so
    every survivor set decodes; the fp64 elimination leaves rounding of order
    1e-15 of the largest term, which fp32 output rounding does not remove
    near zero, so the outputs are held to that."""
    from tests.test_gpu_parity import vandermonde_parity
    n, k, q, r = 6, 4, 1003, 516
    _, A, X = make_inputs(n, k, q, r, 1, 42, integer=True)
    P = vandermonde_parity(n, k)
    code = lib.Code.systematic(P, 2)
    dA, dx = device_tensor(A), device_tensor(X[:, 0])
    par = lib.alloc_parity(code, q, r, torch.float32)
    exact = oc.plain_product(A, X)[:, 0]
    bound = 1e-12 * max(1.0, float(np.max(np.abs(exact))))
    for draw in range(6):
        out, surv, Y1, info = one_pass(lib, torch, code, dA, par, dx, q, 42, draw, parity_ready=False)
        p3, Y3, out3, info3 = three_steps(lib, torch, code, dA, dx, q, r, surv)
        assert info == 0 and info3 == 0
        assert np.array_equal(Y1, Y3)
        assert float(np.max(np.abs(out.astype(np.float64) - exact))) <= bound
        assert float(np.max(np.abs(out3.astype(np.float64) - exact))) <= bound


def test_one_pass_singular_set_leaves_out_untouched(lib, torch):
    """Dependent parity rows and both parity workers surviving: info names the
    zero pivot, out is not written (as coded_decode), and Y still holds every
    worker's product."""
    n, k, q, r, seed = 4, 2, 64, 16, 3
    P = np.array([[1.0, 2.0], [2.0, 4.0]])
    rng = np.random.default_rng(5)
    A = rng.integers(-3, 4, size=(q, r)).astype(np.float32)
    x = rng.integers(-3, 4, size=r).astype(np.float32)
    code = lib.Code.systematic(P, 2)
    dA, dx = device_tensor(A), device_tensor(x)
    par = lib.alloc_parity(code, q, r, torch.float32)
    draw = next(d for d in range(10000) if list(oc.draw_survivors(n, k, seed, d)[0]) == [2, 3])
    out = torch.full((q,), 9.0, dtype=torch.float32, device="cuda")
    ws = lib.matmul_workspace(code, dA, dx)
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    surv, _ = lib.coded_matmul(code, dA, par, dx, out, ws, info, seed, draw, parity_ready=False)
    torch.cuda.synchronize()
    assert list(surv) == [2, 3]
    assert int(info.item()) == 2          # pivot 2 of the 2 x 2 LU is zero
    assert bool(torch.all(out == 9.0))
    qb = code.qb(q)
    Y = ws[: 8 * n * qb].view(torch.float64).view(n, qb).cpu().numpy()
    G = oc.systematic_generator(P)
    ref = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), x[:, None])[..., 0]
    assert np.array_equal(Y, ref)


@pytest.mark.parametrize("n,k,q,r", [(4, 2, 2048, 512), (6, 4, 1001, 260), (16, 8, 2000, 2048)])
def test_one_pass_every_missing_count(lib, torch, n, k, q, r):
    """Draws chosen so that every number of missing systematic blocks occurs,
    from none (wave 0 streams beside the others and forms no decoding
    matrix) to min(k, n - k) (the most parity survivors a set can hold): the
    set bookkeeping wave 0 builds from the survivors' bit mask must give the
    separate steps' outputs in each case."""
    seed = 43
    P, A, X = make_inputs(n, k, q, r, 1, seed)
    code = lib.Code.systematic(P, 2)
    dA, dx = device_tensor(A), device_tensor(X[:, 0])
    par = lib.alloc_parity(code, q, r, torch.float32)
    ref = oc.plain_product(A, X)
    wanted = set(range(min(k, n - k) + 1))
    draws = {}
    for d in range(20000):
        m = int(np.sum(oc.draw_survivors(n, k, seed, d)[0] >= k))
        draws.setdefault(m, d)
        if wanted <= set(draws):
            break
    assert wanted <= set(draws), f"no draw with m in {sorted(wanted - set(draws))}"
    for m in sorted(wanted):
        out, surv, Y1, info = one_pass(lib, torch, code, dA, par, dx, q, seed, draws[m], parity_ready=False)
        assert info == 0 and int(np.sum(surv >= k)) == m
        p3, Y3, out3, info3 = three_steps(lib, torch, code, dA, dx, q, r, surv)
        assert info3 == 0 and torch.equal(par, p3)
        planes_np = np.abs(p3.cpu().numpy().astype(np.float64)).sum(axis=0)
        mag = oc.worker_products(np.concatenate([np.abs(oc.pad_and_split(A, k)), planes_np]), np.abs(X))[..., 0]
        assert np.all(np.abs(Y1 - Y3) <= 2 * r * 2.0 ** -52 * mag)
        assert normwise_rel_err(out, out3) <= 1e-6
        assert normwise_rel_err(out, ref) <= 1e-4
