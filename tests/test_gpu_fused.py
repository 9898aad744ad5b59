"""The bf16 encode on the matrix cores and the single-pass encode + worker
products (coded_encode_worker_mm) of the (32,24) two-plane code, against the
fp64 oracle and against the two-step calls.

Shapes cover a ragged last tile with zero-padded rows of the last block, tiles
shared between two workgroups (more tiles than compute units, several K
stages), shapes without padding, and the fallbacks (s != 64, other codes).
Integer-valued inputs make every sum exact, so those compare bit for bit."""
import numpy as np
import pytest

from oracle import coded as oc
from tests.gpu_helpers import device_tensor, make_inputs, normwise_rel_err, torch_mod

pytestmark = pytest.mark.gpu

N, K = 32, 24
# (q, r): ragged tile + padded block; 300 tiles of 2 stages; 300 tiles of 5 stages (loaded in groups of four, so
# each tile ends with three empty stages, and 12-unit runs split tiles between two workgroups); no padding; one
# row in the last tile; one row per block (one tile, one stage); a single row of A (every other block is padding)
SHAPES = [(1000, 1024), (115200, 128), (115200, 320), (1152, 192), (24 * 17, 64), (24, 64), (1, 128)]


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def to_np(t):
    torch = torch_mod()
    import synth
    if t.dtype == torch.bfloat16:
        return synth.bf16_from_bits(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


def run_both(lib, torch, P, A, X):
    q, r = A.shape
    s = X.shape[1]
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A, "bf16"), device_tensor(X, "bf16")
    par_e = lib.alloc_parity(code, q, r, torch.bfloat16)
    par_f = lib.alloc_parity(code, q, r, torch.bfloat16)
    par_e.fill_(3)
    par_f.fill_(5)
    lib.coded_encode(code, dA, par_e)
    Y = lib.alloc_y(code, q, s, torch.float32)
    Y.fill_(float("nan"))
    lib.coded_encode_worker_mm(code, dA, par_f, dX, Y)
    Y2 = lib.alloc_y(code, q, s, torch.float32)
    lib.coded_worker_mm(code, dA, par_e, dX, Y2)
    torch.cuda.synchronize()
    return code, to_np(par_e).astype(np.float64), to_np(par_f).astype(np.float64), \
        Y.cpu().numpy().astype(np.float64), Y2.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("q,r", SHAPES)
def test_single_pass_gaussian(lib, torch, q, r):
    P, A, X = make_inputs(N, K, q, r, 64, 31, "bf16")
    code, pe, pf, Y, Y2 = run_both(lib, torch, P, A, X)
    # the same planes from both entry points
    assert np.array_equal(pe, pf)
    # parity against the exact sums: fp32 rounding of the sum and the bf16 lo plane
    blocks = oc.pad_and_split(A, K)
    G = oc.systematic_generator(P)
    ref = oc.encode(G, blocks)[K:]
    scale = np.abs(oc.encode(oc.systematic_generator(np.abs(P)), np.abs(blocks))[K:])
    assert np.all(np.abs(pf[0] + pf[1] - ref) <= K * 2.0 ** -23 * scale + 2.0 ** -16 * np.abs(ref))
    # products of the stored blocks (systematic: A itself; parity: hi + lo planes) in fp64
    coded = np.concatenate([blocks, pf[0] + pf[1]])
    Yref = oc.worker_products(coded, X)
    assert np.all(np.isfinite(Y))
    # products of bf16 values are exact in fp32; summing r of them (hi and lo planes: 2r) in fp32 errs by at
    # most 2r * 2^-24 of the sum of their magnitudes, elementwise
    mag = oc.worker_products(np.abs(np.concatenate([blocks, pf[0], pf[1]])), np.abs(X))
    mag = np.concatenate([mag[:K], mag[K:K + N - K] + mag[N:]])
    assert np.all(np.abs(Y - Yref) <= 2 * r * 2.0 ** -24 * mag)
    # and the two-step products, summed in another order
    assert np.all(np.abs(Y - Y2) <= 4 * r * 2.0 ** -24 * mag)


@pytest.mark.parametrize("q,r", [(1000, 1024), (115200, 128), (115200, 320), (24 * 17, 64), (1, 64)])
def test_single_pass_integer_bit_exact(lib, torch, q, r):
    P, A, X = make_inputs(N, K, q, r, 64, 32, "bf16", integer=True)
    code, pe, pf, Y, Y2 = run_both(lib, torch, P, A, X)
    blocks = oc.pad_and_split(A, K)
    G = oc.systematic_generator(P)
    ref = oc.encode(G, blocks)
    assert np.array_equal(pf[0], ref[K:]) and np.all(pf[1] == 0)
    assert np.array_equal(pe, pf)
    Yref = oc.worker_products(ref, X)
    assert np.array_equal(Y, Yref)
    assert np.array_equal(Y2, Yref)


@pytest.mark.parametrize("n,k,s", [(32, 24, 32), (16, 12, 64), (32, 24, 65)])
def test_fallback_shapes_match_two_steps(lib, torch, n, k, s):
    """Shapes the single pass does not serve run the encode and the products
    one after the other: results equal the two separate calls bit for bit."""
    q, r = 700, 256
    P, A, X = make_inputs(n, k, q, r, s, 33, "bf16")
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A, "bf16"), device_tensor(X, "bf16")
    par_a = lib.alloc_parity(code, q, r, torch.bfloat16)
    par_b = lib.alloc_parity(code, q, r, torch.bfloat16)
    Ya = lib.alloc_y(code, q, s, torch.float32)
    Yb = lib.alloc_y(code, q, s, torch.float32)
    lib.coded_encode_worker_mm(code, dA, par_a, dX, Ya)
    lib.coded_encode(code, dA, par_b)
    lib.coded_worker_mm(code, dA, par_b, dX, Yb)
    torch.cuda.synchronize()
    assert torch.equal(par_a.view(torch.int16), par_b.view(torch.int16))
    assert torch.equal(Ya, Yb)


def test_single_pass_f32_inputs_two_steps(lib, torch):
    """fp32 inputs: coded_encode_worker_mm equals coded_encode + coded_worker_mm."""
    n, k, q, r = 16, 12, 600, 256
    P, A, X = make_inputs(n, k, q, r, 1, 34)
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A), device_tensor(X[:, 0])
    par_a = lib.alloc_parity(code, q, r, torch.float32)
    par_b = lib.alloc_parity(code, q, r, torch.float32)
    Ya = lib.alloc_y(code, q, 1, torch.float64)
    Yb = lib.alloc_y(code, q, 1, torch.float64)
    lib.coded_encode_worker_mm(code, dA, par_a, dX, Ya)
    lib.coded_encode(code, dA, par_b)
    lib.coded_worker_mm(code, dA, par_b, dX, Yb)
    torch.cuda.synchronize()
    assert torch.equal(par_a, par_b) and torch.equal(Ya, Yb)


def test_matmul_single_pass_end_to_end(lib, torch):
    """coded_matmul with parity_ready = 0 takes the single pass: decoded A X within
    the bf16 tolerance, and its stored parity equals coded_encode's."""
    from tests.test_gpu_parity import TOL_BF16, run_matmul
    q, r, s = 115200, 128, 64
    P, A, X = make_inputs(N, K, q, r, s, 35, "bf16")
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A, "bf16"), device_tensor(X, "bf16")
    par = lib.alloc_parity(code, q, r, torch.bfloat16)
    ref = oc.plain_product(A, X)
    for draw in range(3):
        out, surv, _ = run_matmul(lib, torch, code, dA, par, dX, q, s, 35, draw, parity_ready=False)
        assert np.array_equal(surv, oc.draw_survivors(N, K, 35, draw)[0])
        assert normwise_rel_err(out, ref) <= TOL_BF16
    par_e = lib.alloc_parity(code, q, r, torch.bfloat16)
    lib.coded_encode(code, dA, par_e)
    torch.cuda.synchronize()
    assert torch.equal(par.view(torch.int16), par_e.view(torch.int16))


def test_single_pass_argument_errors(lib, torch):
    """Bad arguments are refused on the host before anything is enqueued."""
    import ctypes
    q, r, s = 100, 64, 64
    P, A, X = make_inputs(N, K, q, r, s, 36, "bf16")
    code = lib.Code.systematic(P, 2)
    dA, dX = device_tensor(A, "bf16"), device_tensor(X, "bf16")
    par = lib.alloc_parity(code, q, r, torch.bfloat16)
    Y = lib.alloc_y(code, q, s, torch.float32)
    h, vp = lib.lib(), ctypes.c_void_p
    st = vp(torch.cuda.current_stream().cuda_stream)
    ws = lib.worker_workspace(code, dA, dX)
    args = [code.handle, lib.CODED_BF16, vp(dA.data_ptr()), q, r, r, vp(par.data_ptr()), vp(dX.data_ptr()), s, s,
            vp(Y.data_ptr()), lib.CODED_F32, vp(ws.data_ptr()), st]
    assert h.coded_encode_worker_mm(*args) == lib.CODED_OK
    bad = list(args)
    bad[12] = None                                  # bf16 needs the workspace
    assert h.coded_encode_worker_mm(*bad) == lib.CODED_ERR_ARG
    bad = list(args)
    bad[11] = lib.CODED_F64                         # bf16 products are fp32
    assert h.coded_encode_worker_mm(*bad) == lib.CODED_ERR_ARG
    bad = list(args)
    bad[9] = s - 1                                  # ldx < s
    assert h.coded_encode_worker_mm(*bad) == lib.CODED_ERR_SHAPE
    bad = list(args)
    bad[5] = r - 1                                  # lda < r
    assert h.coded_encode_worker_mm(*bad) == lib.CODED_ERR_SHAPE
    torch.cuda.synchronize()


def test_single_pass_strided_a(lib, torch):
    """A with a row stride above r (a column window of a wider matrix): the
    single pass reads it through lda, equal to the contiguous copy's results."""
    q, r, s, pad = 2000, 256, 64, 64
    P, A, X = make_inputs(N, K, q, r, s, 37, "bf16", integer=True)
    code = lib.Code.systematic(P, 2)
    wide = np.zeros((q, r + pad), dtype=np.float32)
    wide[:, :r] = A
    dW = device_tensor(wide, "bf16")
    dA_view = dW[:, :r]                        # lda = r + pad
    dA, dX = device_tensor(A, "bf16"), device_tensor(X, "bf16")
    par_v = lib.alloc_parity(code, q, r, torch.bfloat16)
    par_c = lib.alloc_parity(code, q, r, torch.bfloat16)
    Yv = lib.alloc_y(code, q, s, torch.float32)
    Yc = lib.alloc_y(code, q, s, torch.float32)
    lib.coded_encode_worker_mm(code, dA_view, par_v, dX, Yv)
    lib.coded_encode_worker_mm(code, dA, par_c, dX, Yc)
    torch.cuda.synchronize()
    assert torch.equal(par_v.view(torch.int16), par_c.view(torch.int16))
    assert torch.equal(Yv, Yc)
    ref = oc.encode(oc.systematic_generator(P), oc.pad_and_split(A, K))
    assert np.array_equal(Yv.cpu().numpy().astype(np.float64), oc.worker_products(ref, X))
