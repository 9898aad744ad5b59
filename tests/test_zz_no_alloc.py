"""coded_matmul_noalloc (the entry point for callers that cannot allocate)
against coded_matmul with a caller workspace, through the C ABI: the same
kernels run on the library's static scratch instead of the workspace, so the
outputs, survivors and T_(k) must be identical bit for bit.  Each case makes
two calls in a row, the second on a smaller input, so the scratch holds the
first call's worker results when the second starts."""
import numpy as np
import pytest

import synth
from tests.gpu_helpers import device_tensor, make_inputs, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def _both(lib, torch, P, A, X, dtype, seed, draw, planes=2):
    """(noalloc out, survivors, T) and (workspace out, survivors, T) for one product."""
    n, k = P.shape[0] + P.shape[1], P.shape[1]
    q, r = A.shape
    code = lib.Code.systematic(P, planes)
    dA = device_tensor(A, dtype)
    dX = device_tensor(X[:, 0] if X.shape[1] == 1 else X, dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    res = []
    for noalloc in (True, False):
        par = lib.alloc_parity(code, q, r, tdt)
        out = torch.full((q, X.shape[1]) if X.shape[1] > 1 else (q,), float("nan"), dtype=torch.float32,
                         device="cuda")
        info = torch.full((1,), -5, dtype=torch.int32, device="cuda")
        if noalloc:
            surv, t = lib.coded_matmul_noalloc(code, dA, par, dX, out, info, seed, draw, parity_ready=False)
        else:
            ws = lib.matmul_workspace(code, dA, dX)
            surv, t = lib.coded_matmul(code, dA, par, dX, out, ws, info, seed, draw, parity_ready=False)
        torch.cuda.synchronize()
        assert int(info.item()) == 0
        res.append((out.cpu().numpy(), surv, t, par.cpu()))
    return res


CASES = [
    # (n, k, q, r, s, dtype): first call, then a smaller one
    ((20, 16, 6000, 2048, 4, "f32"), (20, 16, 1001, 512, 2, "f32")),      # fp64 matrix-core worker products
    ((16, 12, 20000, 1024, 1, "f32"), (16, 12, 999, 256, 1, "f32")),      # GEMV, then the one-launch path
    ((32, 24, 3000, 1024, 64, "bf16"), (32, 24, 700, 512, 64, "bf16")),   # bf16 single pass (X^T in the scratch)
    ((64, 48, 4000, 512, 8, "f32"), (6, 4, 50, 64, 3, "f32")),
]


@pytest.mark.parametrize("first,second", CASES)
def test_noalloc_matches_workspace_call_twice(lib, torch, first, second):
    for i, (n, k, q, r, s, dtype) in enumerate((first, second)):
        P, A, X = make_inputs(n, k, q, r, s, 100 + i, dtype=dtype)
        (o1, s1, t1, p1), (o2, s2, t2, p2) = _both(lib, torch, P, A, X, dtype, seed=100 + i, draw=7 + i)
        assert np.array_equal(s1, s2) and t1 == t2
        assert torch.equal(p1, p2)
        assert np.array_equal(o1, o2, equal_nan=False), (first, second, i)


def test_noalloc_rejects_problems_beyond_the_scratch(lib, torch):
    n, k, q, r, s = 32, 24, 131072, 64, 64           # Y alone: 32 * 5462 * 64 * 4 B = 44.7 MB, fits
    P = synth.parity_matrix(n, k, 1, dtype="bf16")
    code = lib.Code.systematic(P, 2)
    sizes = lib.coded_sizes(code, lib.CODED_BF16, lib.CODED_F32, q, r, s)
    assert sizes[2] <= lib.CODED_NOALLOC_SCRATCH_BYTES
    q2 = 2 * q                                      # 89 MB of worker results: refused before any work
    sizes2 = lib.coded_sizes(code, lib.CODED_BF16, lib.CODED_F32, q2, r, s)
    assert sizes2[2] > lib.CODED_NOALLOC_SCRATCH_BYTES
    A = torch.zeros((q2, r), dtype=torch.bfloat16, device="cuda")
    X = torch.zeros((r, s), dtype=torch.bfloat16, device="cuda")
    par = torch.zeros(sizes2[0] // 2, dtype=torch.bfloat16, device="cuda")
    out = torch.full((q2, s), 3.0, dtype=torch.float32, device="cuda")
    info = torch.full((1,), -5, dtype=torch.int32, device="cuda")
    with pytest.raises(lib.CodedError) as e:
        lib.coded_matmul_noalloc(code, A, par, X, out, info, 1, 0, parity_ready=False)
    assert e.value.status == lib.CODED_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert int(info.item()) == -5 and float(out[0, 0].item()) == 3.0      # nothing was enqueued
