"""Real, timed straggling (coded_straggler_matmul): worker products started
on the device at their drawn runtimes, the decode taken from the first k
completions.  The decoded product is checked against the fp64 oracle (any k
results decode exactly, Sec. III-A), the survivors against the draw of the
runtime model wherever the start times are far apart, and the timeline
against the protocol (no worker starts early, the survivors are the first k
completions, survivors-only mode never starts the late workers).
"""
import numpy as np
import pytest

from oracle import coded as oc
from tests.gpu_helpers import device_tensor, make_inputs, normwise_rel_err, torch_mod

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4
TOL_BF16 = 2e-2
JITTER_US = 1000.0      # host polling, launch and kernel time: start gaps above this keep their order


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def setup(lib, torch, n, k, q, r, s, seed, dtype="f32"):
    P, A, X = make_inputs(n, k, q, r, s, seed, dtype)
    code = lib.Code.systematic(P, 2)
    dA = device_tensor(A, dtype)
    dX = device_tensor(X[:, 0] if s == 1 else X, dtype)
    pdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    par = lib.alloc_parity(code, q, r, pdt)
    lib.coded_encode(code, dA, par)
    ydt = torch.float32 if dtype == "bf16" else torch.float64
    Y = lib.alloc_y(code, q, s, ydt)
    ref = oc.plain_product(A, X)
    return code, P, A, X, dA, dX, par, Y, ref


def check_timeline(n, k, surv, tl, latency, launch_all):
    sched, launched, seen = tl[:, 0], tl[:, 1], tl[:, 2]
    ran = launched >= 0
    assert np.all(seen[seen >= 0] >= launched[seen >= 0])
    assert len(set(surv.tolist())) == k and np.all((surv >= 0) & (surv < n))
    assert np.all(seen[surv] >= 0)                                    # every survivor was seen complete
    kth = np.max(seen[surv])
    # before the k-th arrival nobody starts early (launch_all starts the rest after it)
    before = ran & (launched <= kth)
    assert np.all(launched[before] >= sched[before] - 1.0)
    # survivors in arrival order: their completion times do not decrease
    assert np.all(np.diff(seen[surv]) >= 0)
    # a worker left out was not seen complete before the k-th survivor
    others = np.setdiff1d(np.arange(n), surv)
    assert np.all((seen[others] < 0) | (seen[others] >= kth))
    if not launch_all:
        # survivors only: a worker whose start lies after the k-th arrival never ran
        late = sched > kth + 1.0
        assert not np.any(ran & late)
    else:
        assert np.all(ran)
    assert latency >= kth


@pytest.mark.parametrize("launch_all", [False, True])
def test_straggler_product_matches_oracle(lib, torch, launch_all):
    n, k, q, r, s = 4, 2, 2048, 512, 1
    code, P, A, X, dA, dX, par, Y, ref = setup(lib, torch, n, k, q, r, s, 31)
    out = torch.full((q,), float("nan"), dtype=torch.float32, device="cuda")
    info = torch.full((1,), 9, dtype=torch.int32, device="cuda")
    for draw in range(6):
        out.fill_(float("nan"))
        surv, tl, lat = lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 31, draw, 2000.0,
                                                   launch_all=launch_all)
        torch.cuda.synchronize()
        assert int(info.item()) == 0
        assert normwise_rel_err(out.cpu().numpy(), ref[:, 0]) <= TOL_F32, draw
        check_timeline(n, k, surv, tl, lat, launch_all)
        # the drawn start times are the runtime model's task times
        T = oc.worker_runtimes(n, k, 31, draw)
        assert np.allclose(tl[:, 0], T * 2000.0, rtol=1e-12)


def test_straggler_survivors_follow_the_draw(lib, torch):
    """With a long time unit the first k arrivals are the k smallest runtimes,
    except where two start times lie within the timing jitter."""
    n, k, q, r, s = 8, 5, 4096, 256, 1
    code, P, A, X, dA, dX, par, Y, ref = setup(lib, torch, n, k, q, r, s, 32)
    out = torch.empty((q,), dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    unit = 30000.0
    agree = 0
    for draw in range(8):
        surv, tl, lat = lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 32, draw, unit)
        torch.cuda.synchronize()
        assert int(info.item()) == 0
        assert normwise_rel_err(out.cpu().numpy(), ref[:, 0]) <= TOL_F32
        want, _ = oc.draw_survivors(n, k, 32, draw)
        T = np.sort(oc.worker_runtimes(n, k, 32, draw)) * unit
        separated = T[k] - T[k - 1] > JITTER_US
        if separated:
            assert sorted(surv.tolist()) == sorted(want.tolist()), draw
        agree += sorted(surv.tolist()) == sorted(want.tolist())
    assert agree >= 6


def test_straggler_survivors_only_leaves_late_workers_untouched(lib, torch):
    n, k, q, r, s = 16, 12, 6000, 384, 1
    code, P, A, X, dA, dX, par, Y, ref = setup(lib, torch, n, k, q, r, s, 33)
    out = torch.empty((q,), dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    for draw in range(4):
        Y.fill_(float("nan"))
        surv, tl, lat = lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 33, draw, 5000.0)
        torch.cuda.synchronize()
        assert int(info.item()) == 0
        assert normwise_rel_err(out.cpu().numpy(), ref[:, 0]) <= TOL_F32
        ran = tl[:, 1] >= 0
        Yh = Y.cpu().numpy()
        for i in range(n):
            assert np.all(np.isnan(Yh[i])) != bool(ran[i]), (draw, i)
        check_timeline(n, k, surv, tl, lat, False)


def test_straggler_launch_all_computes_every_product(lib, torch):
    n, k, q, r, s = 6, 4, 1000, 256, 1
    code, P, A, X, dA, dX, par, Y, ref = setup(lib, torch, n, k, q, r, s, 34)
    out = torch.empty((q,), dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    Y.fill_(float("nan"))
    lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 34, 0, 3000.0, launch_all=True)
    torch.cuda.synchronize()          # the caller's stream waits for the stragglers
    G = oc.systematic_generator(P)
    want = oc.worker_products(oc.encode(G, oc.pad_and_split(A, k)), X)
    got = Y.cpu().numpy()
    assert np.all(np.isfinite(got))
    assert np.max(np.abs(got - want)) <= 1e-9 * np.max(np.abs(want))


def test_straggler_bf16_dense(lib, torch):
    n, k, q, r, s = 8, 6, 600, 256, 64
    code, P, A, X, dA, dX, par, Y, ref = setup(lib, torch, n, k, q, r, s, 35, "bf16")
    out = torch.empty((q, s), dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    for draw in range(3):
        surv, tl, lat = lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 35, draw, 2000.0,
                                                   launch_all=bool(draw % 2))
        torch.cuda.synchronize()
        assert int(info.item()) == 0
        assert normwise_rel_err(out.cpu().numpy(), ref) <= TOL_BF16
        check_timeline(n, k, surv, tl, lat, bool(draw % 2))


def test_straggler_argument_errors(lib, torch):
    n, k, q, r, s = 4, 2, 64, 32, 1
    code, P, A, X, dA, dX, par, Y, ref = setup(lib, torch, n, k, q, r, s, 36)
    out = torch.empty((q,), dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(lib.CodedError) as e:
        lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 36, 0, -1.0)
    assert e.value.status == lib.CODED_ERR_ARG
    with pytest.raises(lib.CodedError) as e:
        lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 36, 0, 1e9)   # k-th start far past 60 s
    assert e.value.status == lib.CODED_ERR_ARG
    with pytest.raises(lib.CodedError):
        lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 36, 0, 100.0, rate=0.0)
    # a zero time unit starts every worker at once; the product is still exact
    surv, tl, lat = lib.coded_straggler_matmul(code, dA, par, dX, Y, out, info, 36, 1, 0.0)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    assert normwise_rel_err(out.cpu().numpy(), ref[:, 0]) <= TOL_F32
