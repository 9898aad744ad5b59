"""GPU Monte-Carlo of the runtime model against the oracle, draw by draw."""
import numpy as np
import pytest

from oracle import runtime as rt
from tests.gpu_helpers import torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


@pytest.mark.parametrize("n,k,shift,rate", [(10, 5, 1.0, 1.0), (16, 12, 1.0, 1.0), (64, 48, 1.0, 1.0),
                                            (100, 20, 1.0, 1.0), (7, 7, 2.0, 0.5), (12, 4, 0.5, 3.0),
                                            (128, 64, 1.0, 1.0), (1, 1, 1.0, 1.0)])
def test_simulated_runtimes_match_oracle_per_draw(lib, torch, n, k, shift, rate):
    draws, first, seed = 4000, 123, 9
    unc, rep, mds = rt.simulate(n, k, seed, first, draws, rate, shift)
    tu = torch.full((draws,), float("nan"), dtype=torch.float64, device="cuda")
    tr = torch.full((draws,), float("nan"), dtype=torch.float64, device="cuda") if n % k == 0 else None
    tm = torch.full((draws,), float("nan"), dtype=torch.float64, device="cuda")
    lib.coded_simulate_runtimes(n, k, seed, first, tu, tr, tm, shift=shift, rate=rate)
    torch.cuda.synchronize()
    # the order statistics are chosen on integer words: only the final log can differ, by an ulp or so
    for got, ref in ((tu, unc), (tm, mds), (tr, rep)):
        if got is None:
            continue
        g = got.cpu().numpy()
        assert np.all(np.abs(g - ref) <= 4 * np.finfo(np.float64).eps * np.abs(ref))


def test_simulated_means_match_closed_forms(lib, torch):
    """Fig. (runtime_distribution_a) setting, n = 10 and k = 5, ten million draws."""
    n, k, draws = 10, 5, 10_000_000
    out = [torch.empty(draws, dtype=torch.float64, device="cuda") for _ in range(3)]
    lib.coded_simulate_runtimes(n, k, 1, 0, *out)
    torch.cuda.synchronize()
    for t, mean in zip(out, (rt.expected_uncoded(n, 1.0), rt.expected_repetition(n, k, 1.0), rt.expected_mds(n, k, 1.0))):
        m, sd = float(t.mean().item()), float(t.std().item())
        assert abs(m - mean) <= 5 * sd / np.sqrt(draws)
    assert bool((out[2] <= out[1]).all().item())         # MDS never slower than repetition


def test_simulation_argument_errors(lib, torch):
    t = torch.empty(10, dtype=torch.float64, device="cuda")
    with pytest.raises(lib.CodedError):
        lib.coded_simulate_runtimes(10, 4, 0, 0, t_repetition=t)     # 4 does not divide 10
    with pytest.raises(lib.CodedError):
        lib.coded_simulate_runtimes(10, 11, 0, 0, t_mds=t)


def test_simulation_full_launch_sampled_draws(lib, torch):
    """The launch bench.py times: (10,5), seed 6, 2^24 draws starting at draw
    5 * 2^24.  Three windows of 2000 draws (start, middle, end) against the
    oracle draw by draw, and every draw of the launch ordered as the model
    requires (MDS <= 2-repetition, and all three at least the shift)."""
    n, k, seed, draws = 10, 5, 6, 1 << 24
    first = 5 * draws
    out = [torch.full((draws,), float("nan"), dtype=torch.float64, device="cuda") for _ in range(3)]
    lib.coded_simulate_runtimes(n, k, seed, first, *out)
    torch.cuda.synchronize()
    for off in (0, draws // 2 - 1000, draws - 2000):
        ref = rt.simulate(n, k, seed, first + off, 2000, 1.0, 1.0)
        for got, r in zip(out, ref):
            g = got[off:off + 2000].cpu().numpy()
            assert np.all(np.abs(g - r) <= 4 * np.finfo(np.float64).eps * np.abs(r)), off
    tu, tr, tm = out
    assert bool(torch.isfinite(tu).all().item() and torch.isfinite(tr).all().item() and torch.isfinite(tm).all().item())
    assert bool((tm <= tr).all().item())
    # every task time is shift plus a nonnegative exponential, scaled by the task's share
    assert bool((tu >= 1.0 / n).all().item() and (tm >= 1.0 / k).all().item())


def test_simulation_zero_draws(lib, torch):
    """No draws: nothing is enqueued and the call succeeds."""
    out = [torch.empty(0, dtype=torch.float64, device="cuda") for _ in range(3)]
    lib.coded_simulate_runtimes(10, 5, 1, 0, *out)
    torch.cuda.synchronize()
