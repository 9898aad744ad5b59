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
