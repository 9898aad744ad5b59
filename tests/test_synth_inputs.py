"""The seeded input generators: shapes, ranges and determinism of the draws
that feed both the oracle and the device path."""
import numpy as np
import pytest

import synth


@pytest.mark.parametrize("m", [0, 1, 8, 12, 16])
def test_exact_parity_sets(m):
    n, k, B = 64, 48, 300
    S = synth.exact_parity_sets(n, k, m, B, seed=7)
    assert S.shape == (B, k) and S.dtype == np.int32
    assert np.all((S >= 0) & (S < n))
    assert np.all(np.sort(S, axis=1)[:, 1:] != np.sort(S, axis=1)[:, :-1])   # no repeats within a set
    assert np.all((S >= k).sum(axis=1) == m)
    assert np.array_equal(S, synth.exact_parity_sets(n, k, m, B, seed=7))
    if 0 < m < n - k:
        # every parity worker is used somewhere, and rows are not sorted
        assert set(np.unique(S[S >= k])) == set(range(k, n))
        assert not np.all(np.diff(S, axis=1) > 0)


def test_exact_parity_sets_rejects_impossible_counts():
    with pytest.raises(ValueError):
        synth.exact_parity_sets(64, 48, 17, 1, seed=1)
    with pytest.raises(ValueError):
        synth.exact_parity_sets(5, 3, -1, 1, seed=1)
