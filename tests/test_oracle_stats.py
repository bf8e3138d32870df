"""Pins of the oracle's hazard counts (eq. (hazard)) and Kendall tau-b pair
counts (ranking fidelity, Sec. VI-F) against identities and scipy."""
import numpy as np
import pytest
from scipy import stats

import oracle


def test_hazard_identities():
    rng = np.random.default_rng(1)
    for T in (rng.integers(1, 80, 500), rng.geometric(1 / 23.7, 2000), np.full(16, 12),
              np.array([1]), np.array([51, 52, 200])):
        T = T.astype(np.uint32)
        d, n = oracle.hazard_counts(T)
        assert n[0] == len(T)                                   # everyone reaches turn 0
        # sessions live at t but not at t+1 are exactly those ending at t
        assert np.all(n[:-1].astype(int) - n[1:].astype(int) == d[:-1].astype(int))
        assert int(d.sum()) == int((T <= 51).sum())
        # product-limit survival equals the empirical survival without censoring
        h = np.where(n > 0, d / np.maximum(n, 1), 0.0)
        surv = np.cumprod(1 - h)
        emp = np.array([(T > t + 1).mean() for t in range(51)])
        assert np.allclose(surv, emp)


def test_hazard_fixed_turns():
    d, n = oracle.hazard_counts(np.full(16, 12, np.uint32))
    hf = oracle.lut_f32(d, n)
    assert hf[11] == 1.0 and np.all(hf[:11] == 0) and np.all(hf[12:] == 0)


def test_hazard_geometric_is_flat():
    rng = np.random.default_rng(2)
    d, n = oracle.hazard_counts(rng.geometric(0.1, 200_000).astype(np.uint32))
    hf = oracle.lut_f32(d, n)
    assert np.all(np.abs(hf[:20] - 0.1) < 0.01)


def _scipy_tau(x, y):
    return stats.kendalltau(x, y, variant="b").statistic


@pytest.mark.parametrize("n", [2, 3, 7, 40, 300])
def test_kendall_matches_scipy(n):
    rng = np.random.default_rng(n)
    for trial in range(5):
        x = rng.integers(0, max(2, n // 3), n).astype(np.float32)   # forced ties
        y = rng.integers(0, max(2, n // 4), n).astype(np.uint64)
        if trial == 0:
            x[:] = 1.0                                               # all tied in x
        if trial == 1:
            x[rng.random(n) < 0.1] = np.inf
        counts, _ = oracle.kendall(x[None], y[None])
        assert int(counts.sum()) == n * (n - 1) // 2
        tau = oracle.tau_b(counts)[0]
        ref = _scipy_tau(x.astype(np.float64), y.astype(np.float64))
        if np.isnan(ref):
            assert np.isnan(tau)
        else:
            assert abs(tau - ref) < 1e-12


def test_kendall_extremes_and_gather():
    x = np.arange(10, dtype=np.float32)
    y = np.arange(10, dtype=np.uint64)
    c, top = oracle.kendall(x[None], y[None])
    assert c[0].tolist() == [45, 0, 0, 0, 0] and top[0] == 1
    c, top = oracle.kendall(x[None], y[::-1].copy()[None])
    assert c[0].tolist() == [0, 45, 0, 0, 0] and top[0] == 0
    idx = np.array([[9, 0, 5], [1, 2, 3]], np.uint32)
    c, top = oracle.kendall(x, y, idx=idx)
    assert c[:, 0].tolist() == [3, 3] and top.tolist() == [1, 1]


def test_kendall_top1_tie_goes_to_first():
    x = np.array([[1, 5, 5, 0]], np.float32)
    y = np.array([[0, 9, 9, 1]], np.uint64)
    assert oracle.kendall(x, y)[1][0] == 1
    y = np.array([[0, 8, 9, 1]], np.uint64)          # x picks position 1, y position 2
    assert oracle.kendall(x, y)[1][0] == 0
