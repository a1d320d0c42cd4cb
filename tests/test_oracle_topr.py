"""Pins for the oracle's sparsifiers (Section 2 "Sparsification", Section 10.2).

Top-r is "the indices of the r highest-magnitude elements"; ties are broken
by smaller index.  The pins are brute force on tiny inputs full of ties and
signed zeros, and an independent numpy implementation at larger size.
"""
import numpy as np
import pytest

import oracle
from paper_2102_03112_amd import workloads


def _topr_reference(g, r):
    # sort by |g| descending, then index ascending; float64 magnitudes, so no
    # bit tricks are shared with the oracle
    idx = np.arange(g.size)
    order = np.lexsort((idx, -np.abs(g.astype(np.float64))))
    return np.sort(order[:r]).astype(np.uint32)


@pytest.mark.parametrize("d", [1, 2, 3, 7, 31, 32, 33, 64])
def test_topr_brute_force_with_ties(d):
    for seed in range(6):
        g = workloads.tied_values(d, seed)
        for r in range(0, d + 1):
            np.testing.assert_array_equal(oracle.topr(g, r), _topr_reference(g, r))


def test_topr_matches_numpy_at_scale():
    g = workloads.generate(workloads.WORKLOADS["normal_1m"])
    r = oracle.ratio_count(g.size, 1, 100)
    assert r == 10_486
    S = oracle.topr(g, r)
    ref = np.sort(np.argsort(-np.abs(g.astype(np.float64)), kind="stable")[:r]).astype(np.uint32)
    np.testing.assert_array_equal(S, ref)


def test_topr_invariants_on_coarse_values():
    # many equal magnitudes around the threshold
    rng = np.random.default_rng(7)
    g = (rng.integers(-20, 21, 100_000) * 0.25).astype(np.float32)
    for r in (1, 999, 12_345, 99_999):
        S = oracle.topr(g, r)
        assert S.size == r and np.all(np.diff(S.astype(np.int64)) > 0)
        a = np.abs(g)
        inS = np.zeros(g.size, bool)
        inS[S] = True
        thr = a[S].min()
        assert a[~inS].max(initial=0) <= thr
        # co-threshold elements outside S all come after those inside S
        tie_in = np.flatnonzero(inS & (a == thr))
        tie_out = np.flatnonzero(~inS & (a == thr))
        if tie_out.size:
            assert tie_out.min() > tie_in.max()


def test_ratio_count_rounds_up():
    assert oracle.ratio_count(1_048_576, 1, 100) == 10_486
    assert oracle.ratio_count(25_557_032, 1, 100) == 255_571
    assert oracle.ratio_count(138_357_544, 1, 1000) == 138_358
    assert oracle.ratio_count(14_784_299, 1, 100) == 147_843
    assert oracle.ratio_count(14_784_298, 1, 100) == 147_843
    assert oracle.ratio_count(0, 1, 100) == 0


def test_nonzero_support():
    g = workloads.sparse_normal(100_003, seed=3, zero_frac=0.4)
    g[5] = -0.0
    S = oracle.nonzero(g)
    np.testing.assert_array_equal(S, np.flatnonzero(g != 0).astype(np.uint32))
    assert 5 not in set(S.tolist())


def test_nonfinite_rejected():
    g = workloads.normal(100, seed=1)
    for bad in (np.nan, np.inf, -np.inf):
        h = g.copy()
        h[17] = bad
        with pytest.raises(oracle.OracleError):
            oracle.topr(h, 10)
        with pytest.raises(oracle.OracleError):
            oracle.nonzero(h)
