"""Pins of the oracle's index policies (Section 4; Sections 10.4, 10.5).

P0 keeps all of P; P1 keeps r positives chosen at random; the deterministic
policies keep the leftmost, middle or rightmost r of P.  P1's choice comes
from a keyed permutation of the ranks, which must be a bijection (checked by
brute force) and must make every positive equally likely to be kept
(checked statistically over many keys).
"""
import math

import numpy as np
import pytest

import oracle
from paper_2102_03112_amd import workloads as W


@pytest.mark.parametrize("N", [1, 2, 3, 4, 5, 7, 16, 17, 100, 255, 256, 257, 1000, 4097])
@pytest.mark.parametrize("seed", [0, 1, 0xDEADBEEF])
def test_perm_is_a_bijection(N, seed):
    img = [oracle.perm(q, N, seed) for q in range(N)]
    assert sorted(img) == list(range(N))


def test_perm_depends_on_the_key_and_is_not_the_identity():
    N = 1000
    a = np.array([oracle.perm(q, N, 1) for q in range(N)])
    b = np.array([oracle.perm(q, N, 2) for q in range(N)])
    assert np.mean(a == np.arange(N)) < 0.02
    assert np.mean(a == b) < 0.02


def test_perm_walks_back_into_a_domain_far_below_the_word_size():
    # N = 2^(2h-2) + 1 is the worst case for cycle walking (4x oversize)
    for N in [5, 17, 65, 257, 1025]:
        assert sorted(oracle.perm(q, N, 7) for q in range(N)) == list(range(N))


@pytest.mark.parametrize("npos,r", [(0, 0), (1, 1), (10, 3), (10, 10), (11, 4), (12, 5), (100, 37)])
def test_deterministic_policies_take_the_stated_runs(npos, r):
    left, nl = oracle.policy_slots(npos, r, oracle.POLICY_LEFTMOST, 0)
    mid, nm = oracle.policy_slots(npos, r, oracle.POLICY_MIDDLE, 0)
    right, nr = oracle.policy_slots(npos, r, oracle.POLICY_RIGHTMOST, 0)
    keep = min(r, npos)
    assert nl == nm == nr == keep
    q = np.arange(npos)
    exp_left = np.where(q < keep, q, oracle.NO_SLOT)
    s0 = (npos - keep) // 2
    exp_mid = np.where((q >= s0) & (q < s0 + keep), q - s0, oracle.NO_SLOT)
    exp_right = np.where(q >= npos - keep, q - (npos - keep), oracle.NO_SLOT)
    np.testing.assert_array_equal(left, exp_left)
    np.testing.assert_array_equal(mid, exp_mid)
    np.testing.assert_array_equal(right, exp_right)


def test_p0_keeps_everything_in_rank_order():
    slots, nc = oracle.policy_slots(50, 7, oracle.POLICY_P0, 3)
    assert nc == 50
    np.testing.assert_array_equal(slots, np.arange(50))


@pytest.mark.parametrize("npos,r", [(1, 1), (9, 4), (100, 10), (1000, 999)])
def test_random_policy_keeps_exactly_r_with_distinct_value_numbers(npos, r):
    slots, nc = oracle.policy_slots(npos, r, oracle.POLICY_RANDOM, 12345)
    assert nc == r
    kept = slots[slots != oracle.NO_SLOT]
    assert kept.size == r
    np.testing.assert_array_equal(np.sort(kept), np.arange(r))


def test_random_policy_is_uniform_over_positives():
    # each of 40 positives is kept with probability r/npos = 1/4; over 4000
    # keys the counts are binomial(4000, 1/4): mean 1000, sd ~27.4
    npos, r, trials = 40, 10, 4000
    counts = np.zeros(npos)
    for seed in range(trials):
        slots, _ = oracle.policy_slots(npos, r, oracle.POLICY_RANDOM, seed)
        counts += slots != oracle.NO_SLOT
    sd = math.sqrt(trials * 0.25 * 0.75)
    assert np.all(np.abs(counts - trials / 4) < 5 * sd), counts
    # and the chi-square of the 40 counts is in range (39 dof: 5th..99.9th pct)
    chi2 = np.sum((counts - trials / 4) ** 2 / (trials / 4 * 0.75))
    assert 24 < chi2 < 73, chi2


def test_random_policy_pairs_are_not_correlated():
    # P(both q0 and q1 kept) = r(r-1)/(n(n-1)) for a uniform r-subset
    npos, r, trials = 12, 4, 6000
    both = 0
    for seed in range(trials):
        slots, _ = oracle.policy_slots(npos, r, oracle.POLICY_RANDOM, seed)
        both += (slots[3] != oracle.NO_SLOT) and (slots[8] != oracle.NO_SLOT)
    p = r * (r - 1) / (npos * (npos - 1))
    sd = math.sqrt(trials * p * (1 - p))
    assert abs(both - trials * p) < 5 * sd


def test_policy_rejects_unknown_ids():
    with pytest.raises(oracle.OracleError):
        oracle.policy_slots(10, 3, 5, 0)


@pytest.mark.parametrize("policy", [oracle.POLICY_RANDOM, oracle.POLICY_LEFTMOST, oracle.POLICY_MIDDLE,
                                    oracle.POLICY_RIGHTMOST])
def test_round_trip_sends_r_values_and_reconstructs_them_when_interpolating(policy):
    # top-r with r = S * (D + 1) values: every run is interpolated, so the
    # receiver gets g back exactly at the kept positives and 0 elsewhere
    g = W.normal(5000, 99, scale=1e-3)
    r = 8 * 4
    res = oracle.roundtrip_tensor(g, r, 1e-2, 3, 8, policy=policy, seed=77)
    assert res.P.size >= r
    assert res.fit.n == r
    kept = res.slots != oracle.NO_SLOT
    assert kept.sum() == r
    np.testing.assert_array_equal(res.P_dec, res.P)
    pos = res.P[kept].astype(np.int64)
    np.testing.assert_allclose(res.dense[pos], g[pos], rtol=1e-6, atol=0)
    off = np.ones(g.size, bool)
    off[pos] = False
    assert np.all(res.dense[off] == 0)
    if policy == oracle.POLICY_LEFTMOST:
        np.testing.assert_array_equal(pos, res.P[:r])


def test_p0_round_trip_is_unchanged_by_the_policy_plumbing():
    g = W.normal(3000, 5, scale=1e-3)
    a = oracle.roundtrip_tensor(g, 30, 1e-3, 5, 2)
    b = oracle.roundtrip_tensor(g, 30, 1e-3, 5, 2, policy=oracle.POLICY_P0, seed=999)
    np.testing.assert_array_equal(a.dense, b.dense)
    np.testing.assert_array_equal(a.fit.sigma, b.fit.sigma)
    assert a.fit.n == a.P.size
