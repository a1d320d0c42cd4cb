"""Pins of the oracle's double-exponential value fit (Section 5,
"Nonlinear regression": y = a e^(bx) + c e^(dx))."""
import numpy as np
import pytest

import oracle


def _t(n):
    return np.array([(2 * j - (n - 1)) / (n - 1) for j in range(n)])


@pytest.mark.parametrize("theta", [(2.0, 1.5, 0.5, -3.0), (-1.0, 0.3, 4.0, -0.7), (5e-3, 2.0, 1e-3, -4.0)])
def test_recovers_an_exact_double_exponential(theta):
    a, b, c, d = theta
    t = _t(300)
    y = a * np.exp(b * t) + c * np.exp(d * t)
    th, rss = oracle.dexp_fit(t, y)
    model = th[0] * np.exp(th[1] * t) + th[2] * np.exp(th[3] * t)
    assert rss <= 1e-20 * max(1.0, float(np.sum(y * y)))
    np.testing.assert_allclose(model, y, rtol=1e-9, atol=1e-12 * np.abs(y).max())
    # the pair of exponentials is identified up to their order
    got = sorted([(th[1], th[0]), (th[3], th[2])])
    want = sorted([(b, a), (d, c)])
    np.testing.assert_allclose(np.array(got), np.array(want), rtol=1e-6)


def test_at_least_as_good_as_scipy_least_squares():
    from scipy.optimize import least_squares

    rng = np.random.default_rng(5)
    for trial in range(6):
        n = 400
        t = _t(n)
        y = np.sort(rng.laplace(0, 1e-3, n))[::-1] * (1 + trial)
        th, rss = oracle.dexp_fit(t, y)

        def resid(p):
            return y - (p[0] * np.exp(p[1] * t) + p[2] * np.exp(p[3] * t))

        best = np.inf
        for x0 in ([y.mean(), 1.0, 0.0, -1.0], [y[0], -1.0, y[-1], 1.0], [1e-3, 3.0, -1e-3, -3.0]):
            r = least_squares(resid, x0, method="lm", max_nfev=20000, xtol=1e-15, ftol=1e-15, gtol=1e-15)
            best = min(best, float(np.sum(r.fun**2)))
        assert rss <= best * (1 + 1e-3) + 1e-30, (trial, rss, best)


def test_single_exponential_data_is_fitted_exactly():
    t = _t(100)
    y = 3.0 * np.exp(-2.0 * t)
    th, rss = oracle.dexp_fit(t, y)
    model = th[0] * np.exp(th[1] * t) + th[2] * np.exp(th[3] * t)
    np.testing.assert_allclose(model, y, rtol=1e-7)


def test_decoder_evaluates_the_row():
    # one run of 5 values with a hand-made row: the decoder's value at rank
    # j is a e^(b t_j) + c e^(d t_j) with t_j = (2j - 4) / 4
    row = np.array([1.5, 0.5, -0.25, -2.0], dtype=np.float32)
    n = 5
    ranks = np.arange(n)
    b = oracle.sigma_bits(n)
    bits = np.zeros(32 * oracle.sigma_words(n), np.uint8)
    for q, rk in enumerate(ranks):
        for k in range(b):
            bits[q * b + k] = (rk >> k) & 1
    sigma = np.packbits(bits, bitorder="little").view("<u4")
    y = oracle.curvefit_decode_seg(row, sigma, n, 3, np.array([0, n], np.uint64), oracle.FIT_DEXP)
    t = (2 * ranks - 4) / 4.0
    want = (1.5 * np.exp(0.5 * t) - 0.25 * np.exp(-2.0 * t)).astype(np.float32)
    np.testing.assert_array_equal(y, want)


def test_round_trip_with_the_double_exponential():
    from paper_2102_03112_amd import workloads as W

    g = W.generate(W.Workload("t", 50_000, 1, (1, 100), 1e-3, 3, 4, "laplace_5e-4", 3))
    res = oracle.roundtrip_tensor(g, 500, 1e-3, 5, 4, model=oracle.FIT_DEXP)
    assert res.fit.model == oracle.FIT_DEXP and res.fit.D_eff == 3
    V = g[res.P.astype(np.int64)]
    err = np.linalg.norm(res.vals - V) / np.linalg.norm(V)
    poly = oracle.roundtrip_tensor(g, 500, 1e-3, 3, 4)
    err_p = np.linalg.norm(poly.vals - V) / np.linalg.norm(V)
    assert err < 0.2 and err < 2 * err_p + 1e-3
    # fewer than four values: the polynomial through them
    small = oracle.roundtrip_tensor(g[:300], 2, 1e-3, 5, 4, policy=oracle.POLICY_LEFTMOST, model=oracle.FIT_DEXP)
    assert small.fit.n < 4 and small.fit.model == oracle.FIT_POLY
