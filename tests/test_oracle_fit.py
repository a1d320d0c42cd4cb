"""Pins for the oracle's value compressor (Section 5) and reorder map (5.1).

Anchors: the worked example of Figure 1 (Section 1), exact reproduction of
polynomial data, agreement with numpy.polyfit (an independent least-squares
routine, the one the paper's CPU path uses), the orthogonality of the
least-squares residual, an independent stable sort, an independent bit
packer, and the interpolation special case.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2102_03112_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fig1():
    return json.load(open(os.path.join(GOLDEN, "fig1_worked_example.json")))


def test_figure1_line_fit_every_mask():
    """The 4 nonzeros of the 8-element tensor lie on V(i) = 0.6 i + 4.0.
    Reading i as the ordinal of the nonzero (1..4): fitting a line recovers
    a and b, the mask plus a and b rebuild the tensor, and the bit counts are
    the figure's."""
    ex = _fig1()
    d, nnz, a, b = ex["d"], ex["nnz"], ex["a"], ex["b"]
    i = np.arange(1, nnz + 1, dtype=np.float64)
    y = a * i + b
    c = oracle.lsq_fit(i, y, 1)
    assert abs(c[0] - b) < 1e-12 and abs(c[1] - a) < 1e-12
    for pos in itertools.combinations(range(d), nnz):
        dense = np.zeros(d, dtype=np.float32)
        dense[list(pos)] = y.astype(np.float32)
        mask = dense != 0
        assert mask.sum() == nnz
        # receiver: walk the mask, the t-th set bit gets V(t)
        rebuilt = np.zeros(d, dtype=np.float32)
        rebuilt[mask] = (c[1] * np.arange(1, nnz + 1) + c[0]).astype(np.float32)
        np.testing.assert_array_equal(rebuilt, dense)
    assert d * ex["param_bits"] == ex["bits_dense"]
    assert nnz * (32 + ex["param_bits"]) == ex["bits_key_value"]
    assert d * 1 + 2 * ex["param_bits"] == ex["bits_mask_plus_fit"]


def test_figure1_alternative_reading_position_abscissa():
    """Second reading of the figure: i is the tensor position (1..8).  Values
    placed at positions p with V(p) = 0.6 p + 4.0 are fitted exactly too."""
    ex = _fig1()
    for pos in itertools.combinations(range(1, ex["d"] + 1), ex["nnz"]):
        x = np.array(pos, dtype=np.float64)
        c = oracle.lsq_fit(x, ex["a"] * x + ex["b"], 1)
        assert abs(c[0] - ex["b"]) < 1e-12 and abs(c[1] - ex["a"]) < 1e-12


def test_figure1_through_the_codec():
    """The same four values through the codec's own value path: descending
    sort, one segment, abscissa t in [-1, 1].  The sorted values are
    5.5 - 0.9 t, and decoding returns the fp32 inputs."""
    ex = _fig1()
    V = (ex["a"] * np.arange(1, 5) + ex["b"]).astype(np.float32)  # index order
    enc = oracle.curvefit_encode(V, 1, 1)
    assert (enc.S_eff, enc.D_eff, enc.b) == (1, 1, 2)
    assert abs(enc.coef64[0] - 5.5) < 1e-6 and abs(enc.coef64[1] + 0.9) < 1e-6
    np.testing.assert_array_equal(oracle.sigma_unpack(enc.sigma, 4), [3, 2, 1, 0])
    out = oracle.curvefit_decode(enc.coef, enc.sigma, 4, 1, 1)
    np.testing.assert_allclose(out, V, rtol=0, atol=np.spacing(np.float32(6.4)))
    # codec bit count: 8-bit index mask (as in the figure) + 2 fp32 + 4 x 2-bit map
    assert ex["d"] + 2 * 32 + 4 * enc.b == 80


@pytest.mark.parametrize("D", [0, 1, 2, 3, 5, 7])
def test_polynomial_data_is_reproduced(D):
    rng = np.random.default_rng(D)
    c_true = rng.standard_normal(D + 1)
    x = np.linspace(-1, 1, 257)
    y = np.polynomial.polynomial.polyval(x, c_true)
    c = oracle.lsq_fit(x, y, D)
    assert np.max(np.abs(c - c_true)) <= 1e-11 * max(1.0, np.max(np.abs(c_true)))


@pytest.mark.parametrize("n,D", [(6, 5), (50, 3), (1000, 5), (35_000, 5)])
def test_agrees_with_numpy_polyfit_and_residual_is_orthogonal(n, D):
    rng = np.random.default_rng(n)
    x = (2 * np.arange(n) - (n - 1)) / (n - 1)
    y = np.sort(rng.laplace(0, 5e-4, n))[::-1]
    c = oracle.lsq_fit(x, y, D)
    ref = np.polyfit(x, y, D)[::-1]
    assert np.max(np.abs(c - ref)) <= 1e-9 * np.max(np.abs(ref))
    resid = y - np.polynomial.polynomial.polyval(x, c)
    for p in range(D + 1):
        lhs = abs(np.sum(x**p * resid))
        assert lhs <= 1e-10 * np.sum(np.abs(x**p * y))


def _sort_reference(V):
    # descending by value; +0 ahead of -0; equal values keep their order
    q = np.arange(V.size)
    return np.lexsort((q, np.signbit(V), -V.astype(np.float64)))


def test_sort_descending_stable_signed():
    rng = np.random.default_rng(1)
    V = np.concatenate([workloads.tied_values(4000, 2), rng.standard_normal(3000).astype(np.float32)])
    rng.shuffle(V)
    np.testing.assert_array_equal(oracle.sort_desc(V), _sort_reference(V))


@pytest.mark.parametrize("n", [0, 1, 2, 3, 4, 5, 1000, 1024, 1025, 280_873])
def test_sigma_width(n):
    assert oracle.sigma_bits(n) == max(1, (n - 1).bit_length())


def test_sigma_width_matches_paper_scale():
    # Section 5.1 quotes 19-bit map entries for NCF; a ResNet-50-sized top-1%
    # with P0 (about 280,873 values) also needs 19 bits per entry
    assert oracle.sigma_bits(280_873) == 19
    assert oracle.sigma_bits(1 << 16) == 16


def _pack_reference(vals, b):
    n = vals.size
    bits = np.zeros(max(32, ((n * b + 31) // 32) * 32), dtype=np.uint8)
    for t in range(b):
        bits[np.arange(n) * b + t] = (vals >> t) & 1
    return np.packbits(bits, bitorder="little").view("<u4")[: (n * b + 31) // 32]


@pytest.mark.parametrize("n,D,S", [(1, 5, 1), (7, 5, 3), (100, 5, 8), (5000, 3, 16), (40_000, 5, 8)])
def test_sigma_is_the_inverse_sort_permutation_packed_lsb_first(n, D, S):
    V = workloads.tied_values(n, n) * np.float32(1.5) + workloads.normal(n, n, 1.0)
    enc = oracle.curvefit_encode(V, D, S)
    order = _sort_reference(V)
    rank = np.empty(n, dtype=np.uint64)
    rank[order] = np.arange(n, dtype=np.uint64)
    np.testing.assert_array_equal(oracle.sigma_unpack(enc.sigma, n), rank)
    np.testing.assert_array_equal(enc.sigma, _pack_reference(rank, enc.b))


@pytest.mark.parametrize("n,D,S,Se,De", [
    (0, 5, 8, 0, 0), (1, 5, 8, 1, 0), (5, 5, 8, 1, 4), (6, 5, 8, 1, 5), (47, 5, 8, 7, 5),
    (48, 5, 8, 8, 5), (1_000_000, 5, 8, 8, 5), (3, 3, 16, 1, 2),
])
def test_fit_shape(n, D, S, Se, De):
    assert oracle.fit_shape(n, D, S) == (Se, De)


@pytest.mark.parametrize("D,S", [(1, 4), (3, 16), (5, 8)])
def test_interpolation_special_case_round_trips_values(D, S):
    """n = S (D+1): every segment holds exactly D+1 points, so each fit
    interpolates and decoding returns the values up to the fp32 rounding of
    the coefficients.  A wrong segment boundary, rank or abscissa would show
    as an O(1) error."""
    n = S * (D + 1)
    V = workloads.normal(n, seed=D * 100 + S, scale=1.0)
    enc = oracle.curvefit_encode(V, D, S)
    assert (enc.S_eff, enc.D_eff) == (S, D)
    out = oracle.curvefit_decode(enc.coef, enc.sigma, n, D, S)
    order = _sort_reference(V)
    for s in range(S):
        seg = order[s * (D + 1): (s + 1) * (D + 1)]
        scale = np.abs(enc.coef[s * (D + 1): (s + 1) * (D + 1)]).sum()
        assert np.max(np.abs(out[seg] - V[seg])) <= 4 * np.finfo(np.float32).eps * max(scale, 1e-30)


def test_segments_are_equal_count_and_fitted_separately():
    # two segments from two different lines: the fit of each is exact
    n = 2000
    rank = np.arange(n)
    y = np.where(rank < 1000, 10.0 - rank * 1e-3, -5.0 - (rank - 1000) * 2e-3)
    V = np.random.default_rng(0).permutation(y.astype(np.float32))
    enc = oracle.curvefit_encode(V, 1, 2)
    out = oracle.curvefit_decode(enc.coef, enc.sigma, n, 1, 2)
    np.testing.assert_allclose(out, V, rtol=0, atol=2e-5)


def test_decode_rejects_rank_out_of_range():
    V = workloads.normal(5, seed=3)
    enc = oracle.curvefit_encode(V, 1, 1)
    bad = enc.sigma.copy()
    bad[0] |= 0x7  # first entry (3 bits) now reads 7 >= n
    with pytest.raises(oracle.OracleError):
        oracle.curvefit_decode(enc.coef, bad, 5, 1, 1)
