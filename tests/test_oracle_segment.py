"""Pins of the oracle's adaptive segmentation and segment-count heuristic
(Section 5, "Piece-wise approximation", Lemma 1; Remark 4 of Section 10).

The chord rule splits a sorted curve at the point farthest from the line
joining the segment's end points.  On curves made of straight pieces the
farthest point is a known vertex, so the expected segment starts follow
from the construction, not from the oracle."""
import math

import numpy as np
import pytest

import oracle

CH, EQ = oracle.SEG_CHORD, oracle.SEG_EQUAL


def pieces(*knots):
    """A descending piecewise-linear curve through (rank, value) vertices,
    values exact in fp32 (multiples of 1/8)."""
    out = []
    for (r0, v0), (r1, v1) in zip(knots, knots[1:]):
        for r in range(r0, r1):
            out.append(v0 + (v1 - v0) * (r - r0) / (r1 - r0))
    out.append(knots[-1][1])
    return np.array(out, dtype=np.float32)


def test_one_elbow_is_found_and_ends_the_left_segment():
    # steep from rank 0 to 40, then shallow to rank 200: the vertex at rank
    # 40 is farthest from the chord
    C = pieces((0, 100.0), (40, 20.0), (200, 4.0))
    b = oracle.segment(C, 1, 2, CH)
    np.testing.assert_array_equal(b, [0, 41, C.size])


def test_two_elbows_with_three_segments():
    C = pieces((0, 400.0), (30, 100.0), (90, 40.0), (300, 8.0))
    b = oracle.segment(C, 1, 3, CH)
    np.testing.assert_array_equal(b, [0, 31, 91, C.size])


def test_greedy_splits_the_farthest_segment_first():
    # positive part almost straight, negative part with a sharp elbow: with
    # three segments the extra split goes to the negative part
    pos = pieces((0, 8.0), (100, 4.0), (200, 0.5))        # slight bend at 100
    neg = -pieces((0, 0.5), (150, 60.0), (200, 400.0))[::-1]  # descending negatives, sharp bend
    C = np.concatenate([pos, neg]).astype(np.float32)
    b = oracle.segment(C, 1, 3, CH)
    assert b[1] == pos.size  # the sign split
    assert b.size == 4 and b[2] > pos.size  # the third segment comes from the negative part
    b4 = oracle.segment(C, 1, 4, CH)
    assert b4.size == 5 and 0 < b4[1] < pos.size  # only then the positive part


def test_sign_split_comes_first():
    C = np.sort(np.linspace(-3, 5, 97).astype(np.float32))[::-1].copy()
    l = int(np.sum(~np.signbit(C)))
    b = oracle.segment(C, 1, 2, CH)
    np.testing.assert_array_equal(b, [0, l, C.size])
    # one segment requested: no split at all
    np.testing.assert_array_equal(oracle.segment(C, 1, 1, CH), [0, C.size])


def test_no_segment_below_degree_plus_one_points():
    C = pieces((0, 50.0), (3, 10.0), (40, 0.0))
    for D in range(0, 6):
        b = oracle.segment(C, D, 8, CH)
        assert np.all(np.diff(b) >= D + 1), (D, b)
    # 2D + 1 points cannot be split at all
    C5 = pieces((0, 9.0), (5, 1.0), (10, 0.0))  # 11 points
    np.testing.assert_array_equal(oracle.segment(C5, 5, 4, CH), [0, 11])


def test_a_straight_curve_is_not_split():
    C = (np.arange(64, dtype=np.float32)[::-1] * 0.25).copy()
    np.testing.assert_array_equal(oracle.segment(C, 1, 8, CH), [0, 64])


def test_equal_mode_matches_the_closed_form():
    C = np.sort(np.random.default_rng(3).normal(size=1001).astype(np.float32))[::-1].copy()
    for S in (1, 3, 8):
        b = oracle.segment(C, 5, S, EQ)
        se = min(S, max(1, 1001 // 6))
        np.testing.assert_array_equal(b, [s * 1001 // se for s in range(se + 1)])


def test_piecewise_polynomials_are_reproduced_after_chord_segmentation():
    # two cubic pieces meeting at a convex corner at rank 59 (a continuous
    # curve, the corner being the left piece's last point): chord
    # segmentation finds the corner and the degree-3 fits then reproduce
    # both pieces
    u = np.arange(60) / 59.0
    w = np.arange(1, 141) / 140.0
    a = 50 - 30 * u + 4 * u**3
    b = 24 - 2 * w + 0.5 * w**2 - 0.25 * w**3
    V = np.concatenate([a, b]).astype(np.float32)
    rng = np.random.default_rng(1)
    Vs = V[rng.permutation(V.size)]
    fit = oracle.curvefit_encode(Vs, 3, 2, CH)
    np.testing.assert_array_equal(fit.bounds, [0, 60, 200])
    y = oracle.curvefit_decode_seg(fit.coef, fit.sigma, V.size, 3, fit.bounds)
    np.testing.assert_allclose(y, Vs, rtol=2e-6, atol=2e-5)


def test_decode_with_equal_bounds_is_the_plain_decode():
    V = np.random.default_rng(9).laplace(0, 1e-3, 5000).astype(np.float32)
    fit = oracle.curvefit_encode(V, 5, 8, EQ)
    a = oracle.curvefit_decode(fit.coef, fit.sigma, V.size, 5, 8)
    b = oracle.curvefit_decode_seg(fit.coef, fit.sigma, V.size, 5, fit.bounds)
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("M", [0.0, 0.01, 0.25, 1.0, 2.25, 2.26, 6.25, 30.0, 1e3])
def test_heuristic_is_ceil_two_sqrt_m_plus_one(M):
    # C[0] - C[1] = M + 1 and C[n-2] - C[n-1] = 1 give M; the count is p + 1
    # with p = ceil(2 sqrt(M)) (Section 5) for degree >= 1
    C = np.array([M + 3.0, 2.0, 1.5, 1.0, 0.0], dtype=np.float64)
    Mc = abs((np.float32(C[0]) - np.float32(C[1])) - 1.0)
    C = C.astype(np.float32)
    for D in (1, 3):
        assert oracle.seg_heuristic(C, D) == min(4096, math.ceil(2 * math.sqrt(Mc)) + 1)


@pytest.mark.parametrize("M", [0.0, 1.0, 1.5, 2 * math.sqrt(2), 3.0, 100.0])
def test_heuristic_for_constants_follows_remark_4(M):
    C = np.array([M + 3.0, 2.0, 1.5, 1.0, 0.0], dtype=np.float32)
    Mc = abs((float(C[0]) - float(C[1])) - 1.0)
    want = max(0, math.ceil(Mc / math.sqrt(2) - 1 - 1e-12)) + 1
    assert oracle.seg_heuristic(C, 0) == want


def test_heuristic_on_tiny_inputs():
    assert oracle.seg_heuristic(np.zeros(0, np.float32), 1) == 1
    assert oracle.seg_heuristic(np.array([5.0], np.float32), 1) == 1
    # n = 2: both differences are the same one, M = 0
    assert oracle.seg_heuristic(np.array([5.0, 1.0], np.float32), 1) == 1


def test_round_trip_with_chord_segments_and_the_heuristic():
    from paper_2102_03112_amd import workloads as W

    g = W.normal(20_000, 4, scale=1e-3)
    res = oracle.roundtrip_tensor(g, 400, 1e-3, 1, 0, seg_mode=CH)
    assert res.fit.S_eff >= 1 and res.fit.bounds[-1] == res.fit.n
    assert np.all(np.diff(res.fit.bounds.astype(np.int64)) >= 2)
    # the decode recovers values on the sorted curve's fit: error well below
    # the values' spread
    err = np.linalg.norm(res.vals - g[res.P_dec.astype(np.int64)]) / np.linalg.norm(g[res.P_dec.astype(np.int64)])
    assert err < 0.5
