"""Pins for the oracle's diameter of Eq. (3) and centre of gravity of the
whole set (Algorithm 2 steps 1-2; runs without a GPU).

Checked against things other than the oracle itself: scipy's pairwise
distances, an exact brute force in rational arithmetic on small integer-valued
inputs (exact ties, lowest pair), the closed form for one feature (the two
extreme values), the convex hull in the plane (the diameter joins two hull
vertices), necessary conditions of a farthest pair, and an exactly rounded
sum (math.fsum) for the centre of gravity.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
from scipy.spatial import ConvexHull
from scipy.spatial.distance import pdist, squareform

import oracle
import workloads


def _exact_diameter(X):
    Xf = [[Fraction(float(v)) for v in row] for row in X]
    best, pair = None, (0, 0)
    for k, l in itertools.combinations(range(len(Xf)), 2):
        d = sum((a - b) ** 2 for a, b in zip(Xf[k], Xf[l]))
        if best is None or d > best:
            best, pair = d, (k, l)
    return (best if best is not None else Fraction(0)), pair


@pytest.mark.parametrize("n,M,seed", [(12, 2, 0), (20, 3, 1), (15, 1, 2), (30, 4, 3), (9, 2, 4),
                                      (25, 5, 5)])
def test_matches_exact_rule_with_ties(n, M, seed):
    X = np.random.default_rng(seed).integers(-3, 4, (n, M)).astype(np.float32)
    d2, k, l = oracle.diameter(X)
    best, pair = _exact_diameter(X)
    assert (k, l) == pair and d2 == float(best)


@pytest.mark.parametrize("kind", ["blobs", "uniform", "line"])
@pytest.mark.parametrize("n,M,seed", [(2000, 25, 0), (1500, 2, 1), (800, 64, 2), (3000, 7, 3)])
def test_matches_scipy_pdist(kind, n, M, seed):
    X, _ = workloads.random_case(n, M, 1, seed, kind)
    d2, k, l = oracle.diameter(X)
    D = squareform(pdist(X.astype(np.float64), "sqeuclidean"))
    assert d2 == pytest.approx(D.max(), rel=1e-12)
    kk, ll = np.unravel_index(np.argmax(D), D.shape)
    assert (k, l) == (min(kk, ll), max(kk, ll))


@pytest.mark.parametrize("seed", range(5))
def test_one_feature_is_the_extremes(seed):
    x = np.random.default_rng(seed).integers(-20, 21, 300).astype(np.float32)
    d2, k, l = oracle.diameter(x[:, None])
    a, b = int(np.argmin(x)), int(np.argmax(x))
    assert d2 == (float(x.max()) - float(x.min())) ** 2
    assert (k, l) == (min(a, b), max(a, b))


@pytest.mark.parametrize("seed", range(4))
def test_plane_diameter_joins_hull_vertices(seed):
    X = np.random.default_rng(seed).standard_normal((4000, 2)).astype(np.float32)
    d2, k, l = oracle.diameter(X)
    hull = ConvexHull(X.astype(np.float64)).vertices
    assert k in hull and l in hull
    H = X[hull].astype(np.float64)
    assert d2 == pytest.approx(pdist(H, "sqeuclidean").max(), rel=1e-12)


def test_farthest_pair_conditions():
    X, _ = workloads.random_case(3000, 10, 1, 9, "uniform")
    d2, k, l = oracle.diameter(X)
    X64 = X.astype(np.float64)
    dk = ((X64 - X64[k]) ** 2).sum(1)
    dl = ((X64 - X64[l]) ** 2).sum(1)
    # each endpoint is a farthest object from the other, and no object is
    # farther from object 0 than the diameter
    assert dk.max() == pytest.approx(d2, rel=1e-12) and np.argmax(dk) == l
    assert dl.max() == pytest.approx(d2, rel=1e-12) and np.argmax(dl) == k
    d0 = ((X64 - X64[0]) ** 2).sum(1).max()
    assert d0 <= d2 * (1 + 1e-12) and d2 <= 4 * d0 * (1 + 1e-12)


def test_degenerate_sets():
    assert oracle.diameter(np.array([[1.5, -2.0]], np.float32)) == (0.0, 0, 0)
    d2, k, l = oracle.diameter(np.array([[0, 0], [3, 4]], np.float32))
    assert (d2, k, l) == (25.0, 0, 1)
    assert oracle.diameter(np.full((7, 3), 2.5, np.float32)) == (0.0, 0, 1)


@pytest.mark.parametrize("n,M,seed", [(1, 3, 0), (1000, 25, 1), (12345, 10, 2), (50_000, 2, 3)])
def test_centroid_is_the_exactly_rounded_mean(n, M, seed):
    X = (np.random.default_rng(seed).standard_normal((n, M)) * 50 + 10).astype(np.float32)
    c = oracle.centroid(X)
    want = np.array([math.fsum(X[:, j].astype(np.float64)) / n for j in range(M)],
                    np.float32)
    # the fp64 running sum is within a few units of 2^-53 of the exact one, so
    # the fp32 mean can differ from the exactly rounded one only at a rounding
    # boundary, by one unit in the last place
    ulp = np.spacing(np.abs(want))
    assert (np.abs(c.astype(np.float64) - want) <= ulp).all()
    assert (c == want).mean() >= 0.9


def test_centroid_of_a_translated_grid():
    g = np.arange(-4, 5, dtype=np.float32)
    X = np.stack(np.meshgrid(g, g, g), -1).reshape(-1, 3) + np.float32(7.0)
    assert np.array_equal(oracle.centroid(X), np.full(3, 7.0, np.float32))


def test_nonfinite_coordinates_leave_the_diameter_undefined():
    """A NaN or an infinite coordinate anywhere: (nan, -1, -1), whatever the
    other objects (the reading for data outside the real vectors the paper
    defines the diameter on); finite data, however large, keeps its pair."""
    rng = np.random.default_rng(3)
    for bad in (np.nan, np.inf, -np.inf):
        for where in ((0, 0), (5, 2), (19, 3)):
            X = rng.normal(0.0, 1.0, (20, 4)).astype(np.float32)
            X[where] = bad
            d2, k, l = oracle.diameter(X)
            assert np.isnan(d2) and (k, l) == (-1, -1)
    X = rng.normal(0.0, 1.0, (20, 4)).astype(np.float32)
    X[3, 1], X[11, 1] = 3.0e38, -3.0e38
    d2, k, l = oracle.diameter(X)
    assert (k, l) == (3, 11) and d2 > 3.5e77
