"""Pins for the oracle's L1 (city-block) assignment, the other metric the
paper allows in place of Eq. (2); only the assignment changes, the centres
stay the centres of gravity of Eq. (1). Runs without a GPU.

Checked against scipy's cdist with the cityblock metric, an exact rational
brute force on small integer-valued inputs (exact ties, lowest index), the
one-feature case (where L1 and squared Euclidean order centres alike), and
fixed-count runs rebuilt from scipy's assignment and numpy's means.
"""
from fractions import Fraction

import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle
import workloads


@pytest.mark.parametrize("n,M,K,seed", [(1000, 3, 7, 0), (777, 25, 16, 1), (500, 64, 33, 2),
                                        (2000, 2, 300, 3)])
def test_l1_assign_matches_cdist(n, M, K, seed):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, M)).astype(np.float32)
    C = rng.standard_normal((K, M)).astype(np.float32)
    lab, d1, d2 = oracle.assign(X, C, with_dist=True, metric="l1")
    D = cdist(X.astype(np.float64), C.astype(np.float64), "cityblock")
    assert np.array_equal(lab, np.argmin(D, axis=1))
    np.testing.assert_allclose(d1, D.min(axis=1), rtol=1e-12)
    np.testing.assert_allclose(d2, np.sort(D, axis=1)[:, 1], rtol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_l1_assign_exact_with_ties(seed):
    rng = np.random.default_rng(seed)
    X = rng.integers(-3, 4, (40, 3)).astype(np.float32)
    C = rng.integers(-3, 4, (6, 3)).astype(np.float32)
    want = []
    for x in X:
        d = [sum(abs(Fraction(float(a)) - Fraction(float(b))) for a, b in zip(x, c)) for c in C]
        want.append(min(range(len(C)), key=lambda k: (d[k], k)))
    assert oracle.assign(X, C, metric="l1").tolist() == want


def test_l1_one_feature_orders_like_l2():
    rng = np.random.default_rng(4)
    X = rng.uniform(-10, 10, (3000, 1)).astype(np.float32)
    C = rng.uniform(-10, 10, (9, 1)).astype(np.float32)
    assert np.array_equal(oracle.assign(X, C, metric="l1"), oracle.assign(X, C))


@pytest.mark.parametrize("n,M,K,T,seed", [(3000, 4, 6, 7, 0), (5000, 25, 16, 5, 1),
                                          (800, 3, 40, 9, 2)])
def test_l1_fixed_run_rebuilt_from_scipy(n, M, K, T, seed):
    X, C0 = workloads.random_case(n, M, K, seed, "blobs")
    C = C0.copy()
    X64 = X.astype(np.float64)
    for _ in range(T):
        lab = np.argmin(cdist(X64, C.astype(np.float64), "cityblock"), axis=1)
        cnt = np.bincount(lab, minlength=K)
        S = np.zeros((K, M))
        np.add.at(S, lab, X64)
        newC = C.copy()
        nz = cnt > 0
        newC[nz] = (S[nz] / cnt[nz, None]).astype(np.float32)
        C = newC
    olab, oC, ocnt, oit = oracle.run(X, K, C0, T, fixed=True, metric="l1")
    assert oit == T
    assert np.array_equal(olab, lab) and np.array_equal(ocnt, cnt)
    # numpy's add.at sums in another order than the oracle: at most one unit
    # in the last fp32 place
    assert (np.abs(oC.astype(np.float64) - C) <= np.spacing(np.abs(C))).all()


def test_l1_run_stops_on_congruent_centres():
    X, C0 = workloads.random_case(4000, 5, 5, 9, "blobs")
    lab, C, cnt, it = oracle.run(X, 5, C0, 100, metric="l1")
    assert 2 <= it < 100
    lab2, C2, _, _ = oracle.run(X, 5, C, 2, metric="l1")
    assert np.array_equal(C2, C) and np.array_equal(lab2, lab)


def test_unknown_metric_rejected():
    with pytest.raises(ValueError):
        oracle.assign(np.zeros((2, 2), np.float32), np.zeros((1, 2), np.float32), metric="l3")
