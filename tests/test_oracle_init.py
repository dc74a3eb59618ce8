"""Pins for the oracle's initial centres (Algorithm 1 step 1, read as
farthest-point traversal from object 0; runs without a GPU).

The oracle is checked against things other than itself: an exact brute-force
statement of the rule in rational arithmetic on small integer-valued inputs
(where exact ties occur), the independent numpy implementation of the input
recipe (different summation order, so equal where no near-tie exists),
Gonzalez's bound for farthest-point traversal (the covering radius of the
chosen set is at most twice the optimal K-centre radius, found by brute force
over all K-subsets), and invariants of the traversal.
"""
import itertools
from fractions import Fraction

import os

import numpy as np
import pytest

import oracle
import workloads


def _exact_farthest(X, K, seeds=(0,)):
    """The rule written out in exact arithmetic: fp32 inputs are dyadic
    rationals, so Fractions give the exact squared distances."""
    Xf = [[Fraction(float(v)) for v in row] for row in X]
    n = len(Xf)
    chosen = list(seeds)
    while len(chosen) < K:
        best, far = None, None
        for i in range(n):
            if i in chosen:
                continue
            d = min(sum((a - b) ** 2 for a, b in zip(Xf[i], Xf[c])) for c in chosen)
            if best is None or d > best:
                best, far = d, i
        chosen.append(far)
    return chosen


@pytest.mark.parametrize("n,M,K,seed", [(12, 2, 5, 0), (20, 3, 20, 1), (15, 1, 7, 2),
                                        (30, 4, 9, 3), (9, 2, 9, 4)])
def test_matches_exact_rule_with_ties(n, M, K, seed):
    rng = np.random.default_rng(seed)
    # few distinct small-integer points: exact ties between candidates and
    # duplicates of chosen objects are common
    X = rng.integers(-2, 3, (n, M)).astype(np.float32)
    assert oracle.init_farthest(X, K).tolist() == _exact_farthest(X, K)


@pytest.mark.parametrize("n,M,K,seed", [(40, 2, 6, 0), (25, 5, 25, 1), (60, 3, 11, 2)])
def test_matches_exact_rule_on_real_values(n, M, K, seed):
    X = np.random.default_rng(seed).standard_normal((n, M)).astype(np.float32)
    assert oracle.init_farthest(X, K).tolist() == _exact_farthest(X, K)


@pytest.mark.parametrize("kind", ["blobs", "uniform", "line"])
@pytest.mark.parametrize("n,M,K,seed", [(5000, 2, 4, 0), (3000, 25, 16, 1), (2000, 64, 40, 2),
                                        (777, 10, 100, 3)])
def test_matches_numpy_recipe(kind, n, M, K, seed):
    X, _ = workloads.random_case(n, M, 1, seed, kind)
    assert np.array_equal(oracle.init_farthest(X, K), workloads.farthest_point_init(X, K))


def _radius(X, idx):
    d = ((X[:, None, :].astype(np.float64) - X[None, idx, :].astype(np.float64)) ** 2).sum(-1)
    return np.sqrt(d.min(axis=1).max())


@pytest.mark.parametrize("seed", range(8))
def test_gonzalez_two_approximation(seed):
    rng = np.random.default_rng(seed)
    n, M, K = 10, 2, 3
    X = rng.uniform(-5, 5, (n, M)).astype(np.float32)
    idx = oracle.init_farthest(X, K)
    opt = min(_radius(X, list(s)) for s in itertools.combinations(range(n), K))
    assert _radius(X, idx) <= 2 * opt * (1 + 1e-12)


def test_invariants_of_the_traversal():
    X, _ = workloads.random_case(3000, 6, 1, 7, "uniform")
    K = 200
    idx = oracle.init_farthest(X, K)
    assert idx[0] == 0 and len(set(idx.tolist())) == K
    X64 = X.astype(np.float64)
    # the distance at which each object was picked never increases
    near = np.full(X.shape[0], np.inf)
    picked = []
    for m in range(1, K):
        near = np.minimum(near, ((X64 - X64[idx[m - 1]]) ** 2).sum(1))
        picked.append(near[idx[m]])
    assert all(a >= b for a, b in zip(picked, picked[1:]))


def test_k_equals_n_is_a_permutation_and_k1_is_object_0():
    X, _ = workloads.random_case(50, 3, 1, 3, "uniform")
    assert sorted(oracle.init_farthest(X, 50).tolist()) == list(range(50))
    assert oracle.init_farthest(X, 1).tolist() == [0]


def test_duplicates_then_lowest_unchosen_indices():
    # 3 distinct values among 10 objects: after the 3 distinct picks every
    # remaining distance is 0, so the lowest unchosen indices follow in order
    X = np.array([[0, 0], [5, 0], [0, 0], [0, 7], [5, 0], [0, 0], [0, 7], [5, 0], [0, 0],
                  [0, 7]], np.float32)
    idx = oracle.init_farthest(X, 10).tolist()
    assert idx[:3] == [0, 3, 1]
    assert idx[3:] == [2, 4, 5, 6, 7, 8, 9]


def test_rejects_k_above_n():
    X = np.zeros((3, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.init_farthest(X, 4)


@pytest.mark.slow
@pytest.mark.parametrize("name", ["aniso25d-n2m-k16", "blobs25d-n2m-k256"])
def test_stored_workload_init_matches(name):
    """The initial centres stored for the 2*10^6 x 25 workloads (written by the
    numpy recipe) are the oracle's."""
    X, _, idx, _ = workloads.load(name)
    assert np.array_equal(oracle.init_farthest(X, workloads.get(name).K), idx)


@pytest.mark.parametrize("name", ["blobs25d-n2m-k256", "zipfnoise25d-n20m-k64"])
def test_stored_init_is_the_oracles(name):
    """The initial objects stored for the two fixed-30 workloads are the ones
    oracle.init_farthest chose on the same inputs: the trajectory goldens,
    written from the oracle alone (tests/golden/make_trajectories.py), record
    the oracle's indices and the SHA-256 of the inputs they were chosen on."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                        f"trajectory_{name}.npz")
    g = np.load(path, allow_pickle=False)
    entry = workloads._init_table()[name]
    assert entry["sha256_x"] == str(g["sha256_x"])
    assert np.array_equal(np.asarray(entry["init"]), g["init_idx"])


@pytest.mark.parametrize("n,M,K,seeds,seed", [(12, 2, 5, (3, 7), 0), (20, 3, 20, (19, 0, 5), 1),
                                              (15, 1, 7, (4,), 2), (30, 4, 9, (2, 2), 3)])
def test_from_seeds_matches_exact_rule(n, M, K, seeds, seed):
    X = np.random.default_rng(seed).integers(-2, 3, (n, M)).astype(np.float32)
    want = _exact_farthest(X, K, seeds)
    assert oracle.init_farthest_from(X, K, seeds).tolist() == want


def test_from_seed_zero_is_the_plain_traversal():
    X, _ = workloads.random_case(3000, 6, 1, 5, "blobs")
    assert np.array_equal(oracle.init_farthest_from(X, 40, [0]), oracle.init_farthest(X, 40))


def test_from_the_diameter_ends():
    X, _ = workloads.random_case(800, 3, 1, 6, "uniform")
    _, k, l = oracle.diameter(X)
    idx = oracle.init_farthest_from(X, 10, [k, l])
    assert idx[:2].tolist() == [k, l]
    assert idx.tolist() == _exact_farthest(X[:800], 10, (k, l))


def test_from_seeds_rejects_bad_seeds():
    X = np.zeros((5, 2), np.float32)
    for seeds, K in (([5], 2), ([-1], 2), ([0, 1, 2], 2)):
        with pytest.raises(ValueError):
            oracle.init_farthest_from(X, K, seeds)
