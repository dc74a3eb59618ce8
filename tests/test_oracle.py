"""Pins for the CPU oracle (runs without a GPU).

The oracle is checked against things other than itself: hand-derived runs of
Algorithm 1 (tests/golden), library routines for special cases (scipy's vector
quantiser for the assignment step, scipy's Lloyd loop, numpy's bincount for
Eq. (1), a sorted-boundary search for M = 1), brute force over all labelings
of tiny inputs, closed forms (K = 1, K = n), the generator's planted blobs, and
invariants of the Lloyd iteration (objective never increases, a converged
state is a fixed point, counts add up to n, permutation equivariance).
"""
import itertools
import json
import os

import numpy as np
import pytest
from scipy.cluster.vq import kmeans2, vq
from scipy.spatial.distance import cdist

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- worked examples

def test_worked_example_2d_whole_run():
    g = _golden("worked_example_2d.json")
    X = np.array(g["X"], np.float32)
    init = np.array(g["init"], np.float32)
    # the farthest-point rule of the input recipe gives the documented init
    idx = workloads.farthest_point_init(X, g["K"])
    assert np.array_equal(X[idx], init)
    labels, centers, counts, iters = oracle.run(X, g["K"], init, 50)
    assert iters == g["iterations"]
    assert labels.tolist() == g["labels_per_iteration"][-1]
    assert np.array_equal(centers, np.array(g["centers_per_iteration"][-1], np.float32))
    assert counts.tolist() == g["counts_per_iteration"][-1]


def test_worked_example_2d_step_by_step():
    g = _golden("worked_example_2d.json")
    X = np.array(g["X"], np.float32)
    C = np.array(g["init"], np.float32)
    for t in range(g["iterations"]):
        lab = oracle.assign(X, C)
        assert lab.tolist() == g["labels_per_iteration"][t]
        assert oracle.sse(X, lab, C) == pytest.approx(g["objective_before_update"][t], rel=1e-12)
        C, cnt = oracle.update(X, lab, g["K"], C)
        assert np.array_equal(C, np.array(g["centers_per_iteration"][t], np.float32))
        assert cnt.tolist() == g["counts_per_iteration"][t]
        assert oracle.sse(X, lab, C) == pytest.approx(g["objective_after_update"][t], rel=1e-12)
    # max_iter cuts the run: labels and centres of the last executed pass
    for T in (1, 2):
        lab, C, cnt, it = oracle.run(X, g["K"], np.array(g["init"], np.float32), T)
        assert it == T
        assert lab.tolist() == g["labels_per_iteration"][T - 1]
        assert np.array_equal(C, np.array(g["centers_per_iteration"][T - 1], np.float32))


def test_ties_and_empty_cluster():
    g = _golden("ties_empty_3pt.json")
    X = np.array(g["X"], np.float32)
    init = np.array(g["init"], np.float32)
    assert np.array_equal(X[workloads.farthest_point_init(X, g["K"])], init)
    labels, centers, counts, iters = oracle.run(X, g["K"], init, 10)
    assert labels.tolist() == g["labels"]
    assert np.array_equal(centers, np.array(g["centers"], np.float32))
    assert counts.tolist() == g["counts"]
    assert iters == g["iterations"]


# ---------------------------------------------------------------- assignment step

@pytest.mark.parametrize("n,M,K,seed", [(1000, 3, 7, 0), (777, 25, 16, 1), (500, 64, 33, 2),
                                        (300, 1, 5, 3), (400, 10, 1, 4)])
def test_assign_matches_scipy_vq(n, M, K, seed):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, M)).astype(np.float32)
    C = rng.standard_normal((K, M)).astype(np.float32)
    lab = oracle.assign(X, C)
    ref, _ = vq(X.astype(np.float64), C.astype(np.float64))
    assert np.array_equal(lab, ref.astype(np.int32))


def test_assign_one_feature_is_sorted_boundary_search():
    # M = 1: the nearest centre is found by locating x among the midpoints of
    # the sorted centres.
    rng = np.random.default_rng(7)
    c = rng.choice(np.arange(-1000, 1000), 23, replace=False).astype(np.float32) * 0.37
    x = rng.uniform(-500, 500, 5000).astype(np.float32)
    order = np.argsort(c)
    cs = c[order].astype(np.float64)
    mids = (cs[1:] + cs[:-1]) / 2
    pos = np.searchsorted(mids, x.astype(np.float64))
    keep = np.min(np.abs(x[:, None].astype(np.float64) - mids[None, :]), axis=1) > 1e-6
    lab = oracle.assign(x[:, None], c[:, None])
    assert np.array_equal(lab[keep], order[pos][keep])


def test_assign_distances_match_cdist():
    rng = np.random.default_rng(11)
    X = rng.standard_normal((400, 6)).astype(np.float32)
    C = rng.standard_normal((9, 6)).astype(np.float32)
    lab, d1, d2 = oracle.assign(X, C, with_dist=True)
    D = np.sort(cdist(X.astype(np.float64), C.astype(np.float64), "sqeuclidean"), axis=1)
    np.testing.assert_allclose(d1, D[:, 0], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(d2, D[:, 1], rtol=1e-12, atol=1e-12)
    g = oracle.gap_rel(d1, d2)
    assert ((g >= 0) & (g <= 1)).all()
    # a point exactly between two centres has gap 0 and goes to the lower index
    lab, d1, d2 = oracle.assign(np.array([[0.5, 0.0]], np.float32),
                                np.array([[1, 0], [0, 0]], np.float32), with_dist=True)
    assert lab[0] == 0 and oracle.gap_rel(d1, d2)[0] == 0.0
    # K = 1: no competitor
    _, d1, d2 = oracle.assign(X, C[:1], with_dist=True)
    assert np.isinf(d2).all() and (oracle.gap_rel(d1, d2) == 1.0).all()


# ---------------------------------------------------------------- update step (Eq. 1)

@pytest.mark.parametrize("n,M,K,seed", [(1000, 4, 6, 0), (5000, 25, 16, 1), (100, 3, 40, 2)])
def test_update_is_bincount_mean(n, M, K, seed):
    rng = np.random.default_rng(seed)
    X = rng.uniform(-50, 50, (n, M)).astype(np.float32)
    labels = rng.integers(0, K, n).astype(np.int32)
    labels[labels == 3] = 2          # cluster 3 (when present) is empty
    prev = rng.uniform(-1, 1, (K, M)).astype(np.float32)
    C, cnt = oracle.update(X, labels, K, prev)
    ref_cnt = np.bincount(labels, minlength=K)
    assert np.array_equal(cnt, ref_cnt)
    for j in range(M):
        s = np.bincount(labels, weights=X[:, j].astype(np.float64), minlength=K)
        with np.errstate(invalid="ignore", divide="ignore"):
            mean = (s / ref_cnt).astype(np.float32)
        want = np.where(ref_cnt > 0, mean, prev[:, j])
        assert np.array_equal(C[:, j], want)


def test_update_rejects_bad_labels_and_allows_alias():
    X = np.ones((4, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.update(X, np.array([0, 1, 2, 5], np.int32), 3, np.zeros((3, 2), np.float32))
    with pytest.raises(ValueError):
        oracle.update(X, np.array([0, -1, 0, 0], np.int32), 3, np.zeros((3, 2), np.float32))


# ---------------------------------------------------------------- whole loop

@pytest.mark.parametrize("n,M,K,T,seed", [(2000, 2, 4, 5, 0), (3000, 10, 8, 7, 1),
                                          (1500, 25, 16, 4, 2)])
def test_fixed_iterations_match_scipy_kmeans2(n, M, K, T, seed):
    # scipy's kmeans2 with a given code book runs exactly `iter` Lloyd passes:
    # assign, then centroids, empty clusters keep their previous centre. It keeps
    # centres in fp64 where the oracle stores fp32, so centres agree to fp32
    # rounding and labels agree exactly on well-separated data.
    X, init = workloads.random_case(n, M, K, seed, kind="blobs")
    lab, C, cnt, it = oracle.run(X, K, init, T, fixed=True)
    assert it == T
    cb, ref_lab = kmeans2(X.astype(np.float64), init.astype(np.float64), iter=T,
                          minit="matrix", missing="warn")
    assert np.array_equal(lab, ref_lab.astype(np.int32))
    np.testing.assert_allclose(C, cb, rtol=2e-6, atol=1e-5)
    assert np.array_equal(cnt, np.bincount(lab, minlength=K))


def test_k1_is_global_mean():
    rng = np.random.default_rng(3)
    X = rng.uniform(-5, 5, (10007, 7)).astype(np.float32)
    lab, C, cnt, it = oracle.run(X, 1, X[:1], 10)
    assert it == 2 and (lab == 0).all() and cnt.tolist() == [10007]
    mean = X.astype(np.float64).mean(axis=0)
    np.testing.assert_allclose(C[0], mean.astype(np.float32), rtol=0, atol=4e-7)


def test_k_equals_n_distinct_points():
    rng = np.random.default_rng(4)
    X = rng.uniform(-1, 1, (37, 5)).astype(np.float32)
    idx = workloads.farthest_point_init(X, 37)
    lab, C, cnt, it = oracle.run(X, 37, X[idx], 10)
    assert it == 2
    assert np.array_equal(C, X[idx])
    assert (cnt == 1).all()
    assert np.array_equal(idx[lab], np.arange(37))


def test_all_points_identical():
    X = np.full((50, 3), 2.5, np.float32)
    init = np.array([[2.5, 2.5, 2.5], [9, 9, 9], [-1, 0, 1]], np.float32)
    lab, C, cnt, it = oracle.run(X, 3, init, 10)
    assert (lab == 0).all() and cnt.tolist() == [50, 0, 0]
    assert np.array_equal(C, init) and it == 2


def _brute_force_opt(X, K):
    n = X.shape[0]
    Xd = X.astype(np.float64)
    best = np.inf
    for labs in itertools.product(range(K), repeat=n):
        labs = np.array(labs)
        s = 0.0
        for k in range(K):
            m = labs == k
            if m.any():
                s += ((Xd[m] - Xd[m].mean(0)) ** 2).sum()
        best = min(best, s)
    return best


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_optimum_bounds_lloyd(seed):
    rng = np.random.default_rng(100 + seed)
    n, K = int(rng.integers(3, 9)), int(rng.integers(2, 4))
    X = rng.uniform(-3, 3, (n, 2)).astype(np.float32)
    idx = workloads.farthest_point_init(X, K)
    lab, C, cnt, it = oracle.run(X, K, X[idx], 100)
    opt = _brute_force_opt(X, K)
    assert oracle.sse(X, lab, C) >= opt * (1 - 1e-9) - 1e-9
    # local optimality at convergence: no object is strictly closer to another centre
    D = cdist(X.astype(np.float64), C.astype(np.float64), "sqeuclidean")
    assert (D[np.arange(n), lab] <= D.min(axis=1) + 1e-12).all()


def test_brute_force_optimum_reached_when_separated():
    rng = np.random.default_rng(9)
    centers = np.array([[0, 0], [20, 0], [0, 20]], np.float64)
    X = (centers[[0, 0, 1, 1, 1, 2, 2, 0]] + 0.3 * rng.standard_normal((8, 2))).astype(np.float32)
    idx = workloads.farthest_point_init(X, 3)
    lab, C, cnt, it = oracle.run(X, 3, X[idx], 100)
    assert oracle.sse(X, lab, C) == pytest.approx(_brute_force_opt(X, 3), rel=1e-6)


# ---------------------------------------------------------------- invariants

def _trace(X, K, init, T):
    C = init
    out = []
    for _ in range(T):
        lab = oracle.assign(X, C)
        before = oracle.sse(X, lab, C)
        C_new, cnt = oracle.update(X, lab, K, C)
        after = oracle.sse(X, lab, C_new)
        out.append((lab, C, C_new, cnt, before, after))
        C = C_new
    return out


@pytest.mark.parametrize("kind,init", [("blobs", "farthest"), ("uniform", "farthest"),
                                       ("uniform", "random"), ("dups", "random")])
def test_objective_never_increases_and_counts_add_up(kind, init):
    X, C0 = workloads.random_case(3001, 5, 12, 21, kind=kind, init=init)
    tr = _trace(X, 12, C0, 12)
    prev_after = np.inf
    for lab, _, _, cnt, before, after in tr:
        assert cnt.sum() == X.shape[0]
        assert lab.min() >= 0 and lab.max() < 12
        assert before <= prev_after * (1 + 1e-9) + 1e-9
        assert after <= before * (1 + 1e-9) + 1e-9
        prev_after = after


def test_run_equals_stepping_and_converged_state_is_fixed_point():
    X, C0 = workloads.random_case(4000, 6, 10, 5, kind="uniform")
    lab, C, cnt, it = oracle.run(X, 10, C0, 200)
    assert it < 200
    tr = _trace(X, 10, C0, it)
    assert np.array_equal(tr[-1][0], lab) and np.array_equal(tr[-1][2], C)
    assert np.array_equal(tr[-1][1], tr[-1][2])            # step 6: congruent
    if it > 2:
        assert not np.array_equal(tr[-2][1], tr[-2][2])    # ... and not earlier
    assert np.array_equal(oracle.assign(X, C), lab)          # fixed point
    C2, cnt2 = oracle.update(X, lab, 10, C)
    assert np.array_equal(C2, C) and np.array_equal(cnt2, cnt)


def test_permutation_equivariance():
    X, C0 = workloads.random_case(2500, 4, 6, 8, kind="blobs")
    perm = np.random.default_rng(1).permutation(2500)
    lab, C, cnt, it = oracle.run(X, 6, C0, 100)
    lab_p, C_p, cnt_p, it_p = oracle.run(X[perm], 6, C0, 100)
    assert it == it_p and np.array_equal(lab[perm], lab_p) and np.array_equal(cnt, cnt_p)
    np.testing.assert_allclose(C, C_p, rtol=1e-6, atol=1e-6)
    # permuting the initial centres permutes labels and centres
    q = np.array([3, 0, 5, 1, 4, 2])
    lab_q, C_q, cnt_q, it_q = oracle.run(X, 6, C0[q], 100)
    inv = np.argsort(q)
    assert np.array_equal(inv[lab], lab_q) and np.array_equal(C[q], C_q)


@pytest.mark.parametrize("name", ["1", "2"])
def test_planted_blobs_recovered(name):
    w = workloads.get(name)
    X, truth, idx, init = workloads.load(name)
    assert len(set(truth[idx].tolist())) == w.K          # init hits every blob
    lab, C, cnt, it = oracle.run(X, w.K, init, w.max_iter, fixed=w.fixed)
    # labels equal the planted truth up to a permutation of cluster names
    pairs = set(zip(truth.tolist(), lab.tolist()))
    assert len(pairs) == w.K
    mapping = dict(pairs)
    assert sorted(mapping.values()) == list(range(w.K))
    planted, sigma = workloads.planted_params(w)
    for t, k in mapping.items():
        tol = 6 * sigma[t] / np.sqrt(cnt[k])
        assert (np.abs(C[k] - planted[t]) <= tol).all()


def test_max_iter_and_fixed_mode():
    X, C0 = workloads.random_case(1000, 3, 5, 2, kind="blobs")
    _, _, _, it = oracle.run(X, 5, C0, 100)
    lab, C, cnt, it_f = oracle.run(X, 5, C0, it + 4, fixed=True)
    assert it_f == it + 4
    tr = _trace(X, 5, C0, it + 4)
    assert np.array_equal(tr[-1][0], lab) and np.array_equal(tr[-1][2], C)
    lab1, C1, _, it1 = oracle.run(X, 5, C0, 1)
    assert it1 == 1 and np.array_equal(lab1, tr[0][0]) and np.array_equal(C1, tr[0][2])
    with pytest.raises(ValueError):
        oracle.run(X, 5, C0, 0)


# ---------------------------------------------------------------- property-based

from hypothesis import given, settings, strategies as st  # noqa: E402


@settings(max_examples=150, deadline=None)
@given(n=st.integers(1, 40), M=st.integers(1, 5), K=st.integers(1, 9),
       seed=st.integers(0, 2**31 - 1), grid=st.booleans())
def test_properties_random_small(n, M, K, seed, grid):
    # duplicate points, K above the number of distinct points, duplicate centres
    rng = np.random.default_rng(seed)
    X = (rng.integers(-2, 3, (n, M)) if grid else rng.standard_normal((n, M))).astype(np.float32)
    init = X[rng.integers(0, n, K)]
    lab, C, cnt, it = oracle.run(X, K, init, 30)
    assert 1 <= it <= 30
    assert cnt.sum() == n and lab.min() >= 0 and lab.max() < K
    assert np.array_equal(cnt, np.bincount(lab, minlength=K))
    # every label is a nearest centre of the previous pass; empty clusters keep centres
    if it < 30:
        assert np.array_equal(oracle.assign(X, C), lab)
    for k in np.flatnonzero(cnt):
        mean = (X[lab == k].astype(np.float64).sum(0) / cnt[k]).astype(np.float32)
        np.testing.assert_array_equal(C[k], mean)
