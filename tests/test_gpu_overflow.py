"""Objects whose fp32 scores overflow, and non-finite objects.

An object with a coordinate near the largest fp32 value has fp32 scores
|c|^2 - 2 x.c that overflow to infinity for some centres, while its fp64
distances (Eq. (2), the oracle's arithmetic) stay finite. Its |x|^2 bound is
infinite, so every kernel sends it to the fp64 decision; that decision must
then consider every centre an exact argmin could pick, including the ones
whose overflowed score left no usable key. Near 3e38 the squared coordinate
dominates the fp64 sum, so the distances to most centres round to the same
value and the label is the lowest index among them (the oracle's strict
comparison in ascending order): a centre left out of the decision shows up
as a different label. Objects holding NaN or an infinity have no finite
distance; the oracle labels them 0, and so must the kernels.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1402_3788_amd as km

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None

# (K, path): the direct form, the small-K kernel with one and four blocks, tiles
CASES = [(4, "direct"), (16, None), (40, None), (64, None), (300, "tiles")]


def objects(K: int, seed: int):
    rng = np.random.default_rng(seed)
    n, M = 4099, 25
    C = rng.uniform(0.6, 2.0, (K, M)).astype(np.float32)
    X = rng.normal(0.0, 1.0, (n, M)).astype(np.float32)
    big = [(5, 3, 3.0e38), (64, 7, -3.0e38), (100, 0, 3.3e38), (2000, 24, 1.5e38),
           (2001, 12, -2.9e38), (4098, 1, 3.0e38)]
    for i, j, v in big:
        X[i, j] = v
    X[777, 5:9] = 2.5e38                   # several overflowing coordinates
    X[7, 2] = np.nan
    X[8, 4] = np.inf
    X[9, 1] = -np.inf
    X[10, :] = np.nan
    return X, C, [b[0] for b in big] + [777, 7, 8, 9, 10]


@pytest.mark.parametrize("K,path", CASES)
def test_overflowing_and_nonfinite_objects_follow_the_oracle(K, path):
    print(f"[overflow] K={K} path={path}", flush=True)
    for seed in range(3):
        X, C, special = objects(K, 100 * K + seed)
        want = oracle.assign(X, C)
        Xg, Cg = torch.from_numpy(X).to(DEV), torch.from_numpy(C).to(DEV)
        got = km.kmeans_assign(Xg, Cg, path=path).cpu().numpy()
        bad = np.flatnonzero(got != want)
        assert bad.size == 0, (f"seed {seed}: {bad.size} labels differ, e.g. objects {bad[:8].tolist()} "
                               f"(special objects {special}): got {got[bad[:8]].tolist()}, "
                               f"oracle {want[bad[:8]].tolist()}")
        # the fused assign + accumulate launch takes the same decisions
        lab, _, cnt, it = km.kmeans_run(Xg, K, Cg, 1, fixed_iters=True, path=path)
        assert it == 1
        assert np.array_equal(lab.cpu().numpy(), want)
        assert np.array_equal(cnt.cpu().numpy(), np.bincount(want, minlength=K))


def test_l1_overflowing_and_nonfinite_objects_follow_the_oracle():
    """The L1 assignment: objects whose fp32 L1 distances to every centre
    overflow (two coordinates near 3e38) while the fp64 distances still differ
    (the centres are spread by 1e31 along the first coordinate, so the fp64
    sums tell them apart and the farthest-out centre is the nearest), and
    objects holding NaN or an infinity."""
    rng = np.random.default_rng(11)
    n, M, K = 4099, 25, 16
    C = rng.uniform(-1.0, 1.0, (K, M)).astype(np.float32)
    C[:, 0] = (np.arange(K) * 1.0e31).astype(np.float32)
    X = rng.normal(0.0, 1.0, (n, M)).astype(np.float32)
    X[:, 0] += C[rng.integers(0, K, n), 0]
    for i in (3, 500, 4097):
        X[i, 0], X[i, 1] = 3.0e38, 3.0e38
    X[7, 2], X[8, 4], X[9, 1] = np.nan, np.inf, -np.inf
    want = oracle.assign(X, C, metric="l1")
    assert want[3] == K - 1                 # the premise: fp64 tells the centres apart
    Xg, Cg = torch.from_numpy(X).to(DEV), torch.from_numpy(C).to(DEV)
    got = km.kmeans_assign(Xg, Cg, metric="l1").cpu().numpy()
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"objects {bad[:8].tolist()}: got {got[bad[:8]].tolist()}, oracle {want[bad[:8]].tolist()}"
    lab, _, cnt, it = km.kmeans_run(Xg, K, Cg, 1, fixed_iters=True, metric="l1")
    assert it == 1 and np.array_equal(lab.cpu().numpy(), want)
    assert np.array_equal(cnt.cpu().numpy(), np.bincount(want, minlength=K))


@pytest.mark.parametrize("case", ["nan", "inf", "nan_first", "huge"])
def test_farthest_init_with_nonfinite_objects_follows_the_oracle(case):
    """Farthest-point initial centres (Algorithm 1 step 1) on objects with a
    NaN, an infinity (a NaN distance never lowers an object's nearest-centre
    distance, an infinite one makes the object the farthest), a first object
    of NaNs, and coordinates near the fp32 maximum: the same indices as the
    oracle's traversal."""
    rng = np.random.default_rng(5)
    n, M, K = 3001, 25, 16
    X = rng.normal(0.0, 1.0, (n, M)).astype(np.float32)
    if case == "nan":
        X[17, 3] = np.nan
    elif case == "inf":
        X[17, 3] = np.inf
    elif case == "nan_first":
        X[0, :] = np.nan
    else:
        X[100, 2], X[200, 5] = 3.0e38, -3.0e38
    want = np.asarray(oracle.init_farthest(X, K)).ravel()
    got, _ = km.kmeans_init_farthest(torch.from_numpy(X).to(DEV), K)
    got = got.cpu().numpy().ravel() if hasattr(got, "cpu") else np.asarray(got).ravel()
    assert np.array_equal(got[:K], want[:K])
