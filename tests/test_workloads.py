"""The seeded input recipe (runs without a GPU): cluster sizes, shapes and
determinism of the synthetic workloads that stand in for the paper's
confidential data."""
import numpy as np
import pytest

import workloads


def test_zipf_sizes_of_the_noisy_workload():
    # 90 % of 2*10^7 objects in 64 blobs with sizes proportional to (k+1)^-1.2
    s = workloads.zipf_sizes(18_000_000, 64, 1.2)
    assert s.sum() == 18_000_000 and len(s) == 64
    assert s[0] == 5_265_319 and s[-1] == 35_810
    assert (np.diff(s) <= 0).all()
    w = np.arange(1, 65, dtype=np.float64) ** -1.2
    assert np.abs(s - 18_000_000 * w / w.sum()).max() < 1.0


def test_equal_sizes_give_the_remainder_to_the_first_clusters():
    s = workloads.equal_sizes(2_000_000, 256)
    assert s.sum() == 2_000_000 and s.max() - s.min() == 1
    assert (s[:128] == 7813).all() and (s[128:] == 7812).all()


@pytest.mark.parametrize("name", ["1", "2"])
def test_small_workloads_are_seeded_and_shaped(name):
    w = workloads.get(name)
    X1, t1 = workloads.generate(w)
    X2, t2 = workloads.generate(w)
    assert X1.shape == (w.n, w.M) and X1.dtype == np.float32 and X1.flags.c_contiguous
    assert np.array_equal(X1, X2) and np.array_equal(t1, t2)
    assert set(np.unique(t1)) == set(range(w.K))
    # objects are shuffled: the truth labels are not sorted
    assert (np.diff(t1) != 0).mean() > 0.5


def test_random_case_kinds():
    for kind in ("blobs", "uniform", "dups", "line"):
        X, C = workloads.random_case(500, 3, 7, 1, kind)
        assert X.shape == (500, 3) and C.shape == (7, 3)
        assert X.dtype == np.float32 and C.dtype == np.float32
    X, C = workloads.random_case(5, 2, 9, 0, "uniform", init="random")
    assert C.shape == (9, 2)
    with pytest.raises(ValueError):
        workloads.random_case(5, 2, 9, 0, "uniform", init="farthest")
