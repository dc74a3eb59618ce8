"""The multi-threaded CPU regime (Algorithm 3) against the single-threaded
oracle (runs without a GPU).

Its assignment is the oracle's arithmetic, so labels, counts and iteration
counts must be identical; with one thread its sums are added in the oracle's
order, so centres must be identical bit for bit; with several threads the
partial sums are added per thread and then across threads, so a centre may
differ in its last fp32 bit (checked within 1e-5 relative, as for the GPU).
"""
import numpy as np
import pytest

import oracle
import workloads


@pytest.mark.parametrize("n,M,K,kind,max_iter,fixed", [
    (5000, 2, 4, "blobs", 50, False), (20_001, 10, 8, "blobs", 100, False),
    (30_000, 25, 16, "uniform", 6, True), (777, 3, 40, "dups", 20, False),
    (1, 4, 1, "uniform", 3, False), (64, 5, 64, "uniform", 5, True),
])
@pytest.mark.parametrize("threads", [1, 3, 8])
def test_alg3_matches_oracle(n, M, K, kind, max_iter, fixed, threads):
    X, init = workloads.random_case(n, M, K, seed=n + K, kind=kind,
                                    init="farthest" if K <= n else "random")
    lab, C, cnt, it, used = oracle.alg3_run(X, K, init, max_iter, fixed, threads)
    olab, oC, ocnt, oit = oracle.run(X, K, init, max_iter, fixed)
    assert used == threads
    assert it == oit
    assert np.array_equal(lab, olab) and np.array_equal(cnt, ocnt)
    if threads == 1:
        assert np.array_equal(C.view(np.uint32), oC.view(np.uint32))
    scale = np.maximum(np.abs(oC).max(axis=1, keepdims=True), 1e-30)
    assert (np.abs(C.astype(np.float64) - oC) <= 1e-5 * scale).all()
