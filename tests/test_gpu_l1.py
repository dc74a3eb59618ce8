"""GPU parity of the L1 (city-block) assignment and of Lloyd runs that use it
(KMEANS_METRIC_L1), against the CPU oracle, through the C ABI.

The library re-decides every fp32 call too close to make in fp64 in the
oracle's operation order, so labels must be identical to the oracle's
everywhere (exact ties included); centres are the centres of gravity of those
labels, within 1e-5 (in practice bit-identical); iteration counts equal.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1402_3788_amd as km
import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None


def _say(msg):
    print(msg, flush=True)


def _gpu(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _gamma(m):
    u = 2.0 ** -24
    return m * u / (1 - m * u)


@pytest.mark.parametrize("n,M,K,kind", [(1, 1, 1, "uniform"), (777, 2, 3, "dups"),
                                        (65_537, 25, 16, "blobs"), (10_000, 64, 200, "uniform"),
                                        (4_000, 16, 1024, "uniform"), (3_000, 33, 100, "dups"),
                                        (50_001, 7, 9, "line"), (64, 5, 70, "uniform")])
def test_l1_assign_parity(n, M, K, kind):
    _say(f"[l1 assign] n={n} M={M} K={K} kind={kind}")
    X, C = workloads.random_case(n, M, K, seed=n + K, kind=kind,
                                 init="farthest" if K <= n else "random")
    lab, d = km.kmeans_assign(_gpu(X), _gpu(C), with_min_d2=True, metric="l1")
    torch.cuda.synchronize()
    olab, d1, _ = oracle.assign(X, C, with_dist=True, metric="l1")
    assert np.array_equal(lab.cpu().numpy(), olab)
    d = d.cpu().numpy().astype(np.float64)
    assert (np.abs(d - d1) <= 1.01 * _gamma(M) * d1 + 1e-30).all()


@pytest.mark.parametrize("n,M,K,max_iter,fixed", [(5_000, 2, 4, 50, False),
                                                  (50_003, 25, 16, 30, False),
                                                  (20_011, 10, 64, 12, True),
                                                  (9_999, 64, 100, 8, True),
                                                  (30_001, 25, 256, 6, True)])
def test_l1_run_parity(n, M, K, max_iter, fixed):
    _say(f"[l1 run] n={n} M={M} K={K} max_iter={max_iter} fixed={fixed}")
    X, C0 = workloads.random_case(n, M, K, seed=n, kind="blobs")
    lab, C, cnt, it = km.kmeans_run(_gpu(X), K, _gpu(C0), max_iter, fixed_iters=fixed,
                                    metric="l1")
    olab, oC, ocnt, oit = oracle.run(X, K, C0, max_iter, fixed=fixed, metric="l1")
    assert it == oit
    assert np.array_equal(lab.cpu().numpy(), olab)
    assert np.array_equal(cnt.cpu().numpy(), ocnt)
    C = C.cpu().numpy()
    scale = np.maximum(np.abs(oC).max(axis=1, keepdims=True), 1e-30)
    assert (np.abs(C.astype(np.float64) - oC) <= 1e-5 * scale).all()
    _say(f"[l1 run] iterations {it}, centre coordinates not bit-identical "
         f"{int((C.view(np.uint32) != oC.view(np.uint32)).sum())}")


def test_l1_workload3_fixed_iterations():
    """The 2*10^6 x 25, K = 16 workload, 4 fixed L1 iterations."""
    X, _, _, init = workloads.load("aniso25d-n2m-k16")
    _say("[l1 run] aniso25d-n2m-k16 fixed 4")
    lab, C, cnt, it = km.kmeans_run(_gpu(X), 16, _gpu(init), 4, fixed_iters=True, metric="l1")
    olab, oC, ocnt, oit = oracle.run(X, 16, init, 4, fixed=True, metric="l1")
    assert it == oit == 4
    assert np.array_equal(lab.cpu().numpy(), olab) and np.array_equal(cnt.cpu().numpy(), ocnt)
    C = C.cpu().numpy()
    scale = np.maximum(np.abs(oC).max(axis=1, keepdims=True), 1e-30)
    assert (np.abs(C.astype(np.float64) - oC) <= 1e-5 * scale).all()
