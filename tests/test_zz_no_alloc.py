"""kmeans_run_noalloc (the entry point for callers that cannot allocate) against
kmeans_run with a caller workspace: identical labels, centres, counts and
iteration counts, on two calls in a row, the second with a smaller input
(the static per-GPU workspace keeps the first call's contents), on each
distance path; and the refusal of a shape whose workspace exceeds the static
array."""
import numpy as np
import pytest
import torch

import paper_1402_3788_amd as km
import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None


def _both(X, C0, K, max_iter, fixed, path=None, metric="l2"):
    Xg, Cg = torch.from_numpy(X).to(DEV), torch.from_numpy(C0).to(DEV)
    n, M = X.shape
    ref = km.kmeans_run(Xg, K, Cg, max_iter, fixed_iters=fixed, path=path, metric=metric)
    out = (torch.full((n,), -7, dtype=torch.int32, device=DEV),
           torch.full((K, M), 9.0, dtype=torch.float32, device=DEV),
           torch.full((K,), -7, dtype=torch.int32, device=DEV))
    it = km.kmeans_run_noalloc(Xg, K, Cg, max_iter, out, fixed_iters=fixed, path=path,
                               metric=metric)
    assert it == ref[3]
    assert torch.equal(out[0], ref[0])
    assert torch.equal(out[1].view(torch.int32), ref[1].view(torch.int32))
    assert torch.equal(out[2], ref[2])
    return it


@pytest.mark.parametrize("path,K,metric", [(None, 16, "l2"), ("tiles", 64, "l2"),
                                            ("direct", 4, "l2"), (None, 12, "l1"),
                                            ("tiles", 256, "l2")])
def test_noalloc_equals_workspace_run(path, K, metric):
    print(f"[noalloc] path={path} K={K} metric={metric}", flush=True)
    for n, seed, fixed in ((200_003, 1, False), (50_001, 2, True)):
        X, C0 = workloads.random_case(n, 25, K, seed=seed + K, kind="blobs")
        assert km.kmeans_workspace_bytes(n, 25, K) <= km.NOALLOC_MAX_WORKSPACE
        it = _both(X, C0, K, 30, fixed, path=path, metric=metric)
        print(f"[noalloc] n={n}: {it} iterations, identical to the workspace run", flush=True)


def test_noalloc_refuses_oversized_workspace():
    n, M, K = 1_000_000, 16, 1024
    assert km.kmeans_workspace_bytes(n, M, K) > km.NOALLOC_MAX_WORKSPACE
    X = torch.zeros((n, M), dtype=torch.float32, device=DEV)
    C = torch.zeros((K, M), dtype=torch.float32, device=DEV)
    out = (torch.empty(n, dtype=torch.int32, device=DEV), torch.empty((K, M), device=DEV),
           torch.empty(K, dtype=torch.int32, device=DEV))
    with pytest.raises(km.KmeansError) as e:
        km.kmeans_run_noalloc(X, K, C, 5, out)
    assert e.value.code == km.KMEANS_EWORKSPACE
    # and a call that fits still works afterwards
    Xs, Cs = workloads.random_case(10_000, 25, 16, seed=3, kind="blobs")
    _both(Xs, Cs, 16, 20, False)
