"""GPU parity of the farthest-point initial centres (Algorithm 1 step 1 as
read from object 0) against the CPU oracle, through the C ABI.

The chosen indices are an argmax decided by fp64 distances in one fixed
operation order on both sides, so the bar is bit-exact: the same indices, and
centres equal to the chosen rows bit for bit.
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


def _case(n, M, kind, seed):
    X, _ = workloads.random_case(n, M, 1, seed, kind)
    return X


def check_init(X, K, name=""):
    _say(f"[init] {name} n={X.shape[0]} M={X.shape[1]} K={K}")
    Xd = torch.from_numpy(X).to(DEV)
    idx, C = km.kmeans_init_farthest(Xd, K)
    torch.cuda.synchronize()
    idx, C = idx.cpu().numpy(), C.cpu().numpy()
    want = oracle.init_farthest(X, K)
    assert np.array_equal(idx, want), f"first difference at m={int(np.argmax(idx != want))}"
    assert np.array_equal(C.view(np.uint32), X[want].view(np.uint32))
    return idx


@pytest.mark.parametrize("n,M,K,kind", [
    (1, 1, 1, "uniform"), (1, 7, 1, "uniform"), (2, 3, 2, "uniform"),
    (63, 3, 10, "dups"), (64, 2, 64, "uniform"), (65, 25, 16, "blobs"),
    (130, 5, 130, "dups"), (1000, 1, 50, "line"), (4097, 7, 33, "dups"),
    (4097, 4, 3, "uniform"), (100_003, 25, 16, "blobs"), (50_000, 64, 100, "uniform"),
    (20_011, 16, 1024, "uniform"), (30_000, 64, 256, "blobs"), (70_001, 33, 40, "dups"),
    (200_000, 10, 8, "blobs"), (10_000, 2, 4, "blobs"),
])
def test_init_parity(n, M, K, kind):
    check_init(_case(n, M, kind, seed=n + 3 * M + K), K, kind)


def test_init_ties_and_duplicates_exact():
    # three distinct values: (0,7) is farthest from object 0, then (5,0); after
    # them every distance is 0 and the lowest unchosen indices follow in order
    X = np.tile(np.array([[0, 0], [5, 0], [0, 7]], np.float32), (700, 1))
    idx = check_init(X, 40, "three values repeated")
    assert idx[:3].tolist() == [0, 2, 1] and idx[3:].tolist() == list(range(3, 40))


def test_init_repeatable_and_reuses_workspace():
    X = _case(300_001, 25, "uniform", 5)
    Xd = torch.from_numpy(X).to(DEV)
    ws = torch.empty(km.kmeans_init_workspace_bytes(300_001, 25, 64), dtype=torch.uint8,
                     device=DEV)
    a = km.kmeans_init_farthest(Xd, 64, ws=ws)[0].cpu()
    b = km.kmeans_init_farthest(Xd, 17, ws=ws)[0].cpu()
    c = km.kmeans_init_farthest(Xd, 64, ws=ws)[0].cpu()
    assert torch.equal(a, c) and torch.equal(a[:17], b)
    assert np.array_equal(a.numpy(), oracle.init_farthest(X, 64))


@pytest.mark.parametrize("name", ["aniso25d-n2m-k16", "blobs25d-n2m-k256"])
def test_init_workload_full_size(name):
    """The 2*10^6 x 25 workloads at their K. The stored initial centres of
    these workloads are the oracle's (a CPU test checks that); K = 16 is also
    recomputed by the oracle here."""
    w = workloads.get(name)
    X, _, stored, _ = workloads.load(name)
    _say(f"[init] {name} n={w.n} M={w.M} K={w.K}")
    Xd = torch.from_numpy(X).to(DEV)
    idx, C = km.kmeans_init_farthest(Xd, w.K)
    torch.cuda.synchronize()
    idx = idx.cpu().numpy()
    assert np.array_equal(idx, stored)
    assert np.array_equal(C.cpu().numpy().view(np.uint32), X[stored].view(np.uint32))
    if w.K <= 16:
        assert np.array_equal(idx, oracle.init_farthest(X, w.K))


@pytest.mark.parametrize("n,M,K,seeds,kind", [(1000, 3, 10, (999, 0), "uniform"),
                                              (70_001, 25, 16, (5, 5, 70_000), "dups"),
                                              (4097, 7, 33, (17,), "blobs"),
                                              (64, 2, 64, (63, 1, 2, 3), "uniform"),
                                              # as many seeds as centres: the last,
                                              # one-workgroup launch takes a seed
                                              (500, 4, 6, (7, 3, 499, 0, 3, 250), "uniform"),
                                              (40, 3, 40, tuple(range(39, -1, -1)), "blobs")])
def test_init_from_seeds_parity(n, M, K, seeds, kind):
    X = _case(n, M, kind, seed=n + K)
    _say(f"[init from seeds] n={n} M={M} K={K} seeds={seeds}")
    s = torch.tensor(seeds, dtype=torch.int32, device=DEV)
    idx, C = km.kmeans_init_farthest(torch.from_numpy(X).to(DEV), K, seeds=s)
    torch.cuda.synchronize()
    want = oracle.init_farthest_from(X, K, list(seeds))
    assert np.array_equal(idx.cpu().numpy(), want)
    assert np.array_equal(C.cpu().numpy().view(np.uint32), X[want].view(np.uint32))


@pytest.mark.parametrize("seeds", [(5, 1000), (-1,), (3, 7, 2**31 - 1)])
def test_init_from_seeds_outside_the_set_are_refused(seeds):
    # the oracle refuses them too; nothing is written
    X = _case(1000, 3, "uniform", seed=4)
    Xd = torch.from_numpy(X).to(DEV)
    idx = torch.full((8,), -5, dtype=torch.int32, device=DEV)
    C = torch.full((8, 3), 7.0, dtype=torch.float32, device=DEV)
    with pytest.raises(km.KmeansError) as e:
        km.kmeans_init_farthest(Xd, 8, seeds=torch.tensor(seeds, dtype=torch.int32, device=DEV),
                                out=(idx, C))
    assert e.value.code == km.KMEANS_EINVAL
    assert (idx == -5).all() and (C == 7.0).all()
    with pytest.raises(ValueError):
        oracle.init_farthest_from(X, 8, list(seeds))


@pytest.mark.parametrize("n,M,K", [(20_000, 25, 16), (5_000, 3, 40)])
def test_init_from_the_diameter_on_the_device(n, M, K):
    """Algorithm 2 steps 1 and 3 composed on the device: the diameter's pair,
    left in device memory by kmeans_diameter, seeds the traversal."""
    X = _case(n, M, "blobs", seed=n)
    Xd = torch.from_numpy(X).to(DEV)
    _, pair, _ = km.kmeans_diameter(Xd)
    idx, _ = km.kmeans_init_farthest(Xd, K, seeds=pair)
    torch.cuda.synchronize()
    _, k, l = oracle.diameter(X)
    assert np.array_equal(idx.cpu().numpy(), oracle.init_farthest_from(X, K, [k, l]))
