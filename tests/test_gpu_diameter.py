"""GPU parity of the diameter of Eq. (3) and the centre of gravity of the whole
set (Algorithm 2 steps 1-2) against the CPU oracle, through the C ABI.

The diameter's pair is an argmax decided by fp64 distances in one fixed
operation order on both sides, so the bar is bit-exact: the same pair and the
same fp64 squared distance. The centre of gravity sums in fp64 in another
fixed order than the oracle, so each coordinate may differ by one unit in the
last fp32 place (it rounds the same fp64 value otherwise). At 2*10^6 objects,
where the O(n^2) oracle cannot run, the result is checked by properties that
hold at any size.
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


def _seq_d2(a, b):
    """fp64 squared distance in the fixed order (features ascending)."""
    d = 0.0
    for x, y in zip(a.astype(np.float64), b.astype(np.float64)):
        e = x - y
        d = d + e * e
    return d


def gpu_diameter(X):
    d2, pair, c = km.kmeans_diameter(torch.from_numpy(np.ascontiguousarray(X)).to(DEV))
    torch.cuda.synchronize()
    return float(d2.item()), tuple(int(v) for v in pair.cpu().numpy()), c.cpu().numpy()


def check_centroid(c, X):
    want = oracle.centroid(X)
    ulp = np.spacing(np.abs(want)).astype(np.float64)
    assert (np.abs(c.astype(np.float64) - want) <= ulp).all()
    return int((c != want).sum())


def _case(n, M, kind, seed, offset=0.0):
    if kind == "same":
        return np.full((n, M), 2.5, np.float32)
    if kind == "corners":
        # the 2^M corners of a cube, shuffled and repeated: every antipodal
        # pair of copies ties exactly at the maximum, across many work items
        rng = np.random.default_rng(seed)
        corners = ((np.arange(2 ** M)[:, None] >> np.arange(M)) & 1).astype(np.float32)
        return np.ascontiguousarray(corners[rng.integers(0, 2 ** M, n)] * 3 - 1.5
                                    + np.float32(offset))
    X, _ = workloads.random_case(n, M, 1, seed, kind)
    return (X + np.float32(offset)).astype(np.float32)


@pytest.mark.parametrize("n,M,kind,offset", [
    (1, 3, "uniform", 0.0), (2, 2, "uniform", 0.0), (7, 3, "same", 0.0), (100, 2, "dups", 0.0),
    (1000, 25, "blobs", 0.0), (5000, 25, "uniform", 0.0), (3000, 64, "blobs", 0.0),
    (4097, 33, "dups", 0.0), (8193, 10, "line", 0.0), (5000, 10, "blobs", 1000.0),
    (2500, 30, "uniform", 0.0), (2500, 31, "uniform", 0.0), (600, 1, "line", 0.0),
    (20_000, 25, "blobs", 0.0), (8192, 4, "uniform", 0.0), (1024, 2, "line", 0.0),
    (24_000, 3, "corners", 0.0), (20_000, 5, "corners", 7.0),
])
def test_diameter_parity(n, M, kind, offset):
    X = _case(n, M, kind, seed=n + M, offset=offset)
    _say(f"[diameter] n={n} M={M} kind={kind} offset={offset}")
    d2, pair, c = gpu_diameter(X)
    od2, k, l = oracle.diameter(X)
    assert pair == (k, l) and d2 == od2, (pair, (k, l), d2, od2)
    check_centroid(c, X)


@pytest.mark.parametrize("n,M", [(1, 1), (999, 7), (200_003, 25), (1_000_000, 64)])
def test_centroid_parity(n, M):
    X = _case(n, M, "blobs", seed=3, offset=-20.0)
    _say(f"[centroid] n={n} M={M}")
    c = km.kmeans_centroid(torch.from_numpy(X).to(DEV))
    torch.cuda.synchronize()
    check_centroid(c.cpu().numpy(), X)


def test_diameter_full_size_properties():
    """The 2*10^6 x 25 workload: the reported value is the pair's own fp64
    distance, each endpoint is a farthest object from the other, no sampled
    pair is farther, and the centre of gravity matches the oracle's."""
    X, _, _, _ = workloads.load("aniso25d-n2m-k16")
    _say("[diameter] aniso25d-n2m-k16 n=2000000 M=25")
    d2, (k, l), c = gpu_diameter(X)
    assert 0 <= k < l < X.shape[0]
    assert d2 == _seq_d2(X[k], X[l])
    X64 = X.astype(np.float64)
    for a, b in ((k, l), (l, k)):
        da = ((X64 - X64[a]) ** 2).sum(1)
        assert da.max() <= d2 * (1 + 1e-12)
        assert da[b] == pytest.approx(d2, rel=1e-12)
    rng = np.random.default_rng(0)
    i, j = rng.integers(0, X.shape[0], (2, 1_000_000))
    assert (((X64[i] - X64[j]) ** 2).sum(1) <= d2 * (1 + 1e-12)).all()
    check_centroid(c, X)


@pytest.mark.gpu
@pytest.mark.parametrize("bad", [float("nan"), float("inf"), float("-inf")])
def test_nonfinite_coordinates_give_no_diameter(bad):
    """A NaN or an infinite coordinate: the diameter is not defined, the GPU
    reports (NaN, -1, -1) as the oracle does, and a farthest-point traversal
    seeded with that pair is refused. Finite data that overflows fp32 squares
    (coordinates near 3e38) still gives the oracle's pair."""
    print(f"[diam-nonfinite] {bad}", flush=True)
    rng = np.random.default_rng(21)
    X = rng.normal(0.0, 1.0, (3000, 25)).astype(np.float32)
    X[1234, 7] = bad
    d2w, kw, lw = oracle.diameter(X)
    assert np.isnan(d2w) and (kw, lw) == (-1, -1)
    Xg = torch.from_numpy(X).to(DEV)
    ws = torch.empty(km.kmeans_diameter_workspace_bytes(*X.shape), dtype=torch.uint8, device=DEV)
    d2, pair, _ = km.kmeans_diameter(Xg, ws=ws)
    assert np.isnan(d2.item()) and pair.cpu().tolist() == [-1, -1]
    with pytest.raises(km.KmeansError):
        km.kmeans_init_farthest(Xg, 4, seeds=pair)
    # the same workspace then serves finite data (the flag is reset per call);
    # squares near 1e77 overflow fp32, so every pair is re-evaluated in fp64
    X[1234, 7] = 0.5
    X[10, 3], X[2999, 3] = 3.0e38, -3.0e38
    d2w, kw, lw = oracle.diameter(X)
    d2, pair, _ = km.kmeans_diameter(torch.from_numpy(X).to(DEV), ws=ws)
    assert pair.cpu().tolist() == [kw, lw] == [10, 2999] and d2.item() == d2w
