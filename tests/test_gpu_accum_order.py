"""The order of the fp64 additions that form the sums of Eq. (1) on the GPU.

The centres must be bitwise reproducible (the congruence test of Algorithm 1
steps 6-7 compares them bit for bit), so every fp64 addition has to happen in
an order fixed by the problem shape. Three accumulation forms let several
lanes of one LDS fp64 add hit the same address -- in the small-K kernel with
four 16-centre blocks (33 <= K <= 64) the one slab per wave that the two
objects of a step share, in the 64-object-tile kernel (larger K, or more than
32 features) a slab shared the same way and the workgroup slab that the waves
add into in turn, one lane per object -- and so rely on the LDS applying those
lanes in ascending lane order. (With one or two blocks the small-K kernel adds
the halves of a tile to two slabs and never lets two lanes of one add meet.)
These tests check that property on order-sensitive data instead of assuming
it.

With n = 64 objects the launch is one wave of one workgroup with one tile.
The forms whose adds can collide then form a cluster's sums in ascending
object order -- the order the oracle's Eq. (1) uses -- exactly when the LDS
applies the lanes of an add in ascending order; the other forms add into
several slabs with no collision (objects of an index class per slab, or the
two halves of the tile) and the slabs in order. Each feature of the 64 objects
holds +2^40 or
-2^40 in the first object, its negation in the last, and values in [-1, 1]
in between: every small value meets a partial sum of magnitude 2^40 (spacing
2^-12) and loses its low bits, so the fp64 sum, and after division the fp32
centre, depends on the order (the CPU test below shows that the reverse order,
or the two objects of every step taken upper half first, changes it for most
features).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1402_3788_amd as km

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None


def order_sensitive(M: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    X = rng.uniform(-1.0, 1.0, (64, M)).astype(np.float32)
    big = (rng.choice([-1.0, 1.0], M) * 2.0 ** 40).astype(np.float32)
    X[0] = big
    X[63] = -big
    return X


def centre(values) -> np.float32:
    """fp32 of the fp64 mean, the values added in the given order."""
    s = 0.0
    for v in values:
        s = s + float(v)
    return np.float32(s / len(values))


def test_construction_is_order_sensitive():
    reversed_ = pairs = 0
    total = 0
    for seed in range(20):
        X = order_sensitive(25, seed)
        for j in range(25):
            col = X[:, j]
            ref = centre(col)
            total += 1
            reversed_ += centre(col[::-1]) != ref
            # the two halves of every pair of objects swapped (objects 2s+1
            # before 2s), as the shared-slab form would add them if the LDS
            # took the upper half-wave first
            pairs += centre(col.reshape(32, 2)[:, ::-1].ravel()) != ref
    # every alternative order is caught on most features
    assert reversed_ > 0.8 * total and pairs > 0.8 * total
    # and the oracle's Eq. (1) adds in ascending object order
    X = order_sensitive(4, 99)
    C, cnt = oracle.update(X, np.zeros(64, np.int32), 2, np.ones((2, 4), np.float32))
    assert cnt[0] == 64 and all(C[0, j] == centre(X[:, j]) for j in range(4))


def slab_orders():
    """Addition orders the code fixes for one tile of 64 objects: slab lists
    (objects in ascending order within a slab, the slabs added in order)."""
    obj = np.arange(64)
    orders = {"ascending": [obj]}
    for P in (2, 4, 8, 16, 32):
        orders[f"interleaved{P}"] = [obj[obj % P == h] for h in range(P)]
    orders["halves"] = [obj[:32], obj[32:]]
    return orders


def expected_centres(X, labels, K, prev, slabs):
    """Eq. (1) with each cluster's sum formed slab by slab (fp64, in order)."""
    C = prev.copy()
    for k in np.unique(labels):
        members = [np.array([i for i in sl if labels[i] == k], int) for sl in slabs]
        count = sum(len(m) for m in members)
        for j in range(X.shape[1]):
            tot = 0.0
            for m in members:
                part = 0.0
                for i in m:
                    part = part + float(X[i, j])
                tot = tot + part
            C[k, j] = np.float32(tot / count)
    return C


# Shapes span both forms of the small-K kernel and every accumulation form of
# the tile kernel (which one a shape takes depends on what fits in LDS:
# per-wave slabs for small K*M, one shared slab per wave, or the workgroup
# slab for large K*M). For the 25-feature shapes of the named workloads the
# form is known: K = 16 adds the halves of a tile to two slabs, K = 64 (small-K
# kernel, four blocks) shares one slab between the two objects of a step in
# ascending object order, K = 256 adds into the workgroup slab with one lane
# per object; the last two must give the ascending order.
SHAPES = [(16, 25, "halves"), (24, 25, "halves"), (48, 25, "ascending"), (64, 25, "ascending"),
          (100, 25, None), (256, 25, "ascending"), (1024, 16, None), (512, 32, None),
          (200, 64, None)]


@pytest.mark.gpu
@pytest.mark.parametrize("K,M,want", SHAPES)
def test_same_address_adds_follow_lane_order(K, M, want):
    """On every shape the centres equal those of one fixed slab order, the
    same for every seed and labelling; an LDS that applied the lanes of an add
    in another order would match none of them."""
    print(f"[order] K={K} M={M}", flush=True)
    prev = np.full((K, M), 3.0, np.float32)
    pg = torch.from_numpy(prev).to(DEV)
    orders = slab_orders()
    matched = None
    for seed in range(12):
        X = order_sensitive(M, 1000 * K + seed)
        # all 64 objects in one cluster (every lane of an add on one row), or
        # two clusters in alternation (the two objects of a step differ)
        for labels in (np.zeros(64, np.int32), (np.arange(64) % 2).astype(np.int32)):
            C, cnt = km.kmeans_update(torch.from_numpy(X).to(DEV),
                                      torch.from_numpy(labels).to(DEV), K, pg)
            assert np.array_equal(cnt.cpu().numpy(), oracle.update(X, labels, K, prev)[1])
            got = C.cpu().numpy().view(np.uint32)
            names = [nm for nm, sl in orders.items()
                     if np.array_equal(got, expected_centres(X, labels, K, prev, sl).view(np.uint32))]
            assert names, f"seed {seed}: centres match no fixed addition order"
            matched = set(names) if matched is None else matched & set(names)
            assert matched, "the addition order changed between calls"
    print(f"[order] K={K} M={M}: sums formed in the order {sorted(matched)}", flush=True)
    if want is not None:
        assert want in matched
    if "ascending" in matched:
        # the oracle's own order: bit-identical centres
        X = order_sensitive(M, 7)
        lab = np.zeros(64, np.int32)
        C, _ = km.kmeans_update(torch.from_numpy(X).to(DEV), torch.from_numpy(lab).to(DEV), K, pg)
        assert np.array_equal(C.cpu().numpy().view(np.uint32),
                              oracle.update(X, lab, K, prev)[0].view(np.uint32))


@pytest.mark.gpu
@pytest.mark.parametrize("K,M", [(16, 25), (64, 25), (256, 25)])
def test_skewed_clusters_reproducible(K, M):
    """Zipf-sized clusters (many lanes of a wave in one cluster) and values
    spread over 2^-30 .. 2^30 with random signs, so that a different addition
    order would almost surely change some sum: repeated updates over many
    tiles and workgroups are bitwise identical, and within the contract's
    tolerance of the oracle."""
    print(f"[reproducible] K={K} M={M}", flush=True)
    rng = np.random.default_rng(K)
    n = 300_000
    X = (rng.choice([-1.0, 1.0], (n, M)) * 2.0 ** rng.uniform(-30, 30, (n, M))).astype(np.float32)
    p = 1.0 / np.arange(1, K + 1) ** 1.2
    labels = rng.choice(K, n, p=p / p.sum()).astype(np.int32)
    prev = np.zeros((K, M), np.float32)
    Xg, lg, pg = (torch.from_numpy(a).to(DEV) for a in (X, labels, prev))
    runs = [km.kmeans_update(Xg, lg, K, pg) for _ in range(3)]
    for C, cnt in runs[1:]:
        assert torch.equal(C.view(torch.int32), runs[0][0].view(torch.int32))
        assert torch.equal(cnt, runs[0][1])
    oC, ocnt = oracle.update(X, labels, K, prev)
    assert np.array_equal(runs[0][1].cpu().numpy(), ocnt)
    C = runs[0][0].cpu().numpy().astype(np.float64)
    scale = np.maximum(np.abs(oC).max(axis=1, keepdims=True), 1e-30)
    assert (np.abs(C - oC) <= 1e-5 * scale).all()


# The assign + accumulate launch of the small-K kernel (K <= 64, M <= 32)
# forms its sums the way the update launch does: with one or two 16-centre
# blocks the halves of a tile go to two slabs (no two lanes of one add meet),
# with four blocks the two objects of a step share one slab, in ascending
# object order only if the LDS applies the lanes of an add in ascending lane
# order. Checked through kmeans_run, whose labels come from the same launch.
RUN_SHAPES = [(16, 25, "halves"), (12, 7, "halves"), (16, 32, "halves"),
              (24, 25, "halves"), (32, 16, "halves"), (48, 25, "ascending"),
              (64, 25, "ascending"), (64, 32, "ascending")]


def labelled_tile(M: int, seed: int, alternate: bool):
    """64 order-sensitive objects whose nearest initial centre is 0 for all
    (alternate=False) or 0 for even and 1 for odd objects: feature 0 stays in
    [-1, 1] (+10^6 for the odd objects when alternating; the squared distances
    to centres 0 and 1 then differ by about 10^12, far above the fp64 spacing
    at the objects' norms), the +-2^40 values sit in the other features of
    the first and last object (and, when alternating, of objects 1 and 62)."""
    X = order_sensitive(M, seed)
    X[0, 0], X[63, 0] = 0.5, -0.5
    if alternate:
        # each cluster gets a +2^40 and a -2^40 object, so its sums cancel to
        # values whose low bits depend on the order
        X[1, 1:], X[62, 1:] = X[0, 1:], X[63, 1:]
        X[1::2, 0] += 1.0e6
    return X


def far_centres(K: int, M: int) -> np.ndarray:
    C = np.zeros((K, M), np.float32)
    C[1, 0] = 1.0e6
    for k in range(2, K):
        C[k, 0] = -1e15 * k           # never the nearest
    return C


@pytest.mark.gpu
@pytest.mark.parametrize("K,M,want", RUN_SHAPES)
def test_assign_accumulate_follows_lane_order(K, M, want):
    """One fixed-count iteration of kmeans_run (assignment and the sums of
    Eq. (1) in one launch) on a one-tile problem: the new centres equal those of
    the addition order the code fixes, on every seed and labelling."""
    print(f"[order-run] K={K} M={M}", flush=True)
    init = far_centres(K, M)
    orders = slab_orders()
    for seed in range(8):
        for alternate in (False, True):
            X = labelled_tile(M, 5000 * K + 10 * M + seed, alternate)
            labels = (np.arange(64) % 2 if alternate else np.zeros(64)).astype(np.int32)
            assert np.array_equal(oracle.assign(X, init), labels)
            lab, C, cnt, it = km.kmeans_run(torch.from_numpy(X).to(DEV), K,
                                            torch.from_numpy(init).to(DEV), 1, fixed_iters=True)
            assert it == 1 and np.array_equal(lab.cpu().numpy(), labels)
            assert np.array_equal(cnt.cpu().numpy(), np.bincount(labels, minlength=K))
            got = C.cpu().numpy().view(np.uint32)
            want_c = expected_centres(X, labels, K, init, orders[want]).view(np.uint32)
            other = [nm for nm, sl in orders.items()
                     if np.array_equal(got, expected_centres(X, labels, K, init, sl).view(np.uint32))]
            assert np.array_equal(got, want_c), f"seed {seed}: centres match {other}, not {want}"
    print(f"[order-run] K={K} M={M}: sums formed in the order {want}", flush=True)
