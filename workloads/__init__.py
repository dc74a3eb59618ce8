"""Seeded synthetic point sets shaped like the paper's clustering problems.

This module only produces inputs: the object matrix X (n objects, M features,
fp32, row-major), the generator's ground-truth blob labels, and the seeded
initial centres. It holds none of the Lloyd iteration's arithmetic and is
shared by the CPU oracle tests and the GPU path alike.

The paper's data are confidential (section "Similar developments"); it states
only the sizes (up to n = 2*10^6 objects with up to M = 25 features, section
"Introduction"). The named workloads below stand in for those data.

Initial centres (Algorithm 1, step 1, "K objects far away from each other";
the method is left open) are chosen by farthest-point traversal starting from
object 0, in fp64: c_0 = X[0], and c_m is the not-yet-chosen object whose
smallest squared distance to c_0..c_{m-1} is largest (lowest index on ties).
This is an input recipe, identical for both sides, not part of the result
being compared.
"""
from __future__ import annotations

import hashlib
import json
import os
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "get", "generate", "farthest_point_init",
    "zipf_sizes", "equal_sizes", "x_sha256", "load", "random_case", "planted_params",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
INIT_TABLE = os.path.join(_HERE, "init_indices.json")


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    M: int
    K: int
    seed: int
    max_iter: int
    fixed: bool            # run exactly max_iter iterations (no early stop)
    center_lo: float
    center_hi: float
    sigma: float | None    # isotropic sigma; None = per-cluster diagonal sigma
    sizes: str             # "equal" | "dirichlet2" | "zipf1.2+noise"
    notes: str = field(default="", compare=False)


WORKLOADS: dict[str, Workload] = {w.name: w for w in [
    Workload("blobs2d-n10k-k4", 10_000, 2, 4, 0, 50, False, -10.0, 10.0, 0.5,
             "equal", "isotropic blobs, sigma 0.5, equal sizes"),
    Workload("dirichlet10d-n200k-k8", 200_000, 10, 8, 1, 100, False, -20.0, 20.0,
             1.0, "dirichlet2", "isotropic blobs, sigma 1, Dirichlet(2) sizes"),
    Workload("aniso25d-n2m-k16", 2_000_000, 25, 16, 2, 100, False, -50.0, 50.0,
             None, "equal",
             "anisotropic blobs, per-cluster diagonal sigma ~ U[0.5,3]; the "
             "paper's largest size"),
    Workload("blobs25d-n2m-k256", 2_000_000, 25, 256, 3, 30, True, -100.0, 100.0,
             2.0, "equal", "isotropic blobs, sigma 2, 256 clusters, 30 iterations"),
    Workload("zipfnoise25d-n20m-k64", 20_000_000, 25, 64, 4, 30, True, -50.0, 50.0,
             1.5, "zipf1.2+noise",
             "90% blobs with Zipf(1.2) sizes, sigma 1.5, plus 10% uniform noise "
             "over [-60,60]^25; 30 iterations"),
]}

# Short aliases: the five workloads in increasing size order.
ALIASES = {str(i + 1): name for i, name in enumerate(WORKLOADS)}


def get(name: str) -> Workload:
    return WORKLOADS[ALIASES.get(name, name)]


def equal_sizes(n: int, K: int) -> np.ndarray:
    """n split into K near-equal parts; the first n mod K parts get one more."""
    base, rem = divmod(n, K)
    s = np.full(K, base, dtype=np.int64)
    s[:rem] += 1
    return s


def zipf_sizes(total: int, K: int, s: float) -> np.ndarray:
    """Sizes proportional to (k+1)^-s, k < K: floor, then the remaining units go
    to the largest fractional parts (ties to the lower k)."""
    w = (np.arange(1, K + 1, dtype=np.float64)) ** (-s)
    raw = total * w / w.sum()
    base = np.floor(raw).astype(np.int64)
    rem = total - int(base.sum())
    frac = raw - base
    order = sorted(range(K), key=lambda k: (-frac[k], k))
    for k in order[:rem]:
        base[k] += 1
    return base


def planted_params(w: Workload | str):
    """The planted blob centres (K, M) and per-cluster sigma (K, M) of a
    workload: the first draws of generate()'s random stream, replayed."""
    if isinstance(w, str):
        w = get(w)
    rng = np.random.default_rng(w.seed)
    centers = rng.uniform(w.center_lo, w.center_hi, (w.K, w.M))
    if w.sigma is None:
        sigma = rng.uniform(0.5, 3.0, (w.K, w.M))
    else:
        sigma = np.full((w.K, w.M), w.sigma)
    return centers, sigma


def generate(w: Workload | str):
    """Return (X fp32 [n,M] C-contiguous, truth int32 [n]) for a workload.

    numpy default_rng(seed) draws, in this order: the planted centres; the
    per-cluster diagonal sigma (anisotropic workload only); the cluster sizes
    (Dirichlet workload only); the blob points cluster by cluster; the uniform
    background noise (noisy workload only); a permutation of all points.
    Noise points carry truth label -1.
    """
    if isinstance(w, str):
        w = get(w)
    rng = np.random.default_rng(w.seed)
    n, M, K = w.n, w.M, w.K
    centers = rng.uniform(w.center_lo, w.center_hi, (K, M))
    if w.sigma is None:
        sigma = rng.uniform(0.5, 3.0, (K, M))
    else:
        sigma = np.full((K, M), w.sigma)
    n_noise = 0
    if w.sizes == "equal":
        sizes = equal_sizes(n, K)
    elif w.sizes == "dirichlet2":
        sizes = rng.multinomial(n, rng.dirichlet([2.0] * K)).astype(np.int64)
    elif w.sizes == "zipf1.2+noise":
        n_noise = n // 10
        sizes = zipf_sizes(n - n_noise, K, 1.2)
    else:
        raise ValueError(w.sizes)
    X = np.empty((n, M), dtype=np.float64)
    truth = np.empty(n, dtype=np.int32)
    pos = 0
    for k in range(K):
        sk = int(sizes[k])
        blk = X[pos:pos + sk]
        rng.standard_normal(out=blk)       # same draws as standard_normal((sk, M))
        blk *= sigma[k]                    # centre + sigma * z, element by element
        blk += centers[k]
        truth[pos:pos + sk] = k
        pos += sk
    if n_noise:
        X[pos:pos + n_noise] = rng.uniform(-60.0, 60.0, (n_noise, M))
        truth[pos:pos + n_noise] = -1
        pos += n_noise
    assert pos == n
    perm = rng.permutation(n)
    Xp = np.empty((n, M), dtype=np.float32)
    step = 1 << 20
    for s in range(0, n, step):
        Xp[s:s + step] = X[perm[s:s + step]]
    del X
    return Xp, truth[perm]


def farthest_point_init(X: np.ndarray, K: int, chunk: int = 1 << 19) -> np.ndarray:
    """Indices of K objects chosen by fp64 farthest-point traversal from object 0.

    c_0 = X[0]; c_m = argmax over not-yet-chosen i of min_{l<m} |X_i - c_l|^2,
    lowest index on ties. Requires K <= n.
    """
    n = X.shape[0]
    if K > n:
        raise ValueError("farthest-point init needs K <= n")
    idx = [0]
    mind = np.full(n, np.inf)
    for _ in range(1, K):
        c = X[idx[-1]].astype(np.float64)
        for s in range(0, n, chunk):
            e = X[s:s + chunk].astype(np.float64)
            e -= c
            np.square(e, out=e)
            d = e.sum(axis=1)
            np.minimum(mind[s:s + chunk], d, out=mind[s:s + chunk])
        mind[idx] = -1.0
        idx.append(int(np.argmax(mind)))
    return np.asarray(idx, dtype=np.int64)


def x_sha256(X: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(X).view(np.uint8)).hexdigest()


def _init_table() -> dict:
    if os.path.exists(INIT_TABLE):
        with open(INIT_TABLE) as f:
            return json.load(f)
    return {}


def load(name: str, verify_hash: bool = True):
    """Generate a named workload and its initial centres.

    Returns (X, truth, init_idx, init_centers). The farthest-point indices of
    the larger workloads are read from init_indices.json (written by
    make_init_table.py) when the generated X has the recorded SHA-256;
    otherwise they are recomputed.
    """
    w = get(name)
    X, truth = generate(w)
    entry = _init_table().get(w.name)
    init_idx = None
    if entry is not None:
        if not verify_hash or entry["sha256_x"] == x_sha256(X):
            init_idx = np.asarray(entry["init"], dtype=np.int64)
    if init_idx is None:
        init_idx = farthest_point_init(X, w.K)
    init = np.ascontiguousarray(X[init_idx])
    return X, truth, init_idx, init


def random_case(n: int, M: int, K: int, seed: int, kind: str = "blobs",
                init: str = "farthest"):
    """Small seeded case for parity and property tests.

    kind: "blobs" (K planted blobs, sigma 1, centres ~ U[-10,10]^M),
          "uniform" (U[-1,1]^M), "dups" (points drawn from a few distinct
          values, so exact distance ties occur), "line" (M = 1 style spread).
    init: "farthest" (farthest-point from object 0, needs K <= n) or
          "random" (K rows drawn with replacement, so duplicate centres and
          empty clusters can occur).
    Returns (X fp32 [n,M], init fp32 [K,M]).
    """
    rng = np.random.default_rng(seed)
    if kind == "blobs":
        c = rng.uniform(-10, 10, (max(K, 1), M))
        lab = rng.integers(0, max(K, 1), n)
        X = c[lab] + rng.standard_normal((n, M))
    elif kind == "uniform":
        X = rng.uniform(-1, 1, (n, M))
    elif kind == "dups":
        vals = rng.integers(-3, 4, (max(2, min(n, 7)), M)).astype(np.float64)
        X = vals[rng.integers(0, vals.shape[0], n)]
    elif kind == "line":
        X = rng.uniform(-100, 100, (n, M))
    else:
        raise ValueError(kind)
    X = np.ascontiguousarray(X.astype(np.float32))
    if init == "farthest":
        idx = farthest_point_init(X, K)
    elif init == "random":
        idx = rng.integers(0, n, K)
    else:
        raise ValueError(init)
    return X, np.ascontiguousarray(X[idx])
