"""ctypes shim over the plain-C CPU oracle (kmeans_oracle.c).

TEST INFRASTRUCTURE ONLY: the oracle is the slow, obviously correct statement
of Algorithm 1's Lloyd iteration (assign by Eq. (2), centres of gravity by
Eq. (1), stop on congruent centres) and of its step 1 (farthest-point initial
centres, and Algorithm 2's steps 1-2: diameter of Eq. (3) and the centre of
gravity of the whole set) that the GPU library is checked against.
Only the tests, the smoke check and the benchmark's CPU-baseline leg use it;
the GPU library never imports, links or calls it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "kmeans_oracle.c")
LIB = os.path.join(_HERE, "libkmeans_oracle.so")
CFLAGS = ["-std=c99", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]
# the multi-threaded CPU regime (Algorithm 3), a baseline checked against the oracle
ALG3_SRC = os.path.join(_HERE, "kmeans_alg3.c")
ALG3_LIB = os.path.join(_HERE, "libkmeans_alg3.so")
ALG3_CFLAGS = ["-std=c99", "-O3", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
               "-shared"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fused multiply-add, no fast-math), and
    the Algorithm 3 baseline beside it."""
    for src, lib, flags in ((SRC, LIB, CFLAGS), (ALG3_SRC, ALG3_LIB, ALG3_CFLAGS)):
        if force or not os.path.exists(lib):
            tmp = lib + ".tmp"
            subprocess.check_call(["gcc", *flags, "-o", tmp, src, "-lm"])
            os.replace(tmp, lib)
    return LIB


def _bind(path: str):
    lib = ctypes.CDLL(path)
    p = ctypes.c_void_p
    i64, i32 = ctypes.c_int64, ctypes.c_int32
    lib.oracle_assign.argtypes = [p, i64, i32, p, i32, p, p, p]
    lib.oracle_assign.restype = ctypes.c_int
    lib.oracle_update.argtypes = [p, i64, i32, p, i32, p, p, p]
    lib.oracle_update.restype = ctypes.c_int
    lib.oracle_run.argtypes = [p, i64, i32, i32, p, i32, i32, p, p, p, p, p, p]
    lib.oracle_run.restype = ctypes.c_int
    lib.oracle_assign_l1.argtypes = [p, i64, i32, p, i32, p, p, p]
    lib.oracle_assign_l1.restype = ctypes.c_int
    lib.oracle_run_l1.argtypes = [p, i64, i32, i32, p, i32, i32, p, p, p, p, p, p]
    lib.oracle_run_l1.restype = ctypes.c_int
    lib.oracle_sse.argtypes = [p, i64, i32, p, p, i32]
    lib.oracle_sse.restype = ctypes.c_double
    lib.oracle_init_farthest.argtypes = [p, i64, i32, i32, p]
    lib.oracle_init_farthest.restype = ctypes.c_int
    lib.oracle_init_farthest_from.argtypes = [p, i64, i32, i32, p, i32, p]
    lib.oracle_init_farthest_from.restype = ctypes.c_int
    lib.oracle_centroid.argtypes = [p, i64, i32, p]
    lib.oracle_centroid.restype = ctypes.c_int
    lib.oracle_diameter.argtypes = [p, i64, i32, p, p, p]
    lib.oracle_diameter.restype = ctypes.c_int
    return lib


_default = None


def _load():
    global _default
    if _default is None:
        # KMEANS_ORACLE_LIB points the shim at another build of the oracle; the
        # tests that plant mistakes in a copy of the oracle source use it.
        path = os.environ.get("KMEANS_ORACLE_LIB")
        if not path:
            path = LIB
            if not os.path.exists(path):
                build(force=False)
        _default = _bind(path)
    return _default


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    if a.ndim != 2:
        raise ValueError("expected a 2-D array")
    return a


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def _metric_fn(metric: str, l2_name: str, l1_name: str):
    if metric == "l2":
        return getattr(_load(), l2_name)
    if metric == "l1":
        return getattr(_load(), l1_name)
    raise ValueError(f"unknown metric {metric!r}")


def assign(X, C, with_dist: bool = False, metric: str = "l2"):
    """Algorithm 1 steps 2/4: nearest centre per object (lowest index on ties).

    metric "l2": squared Euclidean distance (Eq. (2)); "l1": city-block
    distance. Returns labels (int32 [n]); with_dist also returns the best and
    second-best distances (fp64 [n]); second-best is +inf when K == 1.
    """
    X, C = _f32(X), _f32(C)
    n, M = X.shape
    K = C.shape[0]
    if C.shape[1] != M:
        raise ValueError("feature count mismatch")
    labels = np.empty(n, np.int32)
    d1 = np.empty(n, np.float64) if with_dist else None
    d2 = np.empty(n, np.float64) if with_dist else None
    fn = _metric_fn(metric, "oracle_assign", "oracle_assign_l1")
    rc = fn(_ptr(X), n, M, _ptr(C), K, _ptr(labels), _ptr(d1), _ptr(d2))
    if rc:
        raise ValueError(f"oracle_assign failed ({rc})")
    return (labels, d1, d2) if with_dist else labels


def update(X, labels, K: int, prev):
    """Eq. (1): centres of gravity of the labelled objects; empty clusters keep
    prev. Returns (centers fp32 [K,M], counts int32 [K])."""
    X, prev = _f32(X), _f32(prev)
    n, M = X.shape
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    if labels.shape != (n,) or prev.shape != (K, M):
        raise ValueError("shape mismatch")
    centers = np.empty((K, M), np.float32)
    counts = np.empty(K, np.int32)
    rc = _load().oracle_update(_ptr(X), n, M, _ptr(labels), K, _ptr(prev),
                               _ptr(centers), _ptr(counts))
    if rc:
        raise ValueError(f"oracle_update failed ({rc})")
    return centers, counts


def run(X, K: int, init, max_iter: int, fixed: bool = False, with_dist: bool = False,
        metric: str = "l2"):
    """Algorithm 1 steps 2-7 from the given initial centres (assignment by
    the metric: "l2" as Eq. (2), or "l1").

    Returns (labels, centers, counts, iterations) and, with with_dist, the last
    assignment's best / second-best squared distances.
    """
    X, init = _f32(X), _f32(init)
    n, M = X.shape
    if init.shape != (K, M):
        raise ValueError("init shape mismatch")
    labels = np.empty(n, np.int32)
    centers = np.empty((K, M), np.float32)
    counts = np.empty(K, np.int32)
    iters = ctypes.c_int32(0)
    d1 = np.empty(n, np.float64) if with_dist else None
    d2 = np.empty(n, np.float64) if with_dist else None
    fn = _metric_fn(metric, "oracle_run", "oracle_run_l1")
    rc = fn(_ptr(X), n, M, K, _ptr(init), int(max_iter), int(bool(fixed)),
            _ptr(labels), _ptr(centers), _ptr(counts),
            ctypes.byref(iters), _ptr(d1), _ptr(d2))
    if rc:
        raise ValueError(f"oracle_run failed ({rc})")
    out = (labels, centers, counts, int(iters.value))
    return out + (d1, d2) if with_dist else out


def sse(X, labels, C) -> float:
    """Objective: sum of squared distances of objects to their centres (fp64)."""
    X, C = _f32(X), _f32(C)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    return float(_load().oracle_sse(_ptr(X), X.shape[0], X.shape[1], _ptr(labels),
                                    _ptr(C), C.shape[0]))


def init_farthest(X, K: int):
    """Algorithm 1 step 1, read as farthest-point traversal from object 0:
    idx[0] = 0, idx[m] = the not-yet-chosen object whose smallest squared
    distance to the chosen ones is largest (lowest index on ties).
    Returns idx (int32 [K]); the initial centres are X[idx]. Needs K <= n."""
    X = _f32(X)
    n, M = X.shape
    idx = np.empty(int(K), np.int32)
    rc = _load().oracle_init_farthest(_ptr(X), n, M, int(K), _ptr(idx))
    if rc:
        raise ValueError(f"oracle_init_farthest failed ({rc})")
    return idx


def init_farthest_from(X, K: int, seeds):
    """Farthest-point traversal from the given seed objects: idx[:S] = seeds,
    then each next object is the not-yet-chosen one farthest (smallest squared
    distance largest, lowest index on ties) from those chosen. Returns idx
    (int32 [K]). Needs 1 <= S <= K <= n and seeds in [0, n)."""
    X = _f32(X)
    n, M = X.shape
    seeds = np.ascontiguousarray(seeds, dtype=np.int32)
    idx = np.empty(int(K), np.int32)
    rc = _load().oracle_init_farthest_from(_ptr(X), n, M, int(K), _ptr(seeds), len(seeds),
                                           _ptr(idx))
    if rc:
        raise ValueError(f"oracle_init_farthest_from failed ({rc})")
    return idx


def centroid(X):
    """Centre of gravity of the whole set (Algorithm 2 step 2): fp32 of the
    fp64 mean, objects summed in ascending order."""
    X = _f32(X)
    n, M = X.shape
    c = np.empty(M, np.float32)
    rc = _load().oracle_centroid(_ptr(X), n, M, _ptr(c))
    if rc:
        raise ValueError(f"oracle_centroid failed ({rc})")
    return c


def diameter(X):
    """Eq. (3), squared (Algorithm 2 step 1): (d2, k, l) with d2 the largest
    squared distance over pairs k < l (fp64) and (k, l) the lexicographically
    smallest pair reaching it; (0.0, 0, 0) when n == 1; (nan, -1, -1) when a
    coordinate is NaN or infinite (the diameter is not defined). O(n^2 M)."""
    X = _f32(X)
    n, M = X.shape
    d2 = ctypes.c_double(0.0)
    k, l = ctypes.c_int32(0), ctypes.c_int32(0)
    rc = _load().oracle_diameter(_ptr(X), n, M, ctypes.byref(d2), ctypes.byref(k),
                                 ctypes.byref(l))
    if rc:
        raise ValueError(f"oracle_diameter failed ({rc})")
    return float(d2.value), int(k.value), int(l.value)


_alg3 = None


def _load_alg3():
    global _alg3
    if _alg3 is None:
        if not os.path.exists(ALG3_LIB):
            build(force=False)
        lib = ctypes.CDLL(ALG3_LIB)
        p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.alg3_run.argtypes = [p, i64, i32, i32, p, i32, i32, i32, p, p, p, p, p]
        lib.alg3_run.restype = ctypes.c_int
        _alg3 = lib
    return _alg3


def alg3_run(X, K: int, init, max_iter: int, fixed: bool = False, threads: int = 0):
    """The multi-threaded CPU regime (Algorithm 3, steps 4-9) from the given
    initial centres: each of `threads` threads (0 = all OpenMP threads)
    assigns and sums its 1/N of the objects. Returns (labels, centers, counts,
    iterations, threads used)."""
    X, init = _f32(X), _f32(init)
    n, M = X.shape
    if init.shape != (K, M):
        raise ValueError("init shape mismatch")
    labels = np.empty(n, np.int32)
    centers = np.empty((K, M), np.float32)
    counts = np.empty(K, np.int32)
    iters, used = ctypes.c_int32(0), ctypes.c_int32(0)
    rc = _load_alg3().alg3_run(_ptr(X), n, M, int(K), _ptr(init), int(max_iter),
                               int(bool(fixed)), int(threads), _ptr(labels), _ptr(centers),
                               _ptr(counts), ctypes.byref(iters), ctypes.byref(used))
    if rc:
        raise ValueError(f"alg3_run failed ({rc})")
    return labels, centers, counts, int(iters.value), int(used.value)


def gap_rel(d1, d2):
    """(d2 - d1) / d2 per object: 0 at an exact tie, 1 when there is no
    competing centre (K == 1); 0 when d2 == 0."""
    d1 = np.asarray(d1, np.float64)
    d2 = np.asarray(d2, np.float64)
    g = np.ones_like(d1)
    fin = np.isfinite(d2)
    pos = fin & (d2 > 0)
    g[pos] = (d2[pos] - d1[pos]) / d2[pos]
    g[fin & (d2 <= 0)] = 0.0
    return g
