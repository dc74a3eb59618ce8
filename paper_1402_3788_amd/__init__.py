"""MI355X (gfx950) Lloyd-iteration library: Python binding.

Thin ctypes marshalling over libkmeans_mi355x.so (C ABI in include/kmeans.h).
Tensors are PyTorch device tensors; every step of the computation runs in the
library's HIP kernels. Importing this module fails loudly if the library has
not been built (python paper_1402_3788_amd/build.py).

Entry points (same names as the C ABI):
    kmeans_assign(X, centers, with_min_d2=False, path=None, metric="l2") -> labels [, min_d2]
    kmeans_update(X, labels, K, prev_centers, out=None) -> (centers, counts)
    kmeans_run(X, K, init_centers, max_iter, fixed_iters=False, path=None,
               timing=False, metric="l2") -> (labels, centers, counts, iterations[, timing])
    kmeans_init_farthest(X, K, ws=None) -> (init_idx, centers)
    kmeans_centroid(X, ws=None) -> centroid
    kmeans_diameter(X, ws=None) -> (d2, pair, centroid)
    kmeans_run_noalloc(X, K, init_centers, max_iter, out, ...) -> iterations
    kmeans_workspace_bytes(n, M, K, flags=0), kmeans_init_workspace_bytes(n, M, K),
    kmeans_strerror(code)
"""
from __future__ import annotations

import ctypes
import os

import torch  # loads the HIP runtime this library binds to

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkmeans_mi355x.so")

KMEANS_OK = 0
KMEANS_EINVAL = -1
KMEANS_EUNSUPPORTED = -2
KMEANS_EWORKSPACE = -3
KMEANS_EHIP = -4

KMEANS_FIXED_ITERS = 1 << 0
KMEANS_PATH_DIRECT = 1 << 1
KMEANS_PATH_MFMA = 1 << 2
KMEANS_PATH_TILES = 1 << 3
KMEANS_METRIC_L1 = 1 << 4
KMEANS_FORCE_FP64 = 1 << 5

EXPORTED = ("kmeans_workspace_bytes", "kmeans_strerror", "kmeans_assign", "kmeans_update",
            "kmeans_run", "kmeans_init_workspace_bytes", "kmeans_init_farthest",
            "kmeans_init_farthest_from",
            "kmeans_centroid_workspace_bytes", "kmeans_centroid",
            "kmeans_diameter_workspace_bytes", "kmeans_diameter", "kmeans_run_noalloc")


class KmeansTiming(ctypes.Structure):
    _fields_ = [("step_ms", ctypes.c_double), ("assign_ms", ctypes.c_double),
                ("step_launches", ctypes.c_int32), ("assign_samples", ctypes.c_int32),
                ("sample_every", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class KmeansError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn}: {strerror(code)} ({code})")
        self.code = code


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_1402_3788_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    p, i64, i32, u32, sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32,
                            ctypes.c_size_t)
    lib.kmeans_workspace_bytes.argtypes = [i64, i32, i32, u32]
    lib.kmeans_workspace_bytes.restype = sz
    lib.kmeans_strerror.argtypes = [ctypes.c_int]
    lib.kmeans_strerror.restype = ctypes.c_char_p
    lib.kmeans_assign.argtypes = [p, i64, i32, p, i32, p, p, u32, p]
    lib.kmeans_assign.restype = ctypes.c_int
    lib.kmeans_update.argtypes = [p, i64, i32, p, i32, p, p, p, p, sz, p]
    lib.kmeans_update.restype = ctypes.c_int
    lib.kmeans_run.argtypes = [p, i64, i32, i32, p, i32, u32, p, p, p, p, p, sz, p,
                               ctypes.POINTER(KmeansTiming)]
    lib.kmeans_run.restype = ctypes.c_int
    lib.kmeans_init_workspace_bytes.argtypes = [i64, i32, i32]
    lib.kmeans_init_workspace_bytes.restype = sz
    lib.kmeans_init_farthest.argtypes = [p, i64, i32, i32, p, p, p, sz, p]
    lib.kmeans_init_farthest.restype = ctypes.c_int
    lib.kmeans_init_farthest_from.argtypes = [p, i64, i32, i32, p, i32, p, p, p, sz, p]
    lib.kmeans_init_farthest_from.restype = ctypes.c_int
    lib.kmeans_centroid_workspace_bytes.argtypes = [i64, i32]
    lib.kmeans_centroid_workspace_bytes.restype = sz
    lib.kmeans_centroid.argtypes = [p, i64, i32, p, p, sz, p]
    lib.kmeans_centroid.restype = ctypes.c_int
    lib.kmeans_diameter_workspace_bytes.argtypes = [i64, i32]
    lib.kmeans_diameter_workspace_bytes.restype = sz
    lib.kmeans_diameter.argtypes = [p, i64, i32, p, p, p, p, sz, p]
    lib.kmeans_diameter.restype = ctypes.c_int
    lib.kmeans_run_noalloc.argtypes = [p, i64, i32, i32, p, i32, u32, p, p, p, p, p]
    lib.kmeans_run_noalloc.restype = ctypes.c_int
    return lib


_lib = _load()


def strerror(code: int) -> str:
    return _lib.kmeans_strerror(int(code)).decode()


kmeans_strerror = strerror


def kmeans_workspace_bytes(n: int, M: int, K: int, flags: int = 0) -> int:
    return int(_lib.kmeans_workspace_bytes(int(n), int(M), int(K), int(flags)))


def kmeans_init_workspace_bytes(n: int, M: int, K: int) -> int:
    return int(_lib.kmeans_init_workspace_bytes(int(n), int(M), int(K)))


def _stream_ptr(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check_x(X: torch.Tensor):
    if not (isinstance(X, torch.Tensor) and X.is_cuda and X.dtype == torch.float32
            and X.dim() == 2 and X.is_contiguous()):
        raise ValueError("X must be a contiguous float32 [n, M] tensor on a GPU")


def _dev_ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _metric(metric):
    if metric == "l2":
        return 0
    if metric == "l1":
        return KMEANS_METRIC_L1
    raise ValueError(f"unknown metric {metric!r}")


def _flags(path):
    if path is None or path == "auto":
        return 0
    if path == "direct":
        return KMEANS_PATH_DIRECT
    if path == "mfma":
        return KMEANS_PATH_MFMA
    if path == "tiles":
        return KMEANS_PATH_TILES
    raise ValueError(f"unknown path {path!r}")


def workspace(n: int, M: int, K: int, device, flags: int = 0) -> torch.Tensor:
    nbytes = kmeans_workspace_bytes(n, M, K, flags)
    if nbytes == 0:
        raise KmeansError("kmeans_workspace_bytes", KMEANS_EUNSUPPORTED)
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def kmeans_init_farthest(X: torch.Tensor, K: int, ws: torch.Tensor | None = None, out=None,
                         seeds: torch.Tensor | None = None):
    """Algorithm 1 step 1 as farthest-point traversal from object 0, or from
    `seeds` (int32 device tensor, e.g. the diameter's pair).

    Returns (init_idx int32 [K], centers float32 [K, M]) on X's device;
    asynchronous on the current stream. `out` may supply both tensors."""
    _check_x(X)
    n, M = X.shape
    if out is None:
        idx = torch.empty(int(K), dtype=torch.int32, device=X.device)
        centers = torch.empty((int(K), M), dtype=torch.float32, device=X.device)
    else:
        idx, centers = out
    if ws is None:
        nbytes = kmeans_init_workspace_bytes(n, M, K)
        if nbytes == 0:
            raise KmeansError("kmeans_init_workspace_bytes", KMEANS_EINVAL)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=X.device)
    if seeds is None:
        rc = _lib.kmeans_init_farthest(_dev_ptr(X), n, M, int(K), _dev_ptr(idx),
                                       _dev_ptr(centers), _dev_ptr(ws), ws.numel(),
                                       _stream_ptr(X.device))
    else:
        if not (seeds.is_cuda and seeds.dtype == torch.int32 and seeds.dim() == 1):
            raise ValueError("seeds must be an int32 [S] tensor on a GPU")
        seeds = seeds.contiguous()
        rc = _lib.kmeans_init_farthest_from(_dev_ptr(X), n, M, int(K), _dev_ptr(seeds),
                                            seeds.numel(), _dev_ptr(idx), _dev_ptr(centers),
                                            _dev_ptr(ws), ws.numel(), _stream_ptr(X.device))
    if rc:
        raise KmeansError("kmeans_init_farthest", rc)
    return idx, centers


def kmeans_centroid_workspace_bytes(n: int, M: int) -> int:
    return int(_lib.kmeans_centroid_workspace_bytes(int(n), int(M)))


def kmeans_diameter_workspace_bytes(n: int, M: int) -> int:
    return int(_lib.kmeans_diameter_workspace_bytes(int(n), int(M)))


def _ws(nbytes: int, device, fn: str) -> torch.Tensor:
    if nbytes == 0:
        raise KmeansError(fn, KMEANS_EUNSUPPORTED)
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def kmeans_centroid(X: torch.Tensor, ws: torch.Tensor | None = None):
    """Algorithm 2 step 2: the centre of gravity of all objects (float32 [M])."""
    _check_x(X)
    n, M = X.shape
    c = torch.empty(M, dtype=torch.float32, device=X.device)
    if ws is None:
        ws = _ws(kmeans_centroid_workspace_bytes(n, M), X.device, "kmeans_centroid_workspace_bytes")
    rc = _lib.kmeans_centroid(_dev_ptr(X), n, M, _dev_ptr(c), _dev_ptr(ws), ws.numel(),
                              _stream_ptr(X.device))
    if rc:
        raise KmeansError("kmeans_centroid", rc)
    return c


def kmeans_diameter(X: torch.Tensor, ws: torch.Tensor | None = None):
    """Eq. (3), Algorithm 2 step 1: (d2 float64 [1], pair int32 [2], centroid
    float32 [M]) on X's device; the diameter is sqrt(d2), reached by the
    lexicographically smallest pair. Asynchronous on the current stream."""
    _check_x(X)
    n, M = X.shape
    d2 = torch.empty(1, dtype=torch.float64, device=X.device)
    pair = torch.empty(2, dtype=torch.int32, device=X.device)
    c = torch.empty(M, dtype=torch.float32, device=X.device)
    if ws is None:
        ws = _ws(kmeans_diameter_workspace_bytes(n, M), X.device, "kmeans_diameter_workspace_bytes")
    rc = _lib.kmeans_diameter(_dev_ptr(X), n, M, _dev_ptr(d2), _dev_ptr(pair), _dev_ptr(c),
                              _dev_ptr(ws), ws.numel(), _stream_ptr(X.device))
    if rc:
        raise KmeansError("kmeans_diameter", rc)
    return d2, pair, c


def kmeans_assign(X: torch.Tensor, centers: torch.Tensor, with_min_d2: bool = False, path=None,
                  metric: str = "l2", force_fp64: bool = False):
    """Algorithm 1 steps 2/4: labels[i] = nearest centre (lowest index on ties),
    by the squared Euclidean distance of Eq. (2) or, with metric="l1", by the
    city-block distance (min_d2 then holds that distance)."""
    _check_x(X)
    n, M = X.shape
    C = centers.contiguous()
    K = C.shape[0]
    labels = torch.empty(n, dtype=torch.int32, device=X.device)
    d2 = torch.empty(n, dtype=torch.float32, device=X.device) if with_min_d2 else None
    flags = _flags(path) | _metric(metric) | (KMEANS_FORCE_FP64 if force_fp64 else 0)
    rc = _lib.kmeans_assign(_dev_ptr(X), n, M, _dev_ptr(C), K, _dev_ptr(labels), _dev_ptr(d2),
                            flags, _stream_ptr(X.device))
    if rc:
        raise KmeansError("kmeans_assign", rc)
    return (labels, d2) if with_min_d2 else labels


def kmeans_update(X: torch.Tensor, labels: torch.Tensor, K: int, prev_centers: torch.Tensor,
                  out: torch.Tensor | None = None, ws: torch.Tensor | None = None):
    """Eq. (1): centres of gravity of the labelled objects (empty keeps prev)."""
    _check_x(X)
    n, M = X.shape
    prev = prev_centers.contiguous()
    centers = out if out is not None else torch.empty((K, M), dtype=torch.float32, device=X.device)
    counts = torch.empty(K, dtype=torch.int32, device=X.device)
    if ws is None:
        ws = workspace(n, M, K, X.device)
    rc = _lib.kmeans_update(_dev_ptr(X), n, M, _dev_ptr(labels.contiguous()), int(K),
                            _dev_ptr(prev), _dev_ptr(centers), _dev_ptr(counts), _dev_ptr(ws),
                            ws.numel(), _stream_ptr(X.device))
    if rc:
        raise KmeansError("kmeans_update", rc)
    return centers, counts


def kmeans_run(X: torch.Tensor, K: int, init_centers: torch.Tensor, max_iter: int,
               fixed_iters: bool = False, path=None, timing: bool = False,
               out=None, ws: torch.Tensor | None = None, sample_every: int = 0,
               metric: str = "l2", force_fp64: bool = False):
    """Algorithm 1 steps 2-7 from init_centers (synchronous); metric="l1"
    assigns by the city-block distance (the centres stay centres of gravity).

    Returns (labels, centers, counts, iterations), plus a KmeansTiming when
    timing=True (events around the whole call and around the assign launch of
    every sample_every-th iteration; 0 = every 16th). `out` may supply
    (labels, centers, counts) tensors to reuse.
    """
    _check_x(X)
    n, M = X.shape
    init = init_centers.contiguous()
    if out is None:
        labels = torch.empty(n, dtype=torch.int32, device=X.device)
        centers = torch.empty((K, M), dtype=torch.float32, device=X.device)
        counts = torch.empty(K, dtype=torch.int32, device=X.device)
    else:
        labels, centers, counts = out
    flags = (_flags(path) | _metric(metric) | (KMEANS_FIXED_ITERS if fixed_iters else 0)
             | (KMEANS_FORCE_FP64 if force_fp64 else 0))
    if ws is None:
        ws = workspace(n, M, K, X.device, flags)
    iters = ctypes.c_int32(0)
    tm = KmeansTiming() if timing else None
    if tm is not None:
        tm.sample_every = int(sample_every)
    rc = _lib.kmeans_run(_dev_ptr(X), n, M, int(K), _dev_ptr(init), int(max_iter), flags,
                         _dev_ptr(labels), _dev_ptr(centers), _dev_ptr(counts),
                         ctypes.byref(iters), _dev_ptr(ws), ws.numel(), _stream_ptr(X.device),
                         ctypes.byref(tm) if tm is not None else None)
    if rc:
        raise KmeansError("kmeans_run", rc)
    res = (labels, centers, counts, int(iters.value))
    return res + (tm,) if timing else res


NOALLOC_MAX_WORKSPACE = 16 << 20      # KMEANS_NOALLOC_MAX_WORKSPACE


def kmeans_run_noalloc(X: torch.Tensor, K: int, init_centers: torch.Tensor, max_iter: int,
                       out, fixed_iters: bool = False, path=None, metric: str = "l2",
                       force_fp64: bool = False) -> int:
    """kmeans_run on the library's static per-GPU workspace (no allocation in
    the call): `out` = (labels, centers, counts) tensors to fill. Returns the
    iteration count."""
    _check_x(X)
    n, M = X.shape
    init = init_centers.contiguous()
    labels, centers, counts = out
    flags = (_flags(path) | _metric(metric) | (KMEANS_FIXED_ITERS if fixed_iters else 0)
             | (KMEANS_FORCE_FP64 if force_fp64 else 0))
    iters = ctypes.c_int32(0)
    rc = _lib.kmeans_run_noalloc(_dev_ptr(X), n, M, int(K), _dev_ptr(init), int(max_iter), flags,
                                 _dev_ptr(labels), _dev_ptr(centers), _dev_ptr(counts),
                                 ctypes.byref(iters), _stream_ptr(X.device))
    if rc:
        raise KmeansError("kmeans_run_noalloc", rc)
    return int(iters.value)


def ctl_fallbacks(ws: torch.Tensor) -> int:
    """Objects re-decided in fp64 during the last kmeans_run that used `ws`
    (read from the control block at the start of the workspace)."""
    return int(ws[12:16].view(torch.int32).item())


def ctl_reruns(ws: torch.Tensor) -> int:
    """64-object tiles of the tile kernel whose split-precision scores left a
    call too close, recomputed with fp32 products, during the last kmeans_run
    that used `ws` (read from the control block)."""
    return int(ws[16:20].view(torch.int32).item())
