"""The C-ABI library: it loads, exports what include/kmeans.h declares, sizes
its workspace, and rejects bad arguments on the host before touching the GPU.
Runs without a GPU: every call here fails validation before any HIP call."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_1402_3788_amd as km

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kmeans.h")

FAKE = ctypes.c_void_p(0x10000)        # never dereferenced: validation fails first
FAKE_MISALIGNED = ctypes.c_void_p(0x10004)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kmeans_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(km.EXPORTED)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", km.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    syms = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    for name in declared_functions():
        assert name in syms, name
        assert hasattr(km._lib, name)


def test_header_constants_match_binding():
    text = open(HEADER).read()
    for name in ["KMEANS_OK", "KMEANS_EINVAL", "KMEANS_EUNSUPPORTED", "KMEANS_EWORKSPACE",
                 "KMEANS_EHIP"]:
        m = re.search(rf"#define {name}\s+(-?\d+)", text)
        assert int(m.group(1)) == getattr(km, name)
    for name in ["KMEANS_FIXED_ITERS", "KMEANS_PATH_DIRECT", "KMEANS_PATH_MFMA",
                 "KMEANS_PATH_TILES", "KMEANS_METRIC_L1", "KMEANS_FORCE_FP64"]:
        m = re.search(rf"#define {name}\s+\(1u << (\d+)\)", text)
        assert (1 << int(m.group(1))) == getattr(km, name)


def test_strerror_names_every_code():
    for c in [0, -1, -2, -3, -4]:
        assert km.strerror(c) and km.strerror(c) != "unknown status"
    assert km.strerror(-99) == "unknown status"


def test_workspace_bytes():
    assert km.kmeans_workspace_bytes(2_000_000, 25, 16) > 0
    assert km.kmeans_workspace_bytes(0, 25, 16) == 0
    assert km.kmeans_workspace_bytes(10, 65, 16) == 0
    assert km.kmeans_workspace_bytes(10, 25, 1025) == 0
    assert km.kmeans_workspace_bytes(10, 64, 257) == 0          # K*M > 16384
    assert km.kmeans_workspace_bytes(2**31, 4, 4) == 0
    assert km.kmeans_workspace_bytes(10, 4, 4, 1 << 9) == 0     # unknown flag
    assert km.kmeans_workspace_bytes(10**6, 25, 16, km.KMEANS_METRIC_L1) > 0
    assert km.kmeans_workspace_bytes(10, 4, 4, km.KMEANS_METRIC_L1 | km.KMEANS_PATH_MFMA) == 0
    # the all-fp64 decision combines with every path and metric
    for f in (0, km.KMEANS_PATH_DIRECT, km.KMEANS_PATH_MFMA, km.KMEANS_PATH_TILES,
              km.KMEANS_METRIC_L1):
        assert km.kmeans_workspace_bytes(10**5, 25, 16, f | km.KMEANS_FORCE_FP64) == \
            km.kmeans_workspace_bytes(10**5, 25, 16, f)
    # partials grow with K*M; the control block is always there
    assert km.kmeans_workspace_bytes(10**6, 25, 256) > km.kmeans_workspace_bytes(10**6, 25, 16)
    assert km.kmeans_workspace_bytes(1, 1, 1) >= 256


def _assign(X=FAKE, n=100, M=4, C=FAKE, K=3, labels=FAKE, d2=None, flags=0):
    return km._lib.kmeans_assign(X, n, M, C, K, labels, d2, flags, None)


def _update(X=FAKE, n=100, M=4, labels=FAKE, K=3, prev=FAKE, C=FAKE, counts=FAKE, ws=FAKE,
            wsb=None):
    wsb = km.kmeans_workspace_bytes(n, M, K) if wsb is None else wsb
    return km._lib.kmeans_update(X, n, M, labels, K, prev, C, counts, ws, wsb, None)


def _run(X=FAKE, n=100, M=4, K=3, init=FAKE, max_iter=5, flags=0, labels=FAKE, C=FAKE,
         counts=FAKE, iters=None, ws=FAKE, wsb=None):
    it = ctypes.c_int32(0)
    wsb = km.kmeans_workspace_bytes(n, M, K) if wsb is None else wsb
    return km._lib.kmeans_run(X, n, M, K, init, max_iter, flags, labels, C, counts,
                              ctypes.byref(it) if iters is None else iters, ws, wsb, None, None)


@pytest.mark.parametrize("kw,code", [
    (dict(X=None), km.KMEANS_EINVAL), (dict(C=None), km.KMEANS_EINVAL),
    (dict(labels=None), km.KMEANS_EINVAL), (dict(n=0), km.KMEANS_EINVAL),
    (dict(M=0), km.KMEANS_EINVAL), (dict(K=0), km.KMEANS_EINVAL),
    (dict(n=-5), km.KMEANS_EINVAL), (dict(M=65), km.KMEANS_EUNSUPPORTED),
    (dict(K=1025), km.KMEANS_EUNSUPPORTED), (dict(M=64, K=257), km.KMEANS_EUNSUPPORTED),
    (dict(n=2**31), km.KMEANS_EUNSUPPORTED), (dict(X=FAKE_MISALIGNED), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_PATH_DIRECT | km.KMEANS_PATH_MFMA), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_PATH_TILES | km.KMEANS_PATH_MFMA), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_PATH_TILES | km.KMEANS_PATH_DIRECT), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_PATH_TILES, M=16, K=1024), km.KMEANS_EUNSUPPORTED),
    (dict(flags=1 << 7), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_METRIC_L1 | km.KMEANS_PATH_MFMA), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_METRIC_L1 | km.KMEANS_PATH_DIRECT), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_METRIC_L1, M=65), km.KMEANS_EUNSUPPORTED),
])
def test_assign_validation(kw, code):
    assert _assign(**kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(X=None), km.KMEANS_EINVAL), (dict(labels=None), km.KMEANS_EINVAL),
    (dict(prev=None), km.KMEANS_EINVAL), (dict(C=None), km.KMEANS_EINVAL),
    (dict(counts=None), km.KMEANS_EINVAL), (dict(n=0), km.KMEANS_EINVAL),
    (dict(M=65), km.KMEANS_EUNSUPPORTED), (dict(X=FAKE_MISALIGNED), km.KMEANS_EINVAL),
    (dict(ws=None), km.KMEANS_EWORKSPACE), (dict(wsb=0), km.KMEANS_EWORKSPACE),
    (dict(wsb=255), km.KMEANS_EWORKSPACE),
])
def test_update_validation(kw, code):
    assert _update(**kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(X=None), km.KMEANS_EINVAL), (dict(init=None), km.KMEANS_EINVAL),
    (dict(labels=None), km.KMEANS_EINVAL), (dict(C=None), km.KMEANS_EINVAL),
    (dict(counts=None), km.KMEANS_EINVAL), (dict(max_iter=0), km.KMEANS_EINVAL),
    (dict(max_iter=-3), km.KMEANS_EINVAL), (dict(K=0), km.KMEANS_EINVAL),
    (dict(K=2000), km.KMEANS_EUNSUPPORTED), (dict(X=FAKE_MISALIGNED), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_PATH_DIRECT | km.KMEANS_PATH_MFMA), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_PATH_MFMA | km.KMEANS_PATH_TILES), km.KMEANS_EINVAL),
    (dict(flags=km.KMEANS_PATH_TILES, M=16, K=1024, wsb=1 << 30), km.KMEANS_EUNSUPPORTED),
    (dict(flags=1 << 9), km.KMEANS_EINVAL), (dict(ws=None), km.KMEANS_EWORKSPACE),
    (dict(flags=km.KMEANS_METRIC_L1 | km.KMEANS_PATH_TILES), km.KMEANS_EINVAL),
    (dict(wsb=16), km.KMEANS_EWORKSPACE),
])
def test_run_validation(kw, code):
    assert _run(**kw) == code


def test_init_workspace_bytes():
    assert km.kmeans_init_workspace_bytes(2_000_000, 25, 16) >= 2_000_000 * 8
    assert km.kmeans_init_workspace_bytes(10, 2, 11) == 0       # K > n
    assert km.kmeans_init_workspace_bytes(10, 65, 4) == 0
    assert km.kmeans_init_workspace_bytes(0, 2, 1) == 0
    assert km.kmeans_init_workspace_bytes(1, 1, 1) > 0


def _init(X=FAKE, n=100, M=4, K=3, idx=FAKE, C=FAKE, ws=FAKE, wsb=None):
    wsb = km.kmeans_init_workspace_bytes(n, M, K) if wsb is None else wsb
    return km._lib.kmeans_init_farthest(X, n, M, K, idx, C, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(X=None), km.KMEANS_EINVAL), (dict(idx=None), km.KMEANS_EINVAL),
    (dict(C=None), km.KMEANS_EINVAL), (dict(n=0), km.KMEANS_EINVAL),
    (dict(K=0), km.KMEANS_EINVAL), (dict(n=5, K=6), km.KMEANS_EINVAL),
    (dict(M=65), km.KMEANS_EUNSUPPORTED), (dict(K=1025), km.KMEANS_EUNSUPPORTED),
    (dict(X=FAKE_MISALIGNED), km.KMEANS_EINVAL), (dict(ws=None), km.KMEANS_EWORKSPACE),
    (dict(wsb=100 * 8), km.KMEANS_EWORKSPACE),
])
def test_init_validation(kw, code):
    assert _init(**kw) == code


@pytest.mark.parametrize("seeds,nseeds,K,code", [
    (None, 2, 3, km.KMEANS_EINVAL), (FAKE, 0, 3, km.KMEANS_EINVAL), (FAKE, 4, 3, km.KMEANS_EINVAL),
    (FAKE, 2, 101, km.KMEANS_EINVAL),
])
def test_init_from_validation(seeds, nseeds, K, code):
    wsb = km.kmeans_init_workspace_bytes(100, 4, 3)
    assert km._lib.kmeans_init_farthest_from(FAKE, 100, 4, K, seeds, nseeds, FAKE, FAKE, FAKE,
                                             wsb, None) == code


def test_centroid_and_diameter_workspace_bytes():
    assert km.kmeans_centroid_workspace_bytes(2_000_000, 25) > 0
    assert km.kmeans_centroid_workspace_bytes(0, 25) == 0
    assert km.kmeans_centroid_workspace_bytes(10, 65) == 0
    # four bf16 operand arrays of 32 ceil((M+2)/32) values per object (n padded to 16384)
    assert km.kmeans_diameter_workspace_bytes(2_000_000, 25) >= 4 * 2_000_000 * 32 * 2
    assert (km.kmeans_diameter_workspace_bytes(10_000, 40)
            > km.kmeans_diameter_workspace_bytes(10_000, 30))
    assert km.kmeans_diameter_workspace_bytes(1, 1) > 0
    assert km.kmeans_diameter_workspace_bytes(0, 3) == 0
    assert km.kmeans_diameter_workspace_bytes(2**31 - 1, 4) == 0     # too many column chunks


def _centroid(X=FAKE, n=100, M=4, C=FAKE, ws=FAKE, wsb=None):
    wsb = km.kmeans_centroid_workspace_bytes(n, M) if wsb is None else wsb
    return km._lib.kmeans_centroid(X, n, M, C, ws, wsb, None)


def _diameter(X=FAKE, n=100, M=4, d2=FAKE, pair=FAKE, C=FAKE, ws=FAKE, wsb=None):
    wsb = km.kmeans_diameter_workspace_bytes(n, M) if wsb is None else wsb
    return km._lib.kmeans_diameter(X, n, M, d2, pair, C, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(X=None), km.KMEANS_EINVAL), (dict(C=None), km.KMEANS_EINVAL),
    (dict(n=0), km.KMEANS_EINVAL), (dict(M=0), km.KMEANS_EINVAL),
    (dict(M=65), km.KMEANS_EUNSUPPORTED), (dict(X=FAKE_MISALIGNED), km.KMEANS_EINVAL),
    (dict(ws=None), km.KMEANS_EWORKSPACE), (dict(wsb=8), km.KMEANS_EWORKSPACE),
])
def test_centroid_validation(kw, code):
    assert _centroid(**kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(X=None), km.KMEANS_EINVAL), (dict(d2=None), km.KMEANS_EINVAL),
    (dict(pair=None), km.KMEANS_EINVAL), (dict(n=0), km.KMEANS_EINVAL),
    (dict(M=65), km.KMEANS_EUNSUPPORTED), (dict(n=2**31 - 1), km.KMEANS_EUNSUPPORTED),
    (dict(X=FAKE_MISALIGNED), km.KMEANS_EINVAL), (dict(ws=None), km.KMEANS_EWORKSPACE),
    (dict(wsb=4096), km.KMEANS_EWORKSPACE),
])
def test_diameter_validation(kw, code):
    assert _diameter(**kw) == code


def test_plain_c_client(tmp_path):
    """The header compiles as C and a gcc-built client links against the
    library and gets the documented results from the host-side paths."""
    exe = tmp_path / "abi_client"
    subprocess.check_call(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                           os.path.join(ROOT, "tests", "abi_client.c"), "-o", str(exe),
                           "-L", os.path.dirname(km.LIB_PATH), "-lkmeans_mi355x",
                           f"-Wl,-rpath,{os.path.dirname(km.LIB_PATH)}"])
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.count("ok  ") == 18


def test_run_null_iterations_pointer():
    it_null = ctypes.POINTER(ctypes.c_int32)()
    assert _run(iters=it_null) == km.KMEANS_EINVAL


def test_binding_rejects_host_tensors():
    import torch
    X = torch.zeros(10, 2)
    with pytest.raises(ValueError):
        km.kmeans_assign(X, torch.zeros(2, 2))
    with pytest.raises(ValueError):
        km.kmeans_run(X.double(), 2, torch.zeros(2, 2), 5)
