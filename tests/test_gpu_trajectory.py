"""GPU parity over whole trajectories of the two fixed-30-iteration workloads
(2*10^6 x 25 with K = 256, and 2*10^7 x 25 with K = 64, Zipf sizes and
uniform noise), against the CPU oracle's stored run (Algorithm 1 steps 2-7).

The oracle needs minutes per workload at these sizes, so its trajectory is
stored in tests/golden/trajectory_<workload>.npz, written by
tests/golden/make_trajectories.py from the oracle alone: every iteration's
centres and counts, a SHA-256 of every iteration's labels with the near-tie
objects (best-vs-second gap below 1e-5 relative) masked out, and those objects
with their oracle labels.

Checked here, through the C ABI:
  - the generated inputs and the GPU farthest-point initial centres are the
    ones the oracle run started from;
  - for t = 1..T, the GPU's C_t and counts (iteration t of one trajectory from
    C_0, each step started from the GPU's previous centres, which equal the
    oracle's) against the stored ones, and every label of pass t (all n
    objects) against the stored hash, the exempt ones compared one by one;
  - one fixed-count kmeans_run of all T iterations from C_0, whose final
    labels, centres and counts must equal the stepwise ones;
  - on the noisy workload, the assignment of the last pass with every label
    decided in fp64 (KMEANS_FORCE_FP64) gives the same labels as the default
    screening.
"""
import hashlib
import os

import numpy as np
import pytest
import torch

import paper_1402_3788_amd as km
import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None
HERE = os.path.dirname(os.path.abspath(__file__))
CENTER_RTOL = 1e-5


def _say(msg):
    print(msg, flush=True)


def _golden(name):
    w = workloads.get(name)
    path = os.path.join(HERE, "golden", f"trajectory_{w.name}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not written (tests/golden/make_trajectories.py)")
    return w, np.load(path, allow_pickle=False)


def _masked_sha(labels: np.ndarray, exempt: np.ndarray) -> str:
    lab = labels.astype("<i4", copy=True)
    lab[exempt] = -1
    return hashlib.sha256(lab.tobytes()).hexdigest()


def _check_centers(C, oC):
    scale = np.maximum(np.abs(oC).max(axis=1, keepdims=True), 1e-30)
    err = np.abs(C.astype(np.float64) - oC.astype(np.float64))
    assert (err <= CENTER_RTOL * scale).all(), f"max centre error {(err / scale).max():.3g}"
    return int((C.view(np.uint32) != oC.view(np.uint32)).sum())


def _check_pass(gd, t, lab, C, cnt):
    """Iteration t (1-based) of the GPU against the stored oracle iteration."""
    lo, hi = int(gd["exempt_ptr"][t - 1]), int(gd["exempt_ptr"][t])
    ex_idx, ex_lab = gd["exempt_idx"][lo:hi], gd["exempt_lab"][lo:hi]
    assert _masked_sha(lab, ex_idx) == str(gd["labels_sha256"][t - 1]), \
        f"t={t}: labels outside the near-tie band differ from the oracle's"
    nmis = int((lab[ex_idx] != ex_lab).sum())
    ocnt = gd["counts"][t - 1]
    assert np.abs(cnt.astype(np.int64) - ocnt).sum() <= 2 * nmis, f"t={t}: counts"
    nbits = _check_centers(C, gd["centers"][t - 1])
    return nmis, len(ex_idx), nbits


def _trajectory(name):
    w, gd = _golden(name)
    T = int(gd["T"])
    _say(f"[trajectory] {w.name}: generating inputs")
    X, _, init_idx, init = workloads.load(name)
    assert workloads.x_sha256(X) == str(gd["sha256_x"]), "inputs differ from the oracle run's"
    assert np.array_equal(init_idx, gd["init_idx"])
    Xg = torch.from_numpy(X).to(DEV)
    n, M, K = w.n, w.M, w.K
    del X
    # the GPU farthest-point traversal gives the initial objects of the oracle run
    gidx, gC = km.kmeans_init_farthest(Xg, K)
    assert np.array_equal(gidx.cpu().numpy(), gd["init_idx"])
    assert np.array_equal(gC.cpu().numpy().view(np.uint32), init.view(np.uint32))

    ws = km.workspace(n, M, K, DEV, km.KMEANS_FIXED_ITERS)
    lab = torch.empty(n, dtype=torch.int32, device=DEV)
    cnt = torch.empty(K, dtype=torch.int32, device=DEV)
    C = torch.empty((K, M), dtype=torch.float32, device=DEV)
    prev = gC.clone()
    tot_mis = tot_ex = tot_bits = tot_fb = 0
    for t in range(1, T + 1):
        _, _, _, it = km.kmeans_run(Xg, K, prev, 1, fixed_iters=True, out=(lab, C, cnt), ws=ws)
        assert it == 1
        tot_fb += km.ctl_fallbacks(ws)
        nmis, nex, nbits = _check_pass(gd, t, lab.cpu().numpy(), C.cpu().numpy(),
                                       cnt.cpu().numpy())
        tot_mis += nmis
        tot_ex += nex
        tot_bits += nbits
        prev.copy_(C)
    _say(f"[trajectory] {w.name}: {T} iterations match the oracle; exempt objects "
         f"{tot_ex}, of which labelled differently {tot_mis}; centre coordinates not "
         f"bit-identical {tot_bits}; objects re-decided in fp64 {tot_fb}")

    # the same T iterations as one fixed-count call
    lab2, C2, cnt2, it = km.kmeans_run(Xg, K, gC, T, fixed_iters=True, ws=ws)
    assert it == T
    assert torch.equal(lab2, lab) and torch.equal(cnt2, cnt)
    assert torch.equal(C2.view(torch.int32), C.view(torch.int32))
    return w, gd, Xg, prev


def test_trajectory_blobs25d_n2m_k256():
    _trajectory("4")


def test_trajectory_zipfnoise25d_n20m_k64():
    w, gd, Xg, C = _trajectory("5")
    # Last pass again from C_{T-1} (the oracle's, bit for bit here): every
    # label decided with fp64 distances gives the same labels as the
    # screening, and both agree with the stored pass.
    T = int(gd["T"])
    Cprev = torch.from_numpy(np.ascontiguousarray(gd["centers"][T - 2])).to(DEV)
    a = km.kmeans_assign(Xg, Cprev)
    b = km.kmeans_assign(Xg, Cprev, force_fp64=True)
    nd = int((a != b).sum().item())
    assert nd == 0, f"{nd} labels differ between the screened and the all-fp64 assignment"
    lo, hi = int(gd["exempt_ptr"][T - 1]), int(gd["exempt_ptr"][T])
    assert _masked_sha(b.cpu().numpy(), gd["exempt_idx"][lo:hi]) == str(gd["labels_sha256"][T - 1])
    _say(f"[trajectory] {w.name}: all-fp64 assignment of pass {T} equals the screened one")
