"""Write tests/golden/trajectory_<workload>.npz: the CPU oracle's whole Lloyd
trajectory (Algorithm 1 steps 2-7, fixed iteration count) on a named
workload, for the GPU tests that compare every iteration with it.

Only the oracle (oracle/) and the seeded input generator (workloads/) are
called; nothing here comes from the GPU library. The oracle needs minutes per
workload at these sizes (about half a nanosecond per object-centre-feature
term), which is why its results are stored.

Contents of each file (all arrays, no pickles):
  name, n, M, K, T          workload and iteration count
  sha256_x                  SHA-256 of the generated fp32 X (the inputs)
  init_idx                  initial objects, from oracle.init_farthest (the
                            farthest-point traversal of Algorithm 1 step 1),
                            checked against workloads/init_indices.json
  centers  [T, K, M] fp32   C_t for t = 1..T
  counts   [T, K]    int32  cluster sizes of labels_t
  sse      [T]       fp64   objective of labels_t against C_{t-1}
  labels_sha256 [T]         SHA-256 of labels_t (int32, little endian) with
                            every exempt object's label replaced by -1
  exempt_ptr [T+1]          exempt objects of pass t are exempt_idx[ptr[t-1]:ptr[t]]
  exempt_idx, exempt_lab, exempt_gap
                            objects whose best-vs-second gap (d2 - d1)/d2 is
                            below 1e-5 in pass t, with their oracle labels
  final_labels_sha256       SHA-256 of labels_T, unmasked

The loop is stepwise (oracle.assign, then oracle.update from the previous
centres), which is the oracle's own run loop in fixed mode; the script checks
that oracle.run(T, fixed=True) ends on the same labels, centres and counts.

Usage: python tests/golden/make_trajectories.py [4] [5]
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads  # noqa: E402

GAP_EXEMPT = 1e-5


def masked_sha(labels: np.ndarray, exempt: np.ndarray) -> str:
    lab = labels.astype("<i4", copy=True)
    lab[exempt] = -1
    return hashlib.sha256(lab.tobytes()).hexdigest()


def path_for(name: str) -> str:
    return os.path.join(HERE, f"trajectory_{workloads.get(name).name}.npz")


def make(name: str) -> str:
    w = workloads.get(name)
    T = w.max_iter
    t0 = time.time()
    X, _, stored_idx, _ = workloads.load(name)
    sha_x = workloads.x_sha256(X)
    idx = oracle.init_farthest(X, w.K)
    if not np.array_equal(idx, stored_idx):
        raise SystemExit(f"{w.name}: the oracle's initial objects differ from the stored ones")
    C = np.ascontiguousarray(X[idx])
    print(f"{w.name}: inputs and oracle initial centres in {time.time() - t0:.0f}s", flush=True)
    centers, counts, sse, shas = [], [], [], []
    e_ptr, e_idx, e_lab, e_gap = [0], [], [], []
    labels = None
    for t in range(1, T + 1):
        ts = time.time()
        labels, d1, d2 = oracle.assign(X, C, with_dist=True)
        gap = oracle.gap_rel(d1, d2)
        sse.append(float(np.sum(d1)))
        exempt = np.flatnonzero(gap < GAP_EXEMPT).astype(np.int32)
        e_idx.append(exempt)
        e_lab.append(labels[exempt].astype(np.int32))
        e_gap.append(gap[exempt])
        e_ptr.append(e_ptr[-1] + len(exempt))
        shas.append(masked_sha(labels, exempt))
        C, cnt = oracle.update(X, labels, w.K, C)
        centers.append(C.copy())
        counts.append(cnt.copy())
        print(f"{w.name}: t={t} exempt={len(exempt)} sse={sse[-1]:.6e} "
              f"({time.time() - ts:.0f}s)", flush=True)
        del d1, d2, gap
    final_sha = hashlib.sha256(labels.astype("<i4").tobytes()).hexdigest()
    # the stored trajectory is the oracle's own fixed-count run
    rl, rC, rcnt, rit = oracle.run(X, w.K, np.ascontiguousarray(X[idx]), T, fixed=True)
    assert rit == T
    assert np.array_equal(rl, labels), "run loop and stepwise labels differ"
    assert np.array_equal(rC.view(np.uint32), centers[-1].view(np.uint32))
    assert np.array_equal(rcnt, counts[-1])
    out = path_for(name)
    np.savez_compressed(
        out, name=np.array(w.name), n=np.int64(w.n), M=np.int32(w.M), K=np.int32(w.K),
        T=np.int32(T), sha256_x=np.array(sha_x), init_idx=idx.astype(np.int32),
        centers=np.stack(centers).astype(np.float32), counts=np.stack(counts).astype(np.int32),
        sse=np.asarray(sse, np.float64), labels_sha256=np.array(shas),
        exempt_ptr=np.asarray(e_ptr, np.int64), exempt_idx=np.concatenate(e_idx),
        exempt_lab=np.concatenate(e_lab), exempt_gap=np.concatenate(e_gap),
        final_labels_sha256=np.array(final_sha))
    print(f"{w.name}: wrote {out} in {time.time() - t0:.0f}s", flush=True)
    return out


if __name__ == "__main__":
    for nm in sys.argv[1:] or ["4", "5"]:
        make(nm)
