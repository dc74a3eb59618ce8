"""Write workloads/init_indices.json: for each named workload, the SHA-256 of the
generated X and the farthest-point initial indices (fp64, from object 0).

The larger workloads take minutes to initialise on a CPU; storing the indices
lets tests and the benchmark skip that step. workloads.load() uses an entry
only when the freshly generated X has the recorded hash.

Usage: python -m workloads.make_init_table [name ...]
"""
import json
import sys
import time

import workloads as W


def main(names):
    table = W._init_table()
    for name in names:
        w = W.get(name)
        t0 = time.time()
        X, _ = W.generate(w)
        h = W.x_sha256(X)
        idx = W.farthest_point_init(X, w.K)
        table[w.name] = {"n": w.n, "M": w.M, "K": w.K, "seed": w.seed,
                         "sha256_x": h, "init": [int(i) for i in idx]}
        print(f"{w.name}: sha256 {h[:16]}..., {len(idx)} indices, {time.time() - t0:.1f}s",
              flush=True)
        with open(W.INIT_TABLE, "w") as f:
            json.dump(table, f, indent=1)
            f.write("\n")


if __name__ == "__main__":
    main(sys.argv[1:] or list(W.WORKLOADS))
