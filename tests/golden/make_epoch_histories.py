"""Write the oracle's per-epoch RMSE histories of the benchmark workloads.

For each named workload this script draws the seeded inputs (``workloads``),
buckets them with the oracle and runs the oracle's epoch (Algorithm 1's
inner loop, one pass per block) for the workload's stated epoch count,
taking the whole-matrix RMSE after every epoch (Algorithm 1's termination
test).  It calls nothing but ``oracle`` and ``workloads``.  Each output
file ``epoch_history_<name>.json`` records

  * the workload parameters (n, m, nnz, k, p, alpha, beta, epochs),
  * ``input_sha256``: a digest of the generated inputs (rows, cols, vals,
    U0, V0 as raw little-endian bytes, in that order), so that a test can
    check it is comparing against the same problem,
  * ``rmse``: the RMSE after epochs 1..E, and ``rmse0`` before the first,
  * ``norm_U``, ``norm_V``: Frobenius norms (binary64 sums) after each epoch.

The multithreaded oracle epoch is bit-identical to the sequential one (its
threads split the blocks of a stratum, which share no row or column).

Usage: python tests/golden/make_epoch_histories.py medium large vlarge
(workload arrays are cached under $BGMF_WORKLOAD_CACHE when it is set).
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from workloads import make_config  # noqa: E402

# The 250M-rating workload runs at its convergent step (its stated 0.002
# makes exact sequential SGD diverge on ratings in [0, 100] with k = 128).
OVERRIDES = {"vlarge": dict(alpha=5e-4)}


def input_digest(w) -> str:
    h = hashlib.sha256()
    for a in (w.rows, w.cols, w.vals, w.U0, w.V0):
        h.update(memoryview(np.ascontiguousarray(a)).cast("B"))
    return h.hexdigest()


def history(name: str, threads: int) -> dict:
    t0 = time.time()
    w = make_config(name, cache_dir=os.environ.get("BGMF_WORKLOAD_CACHE"),
                    **OVERRIDES.get(name, {}))
    digest = input_digest(w)
    print(f"[{time.time() - t0:7.1f} s] {name}: nnz={w.nnz} sha256={digest[:16]}", flush=True)
    bp, perm = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
    U, V = w.U0.copy(), w.V0.copy()
    out = dict(workload=name, n=w.n, m=w.m, nnz=w.nnz, k=w.k, p=w.p, alpha=w.alpha,
               beta=w.beta, epochs=w.epochs, input_sha256=digest,
               rmse0=oracle.rmse(w.rows, w.cols, w.vals, U, V), rmse=[], norm_U=[], norm_V=[])
    for e in range(w.epochs):
        oracle.epoch_mt(w.p, w.rows, w.cols, w.vals, bp, perm, U, V, w.alpha, w.beta, threads)
        r = oracle.rmse(w.rows, w.cols, w.vals, U, V)
        out["rmse"].append(r)
        out["norm_U"].append(float(np.sqrt(np.square(U, dtype=np.float64).sum())))
        out["norm_V"].append(float(np.sqrt(np.square(V, dtype=np.float64).sum())))
        print(f"[{time.time() - t0:7.1f} s] {name}: epoch {e + 1} rmse {r:.9f}", flush=True)
    out["generated_by"] = "tests/golden/make_epoch_histories.py (oracle epoch_mt, oracle rmse)"
    return out


def main(names):
    threads = os.cpu_count() or 1
    for name in names:
        res = history(name, threads)
        path = os.path.join(HERE, f"epoch_history_{name}.json")
        with open(path + ".tmp", "w") as f:
            json.dump(res, f, indent=1)
            f.write("\n")
        os.replace(path + ".tmp", path)
        print(f"wrote {path}", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or ["medium", "large", "vlarge"])
