"""Writes fc4096_lambda.json: the regulariser strength lambda of the 4096x4096
density sweep (batch 512, densities 1/5/20/50 %, eta 0.01).

lambda is set so that the first l1-phase step (Eq. (prox) applied to all N*K
weights, soft-threshold of Section 2.2) changes about 2 % of the stored
pattern: flips(lambda) = #{(i,k): (W'[i,k] != 0) != (W[i,k] != 0)} equals
0.02 * nnz(W).  flips is large for small lambda (zero weights regrow), falls,
and rises again once deletions dominate; the smaller root is taken (a lambda
that both regrows and deletes a little).  Everything here is computed by the
oracle on the seeded inputs of iteration 0.

Run from the repository root:  python tests/golden/make_fc4096_lambda.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_1905_07931_amd import synth  # noqa: E402

DENSITIES = (0.01, 0.05, 0.20, 0.50)
TARGET = 0.02


def flips_fn(L, dW):
    dense_old = oracle.densify(L.row_ptr, L.col_idx, L.vals, L.K) != 0

    def flips(lam):
        Z, _ = oracle.prox_dense(L.row_ptr, L.col_idx, L.vals, dW, L.eta, lam, L.K)
        return int(np.count_nonzero((Z != 0) != dense_old))
    return flips


def lower_root(flips, nnz):
    """Smallest lambda on a log grid with flips <= TARGET * nnz, refined by bisection."""
    goal = TARGET * nnz
    grid = np.logspace(-4, 1, 101)
    prev = None
    for lam in grid:
        if flips(lam) <= goal:
            lo, hi = (prev if prev is not None else lam / 10), lam
            break
        prev = lam
    else:
        raise RuntimeError("flips never reaches the target")
    for _ in range(40):
        mid = 0.5 * (lo + hi)
        if flips(mid) <= goal:
            hi = mid
        else:
            lo = mid
    return float(np.float32(hi))


def main():
    out = {"_what": "lambda per density for the 4096x4096 sweep (batch 512, eta 0.01): the smaller "
                    "root of flips(lambda) = 0.02 * nnz at iteration 0, from the oracle",
           "_written_by": "tests/golden/make_fc4096_lambda.py", "lambda": {}, "flips": {}, "nnz": {}}
    for d in DENSITIES:
        L = synth.fc4096_sweep(d)
        X, dY = synth.fc4096_batch(0)
        dW = oracle.dense_wgrad(dY, X)
        flips = flips_fn(L, dW)
        lam = lower_root(flips, L.nnz)
        key = f"{int(round(d * 100))}"
        out["lambda"][key] = lam
        out["flips"][key] = flips(lam)
        out["nnz"][key] = int(L.nnz)
        print(f"density {d:.2f}: nnz {L.nnz}, lambda {lam:.6g}, flips {flips(lam)} "
              f"({flips(lam) / L.nnz:.4f} of nnz)", flush=True)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "fc4096_lambda.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")
    print("wrote", path)


if __name__ == "__main__":
    main()
