"""Writes tests/golden/t_need.json: for every matrix of the ImageNet-like
stack and of the stress batch, the number of Björck steps after which the
float64 oracle's iteration has converged (every singular value of the
Frobenius-scaled matrix mapped to within 1e-6 of 1 in sigma^2, computed
from the SVD by the scalar recursion that the iteration applies to each
singular value, Appendix A.5).  The GPU tests run a second pass at
T_conv = max T_need + 2 and gate orthogonality on every matrix.

    python tests/golden/make_t_need.py [--jobs N]

Calls only the oracle and the seeded input generator; takes about half an
hour on 8 cores (the 64 SVDs of 4096 x 4096 matrices dominate).
"""

import argparse
import concurrent.futures as cf
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import bjorck  # noqa: E402
from paper_2601_13776_amd import workloads as wl  # noqa: E402

TOL = 1e-6
NAMES = ("imagenet_backbone25", "stress_4096x64_32x4096")


def one(args):
    name, i = args
    w = wl.WORKLOADS[name]
    r, c = w.matrix_shapes()[i]
    return bjorck.iterations_to_converge(wl.as_f64(wl.stored_matrix(w, i, r, c)), tol=TOL, max_iters=400)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=2)
    args = ap.parse_args()
    out = {"tol": TOL, "workloads": {}}
    for name in NAMES:
        w = wl.WORKLOADS[name]
        n = len(w.matrix_shapes())
        with cf.ThreadPoolExecutor(max_workers=args.jobs) as ex:
            t = list(ex.map(one, [(name, i) for i in range(n)]))
        out["workloads"][name] = {"iters": w.iters, "t_need": t, "t_conv": max(t) + 2}
        print(name, "max T_need", max(t), flush=True)
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "t_need.json")
    with open(path, "w") as f:
        json.dump(out, f, separators=(",", ":"))
        f.write("\n")


if __name__ == "__main__":
    main()
