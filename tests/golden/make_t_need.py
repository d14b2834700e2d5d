"""Writes tests/golden/t_need.json: for every matrix of the ImageNet-like
stack and of the stress batch, the number of Björck steps after which the
float64 oracle's iteration has converged (every singular value of the
Frobenius-scaled matrix mapped to within 1e-6 of 1 in sigma^2, computed
from the SVD by the scalar recursion that the iteration applies to each
singular value, Appendix A.5).  The GPU tests run a second pass at
T_conv = max T_need + 2 and gate orthogonality on every matrix.

    python tests/golden/make_t_need.py [--jobs N]

Calls only the oracle and the seeded input generator; takes about half an
hour on 8 cores (the 64 SVDs of 4096 x 4096 matrices dominate); an interrupted run
resumes from tests/golden/t_need.partial.json.
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
    here = os.path.dirname(os.path.abspath(__file__))
    # results so far, so that an interrupted run resumes where it stopped
    partial = os.path.join(here, "t_need.partial.json")
    done = json.load(open(partial)) if os.path.exists(partial) else {}
    out = {"tol": TOL, "workloads": {}}
    for name in NAMES:
        w = wl.WORKLOADS[name]
        n = len(w.matrix_shapes())
        have = {int(k): v for k, v in done.get(name, {}).items()}
        todo = [i for i in range(n) if i not in have]
        with cf.ThreadPoolExecutor(max_workers=args.jobs) as ex:
            for i, t in zip(todo, ex.map(one, [(name, i) for i in todo])):
                have[i] = t
                done.setdefault(name, {})[str(i)] = t
                if len(have) % 8 == 0 or len(have) == n:
                    with open(partial, "w") as f:
                        json.dump(done, f)
        t = [have[i] for i in range(n)]
        out["workloads"][name] = {"iters": w.iters, "t_need": t, "t_conv": max(t) + 2}
        print(name, "max T_need", max(t), flush=True)
    with open(os.path.join(here, "t_need.json"), "w") as f:
        json.dump(out, f, separators=(",", ":"))
        f.write("\n")
    os.remove(partial)


if __name__ == "__main__":
    main()
