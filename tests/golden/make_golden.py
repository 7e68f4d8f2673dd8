"""Write tests/golden/dyadic_lattice.txt by calling the oracle only.

Workload: integer points in {-2..2}^3 (6 queries, 9 keys, seed 15 of
numpy's PCG64), values in quarter steps, tau = 2 ln 2, so that every kernel
value exp(-tau/2 ||q-k||^2) of Eq. 1 is the power of two 2^(-||q-k||^2) and
each s_m is a finite dyadic sum.  The test re-derives those sums in exact
rational arithmetic and checks the stored oracle output against them and
the live oracle against the stored output.
"""
import math
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402


def inputs():
    r = np.random.default_rng(15)
    q = r.integers(-2, 3, size=(6, 3)).astype(np.float64)
    k = r.integers(-2, 3, size=(9, 3)).astype(np.float64)
    v = r.integers(-8, 9, size=(9, 2)).astype(np.float64) / 4.0
    return q, k, v, 2.0 * math.log(2.0)


def main():
    q, k, v, tau = inputs()
    s, a = oracle.fwd(q, k, v, tau, threads=1)
    path = os.path.join(HERE, "dyadic_lattice.txt")
    with open(path, "w") as f:
        f.write("# Eq. 1 on a dyadic lattice (tau = 2 ln 2); written by make_golden.py via the oracle\n")
        f.write("# columns: m, s[m,0], s[m,1], A[m,0], A[m,1]\n")
        for m in range(s.shape[0]):
            f.write("%d %.17g %.17g %.17g %.17g\n" % (m, s[m, 0], s[m, 1], a[m, 0], a[m, 1]))
    print(path)


if __name__ == "__main__":
    main()
