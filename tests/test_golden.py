"""Stored oracle output for the dyadic-lattice example (Eq. 1 with tau = 2 ln 2)."""
import os
from fractions import Fraction

import numpy as np

import oracle
from golden.make_golden import inputs

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "dyadic_lattice.txt")


def _load():
    rows = [list(map(float, ln.split())) for ln in open(PATH) if not ln.startswith("#")]
    arr = np.array(rows)
    return arr[:, 1:3], arr[:, 3:5]


def test_golden_matches_exact_dyadic_sums():
    q, k, v, _ = inputs()
    s, a = _load()
    for m in range(q.shape[0]):
        for c in range(2):
            tot = Fraction(0)
            tot_abs = Fraction(0)
            for n in range(k.shape[0]):
                d2 = int(sum((int(q[m, d]) - int(k[n, d])) ** 2 for d in range(3)))
                tot += Fraction(1, 2 ** d2) * Fraction(v[n, c])
                tot_abs += Fraction(1, 2 ** d2) * abs(Fraction(v[n, c]))
            assert abs(s[m, c] - float(tot)) <= 1e-13 * max(1.0, abs(float(tot)))
            assert abs(a[m, c] - float(tot_abs)) <= 1e-13 * max(1.0, float(tot_abs))


def test_oracle_reproduces_golden():
    q, k, v, tau = inputs()
    s, a = oracle.fwd(q, k, v, tau)
    s0, a0 = _load()
    assert np.array_equal(s, s0) and np.array_equal(a, a0)
