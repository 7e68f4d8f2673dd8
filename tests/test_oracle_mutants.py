"""Plant plausible mistakes in copies of the oracle (on the CPU) and require
the pins to catch each one: evidence that the pins constrain every term of
the oracle, not only that the oracle agrees with itself."""
import os
import subprocess

import pytest

import oracle
import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "gauss_oracle.c")

# (id, text in gauss_oracle.c, replacement)
MUTANTS = [
    ("dropped_half", "exp(-0.5 * tau * d2)", "exp(-tau * d2)"),
    ("distance_sign", "double t = a[d] - b[d];", "double t = a[d] + b[d];"),
    ("dropped_last_dim", "for (int64_t d = 0; d < D; ++d) {\n    double t", "for (int64_t d = 0; d + 1 < D; ++d) {\n    double t"),
    ("fwd_wrong_value_row", "const double* vn = j->v + n * j->C;\n    double p = phi(qm", "const double* vn = j->v + (n % 2) * j->C;\n    double p = phi(qm"),
    ("abs_scale_not_abs", "a[c] += p * fabs(vn[c]);", "a[c] += p * vn[c];"),
    ("dq_sign", "double diff = kn[d] - qm[d];", "double diff = qm[d] - kn[d];"),
    ("dq_no_tau", "o[d] += j->tau * p * w * diff;\n      a[d] += j->tau * p * wa * fabs(diff);\n      if (nt) nt[d] += j->tau * p * fabs(w) * fabs(diff);\n    }\n  }\n}\n\n/* dk_n",
     "o[d] += p * w * diff;\n      a[d] += j->tau * p * wa * fabs(diff);\n      if (nt) nt[d] += j->tau * p * fabs(w) * fabs(diff);\n    }\n  }\n}\n\n/* dk_n"),
    ("net_scale_no_abs", "if (nt) nt[d] += j->tau * p * fabs(w) * fabs(diff);", "if (nt) nt[d] += j->tau * p * w * fabs(diff);"),
    ("net_scale_uses_abs_terms", "if (nt) nt[d] += j->tau * p * fabs(w) * fabs(diff);", "if (nt) nt[d] += j->tau * p * wa * fabs(diff);"),
    ("grad_scale_uses_w", "a[d] += j->tau * p * wa * fabs(diff);", "a[d] += j->tau * p * fabs(w) * fabs(diff);"),
    ("dq_transposed_g", "const double* gm = j->g + m * j->C;\n  for (int64_t d", "const double* gm = j->g + (m % 2) * j->C;\n  for (int64_t d"),
    ("dk_sign", "double diff = qm[d] - kn[d];", "double diff = kn[d] - qm[d];"),
    ("dk_w_wrong_operand", "double w = dotc(j->g + m * j->C, vn, j->C);", "double w = dotc(j->g + m * j->C, j->v + m % j->N * j->C, j->C);"),
    ("dv_channel_index", "o[c] += p * gm[c];", "o[c] += p * gm[0];"),
    ("dv_uses_v", "o[c] += p * gm[c];", "o[c] += p * j->v[n * j->C + c];"),
    ("dotc_dropped_channel", "for (int64_t c = 0; c < C; ++c) w += gm[c] * vn[c];", "for (int64_t c = 0; c + 1 < C; ++c) w += gm[c] * vn[c];"),
    ("row_index_ignored", "int64_t row = j->rows ? j->rows[r] : r;", "int64_t row = r;"),
]


def _build_mutant(tmpdir, ident, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, "mutation %s does not apply" % ident
    mutated = src.replace(old, new, 1)
    c = os.path.join(tmpdir, ident + ".c")
    so = os.path.join(tmpdir, ident + ".so")
    with open(c, "w") as f:
        f.write(mutated)
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-o", so, c, "-lm", "-lpthread"], check=True)
    return so


@pytest.mark.parametrize("ident,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, ident, old, new):
    so = _build_mutant(str(tmp_path), ident, old, new)
    orc = oracle.Oracle(oracle.load(so))
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(orc)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, "mutant %s passed every pin" % ident
