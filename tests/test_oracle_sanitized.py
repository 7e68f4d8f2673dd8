"""The oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer
(host code only, gcc): every pin runs against an instrumented build of the
oracle and of each planted mutant, and any out-of-bounds access, use after
free or undefined operation aborts the run.  A planted read past the end of
the value array checks that the sanitizer is really active."""
import json
import os
import shutil
import subprocess
import sys

import pytest

import oracle
from test_oracle_mutants import MUTANTS

SRC = os.path.join(os.path.dirname(oracle.__file__), "gauss_oracle.c")
RUNNER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "pin_runner.py")
FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=all", "-fno-fast-math", "-ffp-contract=off",
         "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra"]

# One access past the end of v: the last key's row is read from one row further on.
OVERRUN = ("const double* vn = j->v + n * j->C;\n    double p = phi(qm",
           "const double* vn = j->v + (n + (n + 1 == j->N)) * j->C;\n    double p = phi(qm")


def _asan_runtime():
    if shutil.which("gcc") is None:
        return None
    path = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _build(tmpdir, name, src_text):
    c = os.path.join(tmpdir, name + ".c")
    so = os.path.join(tmpdir, name + ".so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc"] + FLAGS + ["-o", so, c, "-lm", "-lpthread"], check=True)
    return so


def _run(libs):
    env = dict(os.environ, LD_PRELOAD=_asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    return subprocess.run([sys.executable, RUNNER] + libs, capture_output=True, text=True,
                          env=env, timeout=600)


needs_asan = pytest.mark.skipif(
    _asan_runtime() is None or bool(os.environ.get("LD_PRELOAD")),
    reason="needs gcc's AddressSanitizer runtime and no other preloaded library")


@needs_asan
def test_pins_and_mutants_clean_under_sanitizers(tmp_path):
    src = open(SRC).read()
    libs = [_build(str(tmp_path), "oracle", src)]
    for ident, old, new in MUTANTS:
        assert src.count(old) >= 1, ident
        libs.append(_build(str(tmp_path), ident, src.replace(old, new, 1)))
    res = _run(libs)
    assert res.returncode == 0, res.stderr[-4000:]
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, res.stderr[-4000:]
    lines = [json.loads(x) for x in res.stdout.splitlines() if x.startswith("{")]
    assert [x["lib"] for x in lines] == libs
    assert lines[0]["caught"] == [], "sanitized oracle fails pins %s" % lines[0]["caught"]
    for (ident, _, _), rec in zip(MUTANTS, lines[1:]):
        assert rec["caught"], "sanitized mutant %s passed every pin" % ident


@needs_asan
def test_planted_overrun_is_reported(tmp_path):
    src = open(SRC).read()
    assert src.count(OVERRUN[0]) == 1
    lib = _build(str(tmp_path), "overrun", src.replace(*OVERRUN))
    res = _run([lib])
    assert res.returncode != 0
    assert "heap-buffer-overflow" in res.stderr, res.stderr[-4000:]
