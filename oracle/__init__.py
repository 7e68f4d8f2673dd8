"""fp64 CPU oracle for the exact Gauss sum and its gradients.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  It shares no code with the GPU
library: the arithmetic lives in ``gauss_oracle.c`` (plain C, fp64, double
loop in difference form), this module only marshals numpy arrays.

Definitions (paper "Fast Gauss Sums via Flash Attention"):
  * ``fwd``: s_m = sum_n exp(-tau/2 ||q_m - k_n||^2) v_n            (Sec. 1, Eq. 1)
  * ``dq``:  tau sum_n Phi w_mn (k_n - q_m), w_mn = <g_m, v_n>       (Sec. 3, the
    query-gradient equation for MMD flows / SVGD, contracted with g)
  * ``dk``:  tau sum_m Phi w_mn (q_m - k_n)                          (same, w.r.t. k)
  * ``dv``:  sum_m Phi g_m                                           (Eq. 1 is linear in v)

Each call returns ``(value, scale)`` where ``scale`` is the sum of absolute
values of the terms, the yardstick for the tolerance of a reduced-precision
evaluation: sum_n Phi |v_n| for the sum and dv, and for dq / dk (double sums
over keys and channels) tau sum_n Phi (sum_c |g_c v_c|) |k_n - q_m|.
``dq_scales`` / ``dk_scales`` also return the net scale
tau sum_n Phi |sum_c g_c v_c| |k_n - q_m| (the channels summed before the
magnitude: the other reading of the gradient tolerance, at most the first).

Inputs are converted to fp64 from whatever dtype they hold (float16, float32,
float64; bf16 must be passed already upcast), so the oracle sees exactly the
values a GPU kernel receives.  ``tau`` is taken as a Python float; callers pass
the float32 value the GPU library receives.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None


def load(path):
    """Load an oracle shared library at ``path`` and declare its signatures."""
    lib = ctypes.CDLL(path)
    i64, dp, ip = ctypes.c_int64, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)
    for name, has_g in (("gs_oracle_fwd", False), ("gs_oracle_dq", True),
                        ("gs_oracle_dk", True), ("gs_oracle_dv", True)):
        fn = getattr(lib, name)
        args = [i64, i64, i64, i64, dp, dp, dp]
        if has_g:
            args.append(dp)
        args += [ctypes.c_double, ip, i64, dp, dp, ctypes.c_int]
        fn.argtypes = args
        fn.restype = ctypes.c_int
    for name in ("gs_oracle_dq_scales", "gs_oracle_dk_scales"):
        fn = getattr(lib, name)
        fn.argtypes = [i64, i64, i64, i64, dp, dp, dp, dp, ctypes.c_double, ip, i64, dp, dp, dp, ctypes.c_int]
        fn.restype = ctypes.c_int
    return lib


def _lib():
    global _LIB
    if _LIB is None:
        _LIB = load(_build.build(force=False))
    return _LIB


def default_threads() -> int:
    """Threads the oracle uses: every host core this process may run on."""
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


def _f64(a, shape_rank=2):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    if a.ndim != shape_rank:
        raise ValueError("expected a %d-d array, got shape %s" % (shape_rank, a.shape))
    return a


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _rows(rows, limit):
    if rows is None:
        return None, limit
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1))
    return r, r.size


def _call(lib, name, q, k, v, g, tau, rows, out_width_is_c, key_rows, threads, net=False):
    q, k, v = _f64(q), _f64(k), _f64(v)
    M, D = q.shape
    N, Dk = k.shape
    Nv, C = v.shape
    if Dk != D or Nv != N:
        raise ValueError("shape mismatch: q %s, k %s, v %s" % (q.shape, k.shape, v.shape))
    if g is not None:
        g = _f64(g)
        if g.shape != (M, C):
            raise ValueError("g must be %s, got %s" % ((M, C), g.shape))
    r, nrows = _rows(rows, N if key_rows else M)
    width = C if out_width_is_c else D
    out = np.zeros((nrows, width), dtype=np.float64)
    absout = np.zeros((nrows, width), dtype=np.float64)
    netout = np.zeros((nrows, width), dtype=np.float64) if net else None
    rp = r.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if r is not None else None
    fn = getattr(lib, name)
    nt = threads or default_threads()
    args = [M, N, D, C, _ptr(q), _ptr(k), _ptr(v)]
    if g is not None:
        args.append(_ptr(g))
    args += [float(tau), rp, nrows, _ptr(out), _ptr(absout)]
    if net:
        args.append(_ptr(netout))
    args.append(nt)
    st = fn(*args)
    if st != 0:
        raise ValueError("%s failed with status %d" % (name, st))
    return (out, absout, netout) if net else (out, absout)


class Oracle:
    """The four oracle entry points bound to one shared library."""

    def __init__(self, lib=None):
        self._lib = lib

    @property
    def lib(self):
        return self._lib if self._lib is not None else _lib()

    def fwd(self, q, k, v, tau, rows=None, threads=None):
        """Eq. 1 for query rows ``rows`` (all if None): returns (s, sum_n Phi|v|)."""
        return _call(self.lib, "gs_oracle_fwd", q, k, v, None, tau, rows, True, False, threads)

    def dq(self, q, k, v, g, tau, rows=None, threads=None):
        """dL/dq for L = sum g*s on query rows ``rows``: returns (dq, scale)."""
        return _call(self.lib, "gs_oracle_dq", q, k, v, g, tau, rows, False, False, threads)

    def dk(self, q, k, v, g, tau, rows=None, threads=None):
        """dL/dk on key rows ``rows``: returns (dk, scale)."""
        return _call(self.lib, "gs_oracle_dk", q, k, v, g, tau, rows, False, True, threads)

    def dq_scales(self, q, k, v, g, tau, rows=None, threads=None):
        """dq with both scales: returns (dq, sum of |terms| over (n, c),
        tau sum_n Phi |w_mn| |k_n - q_m| (net over c))."""
        return _call(self.lib, "gs_oracle_dq_scales", q, k, v, g, tau, rows, False, False, threads, net=True)

    def dk_scales(self, q, k, v, g, tau, rows=None, threads=None):
        """dk with both scales, as dq_scales."""
        return _call(self.lib, "gs_oracle_dk_scales", q, k, v, g, tau, rows, False, True, threads, net=True)

    def dv(self, q, k, v, g, tau, rows=None, threads=None):
        """dL/dv on key rows ``rows``: returns (dv, scale)."""
        return _call(self.lib, "gs_oracle_dv", q, k, v, g, tau, rows, True, True, threads)


_DEFAULT = Oracle()
fwd = _DEFAULT.fwd
dq = _DEFAULT.dq
dk = _DEFAULT.dk
dv = _DEFAULT.dv
dq_scales = _DEFAULT.dq_scales
dk_scales = _DEFAULT.dk_scales
