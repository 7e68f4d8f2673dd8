"""Thin ctypes binding of the C ABI in include/gauss_sum.h.

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libgauss_sum.so``.  PyTorch provides device memory (inputs,
outputs, workspace) and the stream.  There is no fallback: if the library is
missing or a call fails, an exception is raised.

Entry points mirror the C names:
  gauss_sum_fwd(q, k, v, tau)                       -> s        (Eq. 1; fp32
                                                       points: the fp32-accuracy
                                                       tier, C = 1)
  gauss_sum_bwd(q, k, v, tau, dout, want=...)       -> dq, dk, dv
  gauss_sum_fwd_bwd(q, k, v, tau, dout, want=...)   -> s, dq, dk, dv (one call;
                                                       s and dq from one pass)
  gauss_sum_fwd_workspace_size / gauss_sum_bwd_workspace_size /
  gauss_sum_fwd_bwd_workspace_size
  gauss_sum_fwd_batched / gauss_sum_bwd_batched (B independent problems,
  grid.z) and their workspace sizes; gauss_sum_mmd_flow (s, flow field, MMD^2)
  gauss_sum_status_string / gauss_sum_abi_version
and ``GaussSum`` wraps both in a torch.autograd.Function.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgauss_sum.so")

GS_F32, GS_F16, GS_BF16 = 0, 1, 2
STATUS = {
    0: "GS_SUCCESS", 1: "GS_ERR_NULL_POINTER", 2: "GS_ERR_BAD_SHAPE", 3: "GS_ERR_BAD_TAU",
    4: "GS_ERR_UNSUPPORTED", 5: "GS_ERR_MISALIGNED", 6: "GS_ERR_WORKSPACE", 7: "GS_ERR_HIP",
    8: "GS_ERR_INTERNAL", 9: "GS_ERR_ALIAS", 10: "GS_ERR_SCRATCH_LIMIT",
}
NOALLOC_SCRATCH_BYTES = 128 << 20   # GAUSS_SUM_NOALLOC_SCRATCH_BYTES
EXPORTED = ("gauss_sum_fwd", "gauss_sum_bwd", "gauss_sum_fwd_bwd", "gauss_sum_fwd_workspace_size",
            "gauss_sum_bwd_workspace_size", "gauss_sum_fwd_bwd_workspace_size",
            "gauss_sum_status_string", "gauss_sum_abi_version", "gauss_sum_profile_start",
            "gauss_sum_profile_stop", "gauss_sum_mmd_flow", "gauss_sum_mmd_flow_workspace_size",
            "gauss_sum_fwd_batched", "gauss_sum_bwd_batched", "gauss_sum_fwd_batched_workspace_size",
            "gauss_sum_bwd_batched_workspace_size", "gauss_sum_fwd_bwd_batched",
            "gauss_sum_fwd_bwd_batched_workspace_size", "gauss_sum_svgd", "gauss_sum_svgd_workspace_size",
            "gauss_sum_fwd_noalloc")
PROFILE_FWD, PROFILE_GRAD = 1, 2


class GaussSumError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = "%s failed: %s (%s)" % (where, STATUS.get(status, "?"), status_string(status))
        super().__init__(msg)


class Batch(ctypes.Structure):
    _fields_ = [("count", ctypes.c_int64), ("q_stride", ctypes.c_int64), ("k_stride", ctypes.c_int64),
                ("v_stride", ctypes.c_int64), ("dout_stride", ctypes.c_int64),
                ("out_stride", ctypes.c_int64), ("dq_stride", ctypes.c_int64),
                ("dk_stride", ctypes.c_int64), ("dv_stride", ctypes.c_int64)]


class Problem(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("D", ctypes.c_int64),
                ("C", ctypes.c_int64), ("qk_dtype", ctypes.c_int), ("v_dtype", ctypes.c_int)]


_lib = None


def load(path=LIB_PATH, torch_runtime=True):
    """Load libgauss_sum.so (built in-tree by ``__graft_entry__.build()``).

    torch is imported first (torch_runtime): PyTorch for ROCm ships its own
    HIP runtime, loaded under the unversioned name libamdhip64.so, while
    the library asks for libamdhip64.so.7.  With torch's copy already in the
    process that request binds to it; the other way round the process holds
    two HIP runtimes, and torch's streams and allocations are not valid in
    the library's, so every call fails with GS_ERR_HIP.  Callers of the C
    ABI without torch are not affected."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("HIP library %s is missing: run __graft_entry__.build() first" % path)
    if torch_runtime:
        import torch  # noqa: F401  (its HIP runtime first, see above)
    lib = ctypes.CDLL(path)
    vp, sz, f32p = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p
    P = ctypes.POINTER(Problem)
    lib.gauss_sum_fwd_workspace_size.argtypes = [P]
    lib.gauss_sum_fwd_workspace_size.restype = sz
    lib.gauss_sum_bwd_workspace_size.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.gauss_sum_bwd_workspace_size.restype = sz
    lib.gauss_sum_fwd.argtypes = [P, vp, vp, vp, ctypes.c_float, f32p, vp, sz, vp]
    lib.gauss_sum_fwd.restype = ctypes.c_int
    lib.gauss_sum_fwd_noalloc.argtypes = [P, vp, vp, vp, ctypes.c_float, f32p, vp]
    lib.gauss_sum_fwd_noalloc.restype = ctypes.c_int
    lib.gauss_sum_bwd.argtypes = [P, vp, vp, vp, ctypes.c_float, vp, ctypes.c_int, f32p, f32p, f32p,
                                  vp, sz, vp]
    lib.gauss_sum_bwd.restype = ctypes.c_int
    lib.gauss_sum_fwd_bwd.argtypes = [P, vp, vp, vp, ctypes.c_float, vp, ctypes.c_int, f32p, f32p,
                                      f32p, f32p, vp, sz, vp]
    lib.gauss_sum_fwd_bwd.restype = ctypes.c_int
    lib.gauss_sum_fwd_bwd_workspace_size.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.gauss_sum_fwd_bwd_workspace_size.restype = sz
    BP = ctypes.POINTER(Batch)
    lib.gauss_sum_fwd_batched.argtypes = [P, BP, vp, vp, vp, ctypes.c_float, f32p, vp, sz, vp]
    lib.gauss_sum_fwd_batched.restype = ctypes.c_int
    lib.gauss_sum_bwd_batched.argtypes = [P, BP, vp, vp, vp, ctypes.c_float, vp, ctypes.c_int, f32p,
                                          f32p, f32p, vp, sz, vp]
    lib.gauss_sum_bwd_batched.restype = ctypes.c_int
    lib.gauss_sum_fwd_batched_workspace_size.argtypes = [P, ctypes.c_int64]
    lib.gauss_sum_fwd_batched_workspace_size.restype = sz
    lib.gauss_sum_bwd_batched_workspace_size.argtypes = [P, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                                         ctypes.c_int]
    lib.gauss_sum_bwd_batched_workspace_size.restype = sz
    lib.gauss_sum_fwd_bwd_batched.argtypes = [P, BP, vp, vp, vp, ctypes.c_float, vp, ctypes.c_int,
                                              f32p, f32p, f32p, f32p, vp, sz, vp]
    lib.gauss_sum_fwd_bwd_batched.restype = ctypes.c_int
    lib.gauss_sum_fwd_bwd_batched_workspace_size.argtypes = [P, ctypes.c_int64, ctypes.c_int,
                                                             ctypes.c_int, ctypes.c_int]
    lib.gauss_sum_fwd_bwd_batched_workspace_size.restype = sz
    lib.gauss_sum_mmd_flow.argtypes = [P, vp, vp, ctypes.c_float, f32p, f32p, vp, vp, sz, vp]
    lib.gauss_sum_svgd.argtypes = [P, vp, vp, ctypes.c_float, f32p, vp, sz, vp]
    lib.gauss_sum_svgd.restype = ctypes.c_int
    lib.gauss_sum_svgd_workspace_size.argtypes = [P]
    lib.gauss_sum_svgd_workspace_size.restype = sz
    lib.gauss_sum_mmd_flow.restype = ctypes.c_int
    lib.gauss_sum_mmd_flow_workspace_size.argtypes = [P]
    lib.gauss_sum_mmd_flow_workspace_size.restype = sz
    lib.gauss_sum_status_string.argtypes = [ctypes.c_int]
    lib.gauss_sum_status_string.restype = ctypes.c_char_p
    lib.gauss_sum_abi_version.argtypes = []
    lib.gauss_sum_abi_version.restype = ctypes.c_int
    lib.gauss_sum_profile_start.argtypes = [ctypes.c_int, ctypes.c_int]
    lib.gauss_sum_profile_start.restype = ctypes.c_int
    lib.gauss_sum_profile_stop.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_int]
    lib.gauss_sum_profile_stop.restype = ctypes.c_int
    if path == LIB_PATH:
        _lib = lib
    return lib


def status_string(status):
    return load().gauss_sum_status_string(int(status)).decode()


gauss_sum_status_string = status_string


def gauss_sum_abi_version():
    return load().gauss_sum_abi_version()


def gauss_sum_profile_start(capacity, kind):
    """Start bracketing main-kernel launches of ``kind`` with HIP events."""
    st = load().gauss_sum_profile_start(int(capacity), int(kind))
    if st != 0:
        raise GaussSumError(st, "gauss_sum_profile_start")


def gauss_sum_profile_stop(capacity):
    """Per-launch durations (ms) recorded since gauss_sum_profile_start."""
    buf = (ctypes.c_float * max(1, int(capacity)))()
    n = load().gauss_sum_profile_stop(buf, int(capacity))
    if n < 0:
        raise GaussSumError(7, "gauss_sum_profile_stop")
    return [float(buf[i]) for i in range(min(n, int(capacity)))]


def _dtype_code(t):
    import torch
    codes = {torch.float32: GS_F32, torch.float16: GS_F16, torch.bfloat16: GS_BF16}
    if t not in codes:
        raise TypeError("unsupported dtype %s" % t)
    return codes[t]


def make_problem(M, N, D, C, qk_dtype, v_dtype):
    return Problem(int(M), int(N), int(D), int(C), int(qk_dtype), int(v_dtype))


def gauss_sum_fwd_workspace_size(M, N, D, C, qk_dtype=GS_F16, v_dtype=GS_F32):
    return int(load().gauss_sum_fwd_workspace_size(ctypes.byref(make_problem(M, N, D, C, qk_dtype, v_dtype))))


def gauss_sum_bwd_workspace_size(M, N, D, C, qk_dtype=GS_F16, v_dtype=GS_F32, want_dq=True,
                                 want_dk=True, want_dv=True):
    p = make_problem(M, N, D, C, qk_dtype, v_dtype)
    return int(load().gauss_sum_bwd_workspace_size(ctypes.byref(p), int(bool(want_dq)),
                                                   int(bool(want_dk)), int(bool(want_dv))))


def gauss_sum_fwd_bwd_workspace_size(M, N, D, C, qk_dtype=GS_F16, v_dtype=GS_F32, want_dq=True,
                                     want_dk=True, want_dv=True):
    p = make_problem(M, N, D, C, qk_dtype, v_dtype)
    return int(load().gauss_sum_fwd_bwd_workspace_size(ctypes.byref(p), int(bool(want_dq)),
                                                       int(bool(want_dk)), int(bool(want_dv))))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check_inputs(q, k, v):
    """q: M x D, k: N x D, v: N x C, contiguous, on one GPU; q and k share a
    dtype.  Shapes are checked before devices (so a mismatch is reported the
    same way on any machine)."""
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dim() != 2 or not t.is_contiguous():
            raise ValueError("%s must be a contiguous 2-d tensor" % name)
    if tuple(k.shape) != (v.shape[0], q.shape[1]):
        raise ValueError("k must be %d x %d (rows of v x columns of q), got %s"
                         % (v.shape[0], q.shape[1], tuple(k.shape)))
    if q.dtype != k.dtype:
        raise TypeError("q and k must share a dtype")
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not t.is_cuda:
            raise ValueError("%s must be a GPU tensor" % name)
    if k.device != q.device or v.device != q.device:
        raise ValueError("q, k and v must be on one device")


def _check_tensor(t, name, shape, device, dtype=None):
    """A caller-supplied tensor: the exact shape, contiguous (and of `dtype`
    if given), on `device`."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a tensor" % name)
    if tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError("%s must be a contiguous %s tensor, got %s" % (name, "x".join(map(str, shape)),
                                                                      tuple(t.shape)))
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_cuda or t.device != device:
        raise ValueError("%s must be a GPU tensor on %s" % (name, device))


def _output(out, name, shape, device):
    """`out` checked (fp32, exact shape, contiguous, on device), or a new one."""
    import torch
    if out is None:
        return torch.empty(shape, dtype=torch.float32, device=device)
    _check_tensor(out, name, shape, device, torch.float32)
    return out


def _workspace(nbytes, device):
    import torch
    if nbytes == 0:
        return None, 0
    return torch.empty(nbytes, dtype=torch.uint8, device=device), nbytes


def _workspace_arg(workspace, need, device):
    """(workspace tensor, its bytes): the caller's (contiguous, on device; the
    library checks the size) or a new one of `need` bytes."""
    if workspace is None:
        return _workspace(need, device)
    if not workspace.is_cuda or workspace.device != device or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous GPU tensor on %s" % device)
    return workspace, workspace.numel() * workspace.element_size()


def _stream_of(stream):
    import torch
    return stream if stream is not None else torch.cuda.current_stream()


def _stream(stream):
    return ctypes.c_void_p(_stream_of(stream).cuda_stream)


def _keep_alive(stream, *tensors):
    """Tensors allocated here on torch's current stream but used by kernels
    enqueued on another `stream`: mark them as in use on that stream, so the
    caching allocator does not hand their memory out again before those
    kernels finish."""
    import torch
    if stream is None or stream == torch.cuda.current_stream():
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


def gauss_sum_fwd(q, k, v, tau, out=None, workspace=None, stream=None):
    """s = sum_n exp(-tau/2 ||q_m - k_n||^2) v_n (Eq. 1) as an M x C fp32 tensor."""
    import torch
    _check_inputs(q, k, v)
    M, D = q.shape
    N, C = v.shape
    p = make_problem(M, N, D, C, _dtype_code(q.dtype), _dtype_code(v.dtype))
    lib = load()
    out = _output(out, "out", (M, C), q.device)
    need = int(lib.gauss_sum_fwd_workspace_size(ctypes.byref(p)))
    workspace, wbytes = _workspace_arg(workspace, need, q.device)
    st = lib.gauss_sum_fwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), float(tau), _ptr(out),
                           _ptr(workspace), wbytes, _stream(stream))
    _keep_alive(stream, out, workspace)
    if st != 0:
        raise GaussSumError(st, "gauss_sum_fwd")
    return out


def gauss_sum_fwd_noalloc(q, k, v, tau, out, stream=None):
    """gauss_sum_fwd through the entry point that allocates nothing (its
    workspace is the library's built-in scratch array on the current GPU);
    `out` (M x C fp32) is required.  Calls that overlap in time on one GPU
    race; order them on one stream."""
    _check_inputs(q, k, v)
    M, D = q.shape
    N, C = v.shape
    _check_tensor(out, "out", (M, C), q.device, _torch().float32)
    p = make_problem(M, N, D, C, _dtype_code(q.dtype), _dtype_code(v.dtype))
    st = load().gauss_sum_fwd_noalloc(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), float(tau), _ptr(out),
                                      _stream(stream))
    if st != 0:
        raise GaussSumError(st, "gauss_sum_fwd_noalloc")
    return out


def _torch():
    import torch
    return torch


def gauss_sum_bwd(q, k, v, tau, dout, want=(True, True, True), workspace=None, stream=None):
    """Gradients of L = sum dout * s with respect to (q, k, v); None where not wanted."""
    import torch
    _check_inputs(q, k, v)
    M, D = q.shape
    N, C = v.shape
    _check_tensor(dout, "dout", (M, C), q.device)
    p = make_problem(M, N, D, C, _dtype_code(q.dtype), _dtype_code(v.dtype))
    lib = load()
    dev = q.device
    dq = torch.empty((M, D), dtype=torch.float32, device=dev) if want[0] else None
    dk = torch.empty((N, D), dtype=torch.float32, device=dev) if want[1] else None
    dv = torch.empty((N, C), dtype=torch.float32, device=dev) if want[2] else None
    need = int(lib.gauss_sum_bwd_workspace_size(ctypes.byref(p), int(bool(want[0])),
                                                int(bool(want[1])), int(bool(want[2]))))
    workspace, wbytes = _workspace_arg(workspace, need, dev)
    st = lib.gauss_sum_bwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), float(tau), _ptr(dout),
                           _dtype_code(dout.dtype), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace),
                           wbytes, _stream(stream))
    _keep_alive(stream, dq, dk, dv, workspace)
    if st != 0:
        raise GaussSumError(st, "gauss_sum_bwd")
    return dq, dk, dv


def gauss_sum_fwd_bwd(q, k, v, tau, dout, want=(True, True, True), out=None, workspace=None,
                      stream=None):
    """(s, dq, dk, dv) in one call for a known upstream gradient dout; the
    forward sum and dq come from one pass over the pairs."""
    import torch
    _check_inputs(q, k, v)
    M, D = q.shape
    N, C = v.shape
    _check_tensor(dout, "dout", (M, C), q.device)
    p = make_problem(M, N, D, C, _dtype_code(q.dtype), _dtype_code(v.dtype))
    lib = load()
    dev = q.device
    out = _output(out, "out", (M, C), dev)
    dq = torch.empty((M, D), dtype=torch.float32, device=dev) if want[0] else None
    dk = torch.empty((N, D), dtype=torch.float32, device=dev) if want[1] else None
    dv = torch.empty((N, C), dtype=torch.float32, device=dev) if want[2] else None
    need = int(lib.gauss_sum_fwd_bwd_workspace_size(ctypes.byref(p), int(bool(want[0])),
                                                    int(bool(want[1])), int(bool(want[2]))))
    workspace, wbytes = _workspace_arg(workspace, need, dev)
    st = lib.gauss_sum_fwd_bwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), float(tau), _ptr(dout),
                               _dtype_code(dout.dtype), _ptr(out), _ptr(dq), _ptr(dk), _ptr(dv),
                               _ptr(workspace), wbytes, _stream(stream))
    _keep_alive(stream, out, dq, dk, dv, workspace)
    if st != 0:
        raise GaussSumError(st, "gauss_sum_fwd_bwd")
    return out, dq, dk, dv


def _batched_inputs(q, k, v):
    """(B, M, N, D, C, strides) for q: B x M x D, k: B x N x D or N x D (shared),
    v: B x N x C or N x C (shared); contiguous GPU tensors."""
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not t.is_contiguous():
            raise ValueError("%s must be a contiguous tensor" % name)
    if q.dim() != 3:
        raise ValueError("q must be B x M x D")
    B, M, D = q.shape
    if k.dim() not in (2, 3) or v.dim() not in (2, 3) or k.shape[-1] != D:
        raise ValueError("k must be [B x] N x D and v [B x] N x C")
    N, C = v.shape[-2], v.shape[-1]
    if k.shape[-2] != N or (k.dim() == 3 and k.shape[0] != B) or (v.dim() == 3 and v.shape[0] != B):
        raise ValueError("inconsistent batch shapes")
    if q.dtype != k.dtype:
        raise TypeError("q and k must share a dtype")
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not t.is_cuda:
            raise ValueError("%s must be a GPU tensor" % name)
    if k.device != q.device or v.device != q.device:
        raise ValueError("q, k and v must be on one device")
    ks = N * D if k.dim() == 3 else 0
    vs = N * C if v.dim() == 3 else 0
    return B, M, N, D, C, M * D, ks, vs


def gauss_sum_fwd_batched_workspace_size(M, N, D, C, count, qk_dtype=GS_F16, v_dtype=GS_F32):
    p = make_problem(M, N, D, C, qk_dtype, v_dtype)
    return int(load().gauss_sum_fwd_batched_workspace_size(ctypes.byref(p), int(count)))


def gauss_sum_bwd_batched_workspace_size(M, N, D, C, count, qk_dtype=GS_F16, v_dtype=GS_F32,
                                         want_dq=True, want_dk=True, want_dv=True):
    p = make_problem(M, N, D, C, qk_dtype, v_dtype)
    return int(load().gauss_sum_bwd_batched_workspace_size(ctypes.byref(p), int(count), int(bool(want_dq)),
                                                           int(bool(want_dk)), int(bool(want_dv))))


def gauss_sum_fwd_batched(q, k, v, tau, out=None, workspace=None, stream=None, group=None):
    """B independent forward sums: q is B x M x D, k and v are B x N x (D, C)
    or shared N x (D, C); returns B x M x C fp32.  Without a workspace, one is
    allocated for `group` problems per launch (default: all B)."""
    import torch
    B, M, N, D, C, qs, ks, vs = _batched_inputs(q, k, v)
    p = make_problem(M, N, D, C, _dtype_code(q.dtype), _dtype_code(v.dtype))
    lib = load()
    out = _output(out, "out", (B, M, C), q.device)
    b = Batch(B, qs, ks, vs, 0, M * C, 0, 0, 0)
    need = int(lib.gauss_sum_fwd_batched_workspace_size(ctypes.byref(p), int(group or max(B, 1))))
    workspace, wbytes = _workspace_arg(workspace, need, q.device)
    st = lib.gauss_sum_fwd_batched(ctypes.byref(p), ctypes.byref(b), _ptr(q), _ptr(k), _ptr(v),
                                   float(tau), _ptr(out), _ptr(workspace), wbytes, _stream(stream))
    _keep_alive(stream, out, workspace)
    if st != 0:
        raise GaussSumError(st, "gauss_sum_fwd_batched")
    return out


def gauss_sum_bwd_batched(q, k, v, tau, dout, want=(True, True, True), workspace=None, stream=None,
                          group=None):
    """Gradients of B independent problems (q, k shared as in
    gauss_sum_fwd_batched; dout is B x M x C); each output B x (rows) x (D or C).
    Without a workspace, one is allocated for `group` problems per launch
    (default: all B)."""
    import torch
    B, M, N, D, C, qs, ks, vs = _batched_inputs(q, k, v)
    _check_tensor(dout, "dout", (B, M, C), q.device)
    if (want[1] and ks == 0) or (want[2] and vs == 0):
        raise ValueError("dk / dv of a shared key set: sum the per-problem gradients instead")
    p = make_problem(M, N, D, C, _dtype_code(q.dtype), _dtype_code(v.dtype))
    lib = load()
    dev = q.device
    dq = torch.empty((B, M, D), dtype=torch.float32, device=dev) if want[0] else None
    dk = torch.empty((B, N, D), dtype=torch.float32, device=dev) if want[1] else None
    dv = torch.empty((B, N, C), dtype=torch.float32, device=dev) if want[2] else None
    b = Batch(B, qs, ks, vs, M * C, 0, M * D, N * D, N * C)
    need = int(lib.gauss_sum_bwd_batched_workspace_size(ctypes.byref(p), int(group or max(B, 1)),
                                                        int(bool(want[0])), int(bool(want[1])),
                                                        int(bool(want[2]))))
    workspace, wbytes = _workspace_arg(workspace, need, dev)
    st = lib.gauss_sum_bwd_batched(ctypes.byref(p), ctypes.byref(b), _ptr(q), _ptr(k), _ptr(v),
                                   float(tau), _ptr(dout), _dtype_code(dout.dtype), _ptr(dq), _ptr(dk),
                                   _ptr(dv), _ptr(workspace), wbytes, _stream(stream))
    _keep_alive(stream, dq, dk, dv, workspace)
    if st != 0:
        raise GaussSumError(st, "gauss_sum_bwd_batched")
    return dq, dk, dv


def gauss_sum_fwd_bwd_batched_workspace_size(M, N, D, C, count, qk_dtype=GS_F16, v_dtype=GS_F32,
                                             want_dq=True, want_dk=True, want_dv=True):
    p = make_problem(M, N, D, C, qk_dtype, v_dtype)
    return int(load().gauss_sum_fwd_bwd_batched_workspace_size(ctypes.byref(p), int(count),
                                                               int(bool(want_dq)), int(bool(want_dk)),
                                                               int(bool(want_dv))))


def gauss_sum_fwd_bwd_batched(q, k, v, tau, dout, want=(True, True, True), out=None, workspace=None,
                              stream=None, group=None):
    """(s, dq, dk, dv) of B independent problems in one call (shapes as in
    gauss_sum_bwd_batched; s is B x M x C); the forward sums ride along in the
    dq passes where gauss_sum_fwd_bwd fuses them."""
    import torch
    B, M, N, D, C, qs, ks, vs = _batched_inputs(q, k, v)
    _check_tensor(dout, "dout", (B, M, C), q.device)
    if (want[1] and ks == 0) or (want[2] and vs == 0):
        raise ValueError("dk / dv of a shared key set: sum the per-problem gradients instead")
    p = make_problem(M, N, D, C, _dtype_code(q.dtype), _dtype_code(v.dtype))
    lib = load()
    dev = q.device
    out = _output(out, "out", (B, M, C), dev)
    dq = torch.empty((B, M, D), dtype=torch.float32, device=dev) if want[0] else None
    dk = torch.empty((B, N, D), dtype=torch.float32, device=dev) if want[1] else None
    dv = torch.empty((B, N, C), dtype=torch.float32, device=dev) if want[2] else None
    b = Batch(B, qs, ks, vs, M * C, M * C, M * D, N * D, N * C)
    need = int(lib.gauss_sum_fwd_bwd_batched_workspace_size(ctypes.byref(p), int(group or max(B, 1)),
                                                            int(bool(want[0])), int(bool(want[1])),
                                                            int(bool(want[2]))))
    workspace, wbytes = _workspace_arg(workspace, need, dev)
    st = lib.gauss_sum_fwd_bwd_batched(ctypes.byref(p), ctypes.byref(b), _ptr(q), _ptr(k), _ptr(v),
                                       float(tau), _ptr(dout), _dtype_code(dout.dtype), _ptr(out),
                                       _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), wbytes,
                                       _stream(stream))
    _keep_alive(stream, out, dq, dk, dv, workspace)
    if st != 0:
        raise GaussSumError(st, "gauss_sum_fwd_bwd_batched")
    return out, dq, dk, dv


def gauss_sum_mmd_flow_workspace_size(N, D, qk_dtype=GS_F16, v_dtype=GS_F32):
    p = make_problem(N, N, D, 1, qk_dtype, v_dtype)
    return int(load().gauss_sum_mmd_flow_workspace_size(ctypes.byref(p)))


def gauss_sum_mmd_flow(x, v, tau, want=(True, True, True), workspace=None, stream=None):
    """One MMD-flow evaluation for points x (N x D) and signed weights v (N x 1):
    (s, grad, mmd2) with s = K v, grad[m] = tau (sum_n Phi v_n x_n - x_m s_m)
    and mmd2 = v^T s (a 0-d fp64 tensor); None where not wanted."""
    import torch
    _check_inputs(x, x, v)
    N, D = x.shape
    if tuple(v.shape) != (N, 1):
        raise ValueError("v must be N x 1")
    p = make_problem(N, N, D, 1, _dtype_code(x.dtype), _dtype_code(v.dtype))
    lib = load()
    dev = x.device
    s = torch.empty((N, 1), dtype=torch.float32, device=dev) if want[0] else None
    grad = torch.empty((N, D), dtype=torch.float32, device=dev) if want[1] else None
    mmd2 = torch.empty((), dtype=torch.float64, device=dev) if want[2] else None
    need = int(lib.gauss_sum_mmd_flow_workspace_size(ctypes.byref(p)))
    workspace, wbytes = _workspace_arg(workspace, need, dev)
    st = lib.gauss_sum_mmd_flow(ctypes.byref(p), _ptr(x), _ptr(v), float(tau), _ptr(s), _ptr(grad),
                                _ptr(mmd2), _ptr(workspace), wbytes, _stream(stream))
    _keep_alive(stream, s, grad, mmd2, workspace)
    if st != 0:
        raise GaussSumError(st, "gauss_sum_mmd_flow")
    return s, grad, mmd2


def gauss_sum_svgd_workspace_size(N, D, qk_dtype=GS_F16, v_dtype=GS_F32):
    p = make_problem(N, N, D, D, qk_dtype, v_dtype)
    return int(load().gauss_sum_svgd_workspace_size(ctypes.byref(p)))


def gauss_sum_svgd(x, score, tau, out=None, workspace=None, stream=None):
    """One SVGD update direction (without the 1/N factor) for particles x
    (N x D) and scores score = grad log p(x) (N x D):
    phi[m] = sum_n Phi(x_m, x_n) score_n + tau sum_n Phi(x_m, x_n) (x_m - x_n)."""
    import torch
    _check_inputs(x, x, score)
    N, D = x.shape
    if tuple(score.shape) != (N, D):
        raise ValueError("score must be N x D")
    p = make_problem(N, N, D, D, _dtype_code(x.dtype), _dtype_code(score.dtype))
    lib = load()
    dev = x.device
    out = _output(out, "out", (N, D), dev)
    need = int(lib.gauss_sum_svgd_workspace_size(ctypes.byref(p)))
    workspace, wbytes = _workspace_arg(workspace, need, dev)
    st = lib.gauss_sum_svgd(ctypes.byref(p), _ptr(x), _ptr(score), float(tau), _ptr(out), _ptr(workspace),
                            wbytes, _stream(stream))
    _keep_alive(stream, out, workspace)
    if st != 0:
        raise GaussSumError(st, "gauss_sum_svgd")
    return out


def _make_autograd():
    import torch

    class GaussSum(torch.autograd.Function):
        """s = GaussSum.apply(q, k, v, tau); gradients for q, k and v."""

        @staticmethod
        def forward(ctx, q, k, v, tau):
            ctx.save_for_backward(q, k, v)
            ctx.tau = float(tau)
            return gauss_sum_fwd(q, k, v, tau)

        @staticmethod
        def backward(ctx, g):
            q, k, v = ctx.saved_tensors
            want = ctx.needs_input_grad[:3]
            if not any(want):
                return None, None, None, None
            dq, dk, dv = gauss_sum_bwd(q, k, v, ctx.tau, g.contiguous(), want=want)
            cast = lambda x, ref: None if x is None else x.to(ref.dtype)  # noqa: E731
            return cast(dq, q), cast(dk, k), cast(dv, v), None

    return GaussSum


class _Lazy:
    def __init__(self):
        self._cls = None

    def __getattr__(self, name):
        if self._cls is None:
            self._cls = _make_autograd()
        return getattr(self._cls, name)


GaussSum = _Lazy()
