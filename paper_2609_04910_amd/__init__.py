"""Exact Gauss sums on MI355X (gfx950): s_m = sum_n exp(-tau/2 ||q_m - k_n||^2) v_n
and its gradients, computed by hand-written HIP kernels behind the C ABI
declared in ``include/gauss_sum.h`` (paper "Fast Gauss Sums via Flash
Attention", Eq. 1 and the Sec. 3 gradient).

``paper_2609_04910_amd.gauss_sum`` is the thin ctypes binding; importing this
package does not load the GPU library.
"""
__all__ = ["gauss_sum", "workloads"]
