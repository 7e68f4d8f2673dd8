/*
 * gauss_sum.h -- C ABI of the MI355X (gfx950) exact Gauss-sum library.
 *
 * The library evaluates, for points q_1..q_M, k_1..k_N in R^D, values
 * v_1..v_N in R^C and bandwidth tau > 0, the Gauss sum
 *
 *     s_m = sum_n exp(-tau/2 ||q_m - k_n||^2) v_n ,   m = 1..M
 *
 * (paper "Fast Gauss Sums via Flash Attention", Sec. 1, Eq. 1; the inputs and
 * outputs follow the input/output lines of Alg. 1 and Alg. 2), and the
 * gradients of L = sum_{m,c} dout[m,c] s[m,c] with respect to q, k and v
 * (the query gradient is the Sec. 3 gradient equation used by MMD flows and
 * SVGD; the key gradient is its mirror image; L is linear in v).
 *
 * Memory and ownership
 *   - Every data pointer is a DEVICE pointer owned by the caller.  All arrays
 *     are dense, row-major and contiguous: q is M x D, k is N x D, v is N x C,
 *     dout and out are M x C, dq is M x D, dk is N x D, dv is N x C.
 *   - Each pointer must be aligned to its element size; the workspace to 256
 *     bytes.
 *   - q and k may be the same array (M == N), as in MMD and SVGD.  Outputs
 *     must not overlap any input, the workspace or each other.
 *   - The library allocates nothing.  The caller provides a device workspace
 *     of at least the size returned by the *_workspace_size query; its
 *     contents on entry are ignored and on exit undefined.
 *
 * Execution
 *   - All work is enqueued on `stream` (NULL = the default stream) and runs
 *     asynchronously; the returned status covers argument validation and
 *     kernel launches only.  No call synchronises with the device.
 *   - Arguments are validated before anything is enqueued: on any error
 *     status no kernel has been launched and no output was touched.
 *   - Inputs must stay valid until the enqueued work completes.  Calls on
 *     different streams may overlap only if their workspaces are disjoint.
 *   - Results are deterministic: the same inputs give bitwise identical
 *     outputs on every run (fixed summation order, no atomics on data).
 *   - NaN or Inf inside the data propagate; they are not checked.
 *
 * Precision
 *   - q, k: fp16 or bf16.  v, dout: fp32, fp16 or bf16.  Outputs: fp32.
 *   - Dot products q.k use fp16/bf16 matrix cores with fp32 accumulation; the
 *     exponent tau*q.k - tau/2||q||^2 - tau/2||k||^2 is formed in fp32 and
 *     clamped at <= 0; kernel values and values are contracted in fp16 with
 *     fp32 accumulation after exact power-of-two scaling.  Each result is
 *     within 2e-3 (fp16 q,k) or 5e-3 (bf16 q,k) of sum_n Phi |v_n| per element
 *     of the exact value (and the analogous sums of |terms| for gradients).
 *   - Domain of that bound: tau * ||q_m||^2 and tau * ||k_n||^2 at most 2^13
 *     for all rows.  The fp32 exponent is formed from the expanded square, and
 *     its rounding error grows as about tau * ||x||^2 * 2^-24 (relative error
 *     of the result about 2.5e-4 at the limit, measured 6e-4 at 2.4 times
 *     it).  Point sets far from the origin compared with their spread should
 *     be centred on a common point by the caller first: Eq. 1 and its
 *     gradients are invariant under a common translation of q and k (the
 *     centring of Sec. 2, Remark 2).
 */
#ifndef GAUSS_SUM_H
#define GAUSS_SUM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GAUSS_SUM_ABI_VERSION 1
#define GAUSS_SUM_MAX_DIM 256 /* largest D and C accepted */

typedef enum { GS_F32 = 0, GS_F16 = 1, GS_BF16 = 2 } gs_dtype;

typedef enum {
  GS_SUCCESS = 0,
  GS_ERR_NULL_POINTER = 1, /* a required pointer is NULL, or no output requested */
  GS_ERR_BAD_SHAPE = 2,    /* M or N outside [0, 2^30], D or C outside [1, 256] */
  GS_ERR_BAD_TAU = 3,      /* tau not finite or not > 0 (Eq. 1 needs tau > 0) */
  GS_ERR_UNSUPPORTED = 4,  /* dtype combination not supported */
  GS_ERR_MISALIGNED = 5,   /* pointer not aligned as documented above */
  GS_ERR_WORKSPACE = 6,    /* workspace NULL or smaller than required */
  GS_ERR_HIP = 7,          /* a HIP runtime call or kernel launch failed */
  GS_ERR_INTERNAL = 8,     /* unexpected internal failure */
  GS_ERR_ALIAS = 9,        /* an output overlaps an input or another output */
  GS_ERR_SCRATCH_LIMIT = 10 /* gauss_sum_fwd_noalloc: the problem needs more scratch than
                               GAUSS_SUM_NOALLOC_SCRATCH_BYTES */
} gs_status;

/* Problem description.  qk_dtype: GS_F16 or GS_BF16 (both q and k), or
 * GS_F32 for the fp32-accuracy tier (the single-precision setting of App.
 * A.2): the forward sum (gauss_sum_fwd, gauss_sum_fwd_batched), error per
 * output about one fp32 ulp of sum_n Phi |v_nc| for exponents of order one;
 * the gradient calls and gauss_sum_mmd_flow return GS_ERR_UNSUPPORTED for
 * fp32 points (workspace sizes 0).  Points are aligned to their element size
 * (2 or 4 bytes).
 * v_dtype: GS_F32, GS_F16 or GS_BF16. */
typedef struct {
  int64_t M, N, D, C;
  int32_t qk_dtype; /* a gs_dtype value (an int field: any other value is rejected, not undefined) */
  int32_t v_dtype;  /* a gs_dtype value */
} gs_problem;

/* Bytes of device workspace gauss_sum_fwd needs for problem p (0 if p is
 * invalid or NULL). */
size_t gauss_sum_fwd_workspace_size(const gs_problem* p);

/* Bytes of device workspace gauss_sum_bwd needs for problem p and the
 * requested gradients (flags nonzero = requested; 0 if p is invalid). */
size_t gauss_sum_bwd_workspace_size(const gs_problem* p, int want_dq, int want_dk, int want_dv);

/* Forward, Eq. 1: out[m,c] = s_m[c] for m < M, c < C (fp32, overwritten).
 * M == 0 is a no-op; N == 0 writes zeros. */
gs_status gauss_sum_fwd(const gs_problem* p, const void* q, const void* k, const void* v, float tau,
                        float* out, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Largest workspace gauss_sum_fwd_noalloc can serve from its built-in
 * scratch array (128 MiB per GPU). */
#define GAUSS_SUM_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/* gauss_sum_fwd without a workspace argument and without any allocation,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  Same
 * arguments, validation and results as gauss_sum_fwd (bitwise: the same
 * kernels and launch plan); the workspace is a file-scope device array of
 * the library, GAUSS_SUM_NOALLOC_SCRATCH_BYTES bytes on every GPU the call
 * is made on, held until the process ends.  Returns GS_ERR_SCRATCH_LIMIT
 * (nothing launched) when gauss_sum_fwd_workspace_size(p) exceeds that size.
 * Every call on one GPU uses the same array: calls that may overlap in time
 * on one GPU (different streams without ordering, other host threads) race
 * and give undefined results; order them on one stream.  The first call on
 * a GPU looks up the array's device address (no allocation); every call
 * overwrites what it uses of the array before reading it. */
gs_status gauss_sum_fwd_noalloc(const gs_problem* p, const void* q, const void* k, const void* v,
                                float tau, float* out, hipStream_t stream);

/* Backward: for L = sum_{m,c} dout[m,c] s[m,c] (dout: M x C of dout_dtype,
 * GS_F32, GS_F16 or GS_BF16) writes
 *   dq[m,:] = tau sum_n Phi_mn <dout_m, v_n> (k_n - q_m)   (Sec. 3 gradient)
 *   dk[n,:] = tau sum_m Phi_mn <dout_m, v_n> (q_m - k_n)
 *   dv[n,:] =     sum_m Phi_mn dout_m
 * Any of dq, dk, dv may be NULL (not computed); at least one must be given.
 * Outputs are fp32 and overwritten. */
gs_status gauss_sum_bwd(const gs_problem* p, const void* q, const void* k, const void* v, float tau,
                        const void* dout, int dout_dtype, float* dq, float* dk, float* dv,
                        void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Forward and backward in one call: writes out (as gauss_sum_fwd, required)
 * and any of dq, dk, dv (as gauss_sum_bwd, NULL = not requested) for the
 * given upstream gradient dout.  Sec. 3 of the paper observes that the query
 * gradient is itself one kernel sum over the same pairs (values (v_n k_n,
 * v_n)); with dq requested and C <= 16, the forward sum is produced by the
 * same pass that computes dq, so the kernel values are evaluated once for
 * both (and with dk and dv requested, dv likewise rides in the dk pass; wider
 * values get passes of their own).  Meant for
 * callers that know dout before the forward result (MMD flows use dout = v).
 * Results equal those of separate gauss_sum_fwd and gauss_sum_bwd calls to
 * within the stated tolerance. */
gs_status gauss_sum_fwd_bwd(const gs_problem* p, const void* q, const void* k, const void* v,
                            float tau, const void* dout, int dout_dtype, float* out, float* dq,
                            float* dk, float* dv, void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/* Bytes of device workspace gauss_sum_fwd_bwd needs (0 if p is invalid). */
size_t gauss_sum_fwd_bwd_workspace_size(const gs_problem* p, int want_dq, int want_dk, int want_dv);

/* A batch of `count` independent problems of one shape p (the paper's
 * benchmark evaluates B point clouds at once, Sec. 4).  Problem b reads
 * q + b*q_stride, k + b*k_stride, v + b*v_stride, dout + b*dout_stride and
 * writes out + b*out_stride, dq + b*dq_stride, dk + b*dk_stride,
 * dv + b*dv_stride; strides count elements of each array's own dtype.  Input
 * strides may be 0 (all problems share that array, e.g. one key set); output
 * strides must be at least one problem's output size when count > 1.  Every
 * stride keeps the alignment rules of the single-problem call. */
typedef struct {
  int64_t count;
  int64_t q_stride, k_stride, v_stride, dout_stride;
  int64_t out_stride, dq_stride, dk_stride, dv_stride;
} gs_batch;

/* gauss_sum_fwd for each problem of the batch.  All validation (shapes,
 * strides, alignment, overlaps of any output with any input, the workspace or
 * another output) happens before anything is enqueued; count == 0 is a no-op
 * (no pointer is used).
 *
 * The problems run in launch groups on `stream`: every kernel launch covers
 * a whole group (one grid dimension indexes the problem), each problem of the
 * group using its own slice of the workspace.  The workspace must hold at
 * least one slice, gauss_sum_fwd_workspace_size(p) bytes (then the problems
 * run one at a time); gauss_sum_fwd_batched_workspace_size(p, count) bytes
 * let all of them (up to 65535) share each launch, and any size in between
 * gives groups of as many problems as fit.  Group sizes change how the key
 * range of a problem is split (and so the fp32 summation order): results are
 * reproducible bit for bit for equal arguments, and within the tolerance of
 * the single-problem call otherwise. */
gs_status gauss_sum_fwd_batched(const gs_problem* p, const gs_batch* batch, const void* q,
                                const void* k, const void* v, float tau, float* out,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for gauss_sum_fwd_batched to run `count` problems of shape
 * p in one launch group (count capped at 65535); 0 if p is invalid, empty or
 * count < 1. */
size_t gauss_sum_fwd_batched_workspace_size(const gs_problem* p, int64_t count);

/* gauss_sum_bwd for each problem of the batch (as gauss_sum_fwd_batched; one
 * slice is gauss_sum_bwd_workspace_size(p, ...) bytes). */
gs_status gauss_sum_bwd_batched(const gs_problem* p, const gs_batch* batch, const void* q,
                                const void* k, const void* v, float tau, const void* dout,
                                int dout_dtype, float* dq, float* dk, float* dv,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for gauss_sum_bwd_batched to run `count` problems in one
 * launch group (as gauss_sum_fwd_batched_workspace_size). */
size_t gauss_sum_bwd_batched_workspace_size(const gs_problem* p, int64_t count, int want_dq,
                                            int want_dk, int want_dv);

/* gauss_sum_fwd_bwd for each problem of the batch (as gauss_sum_fwd_batched;
 * the forward sum rides along in the dq pass where gauss_sum_fwd_bwd fuses
 * it; one slice is gauss_sum_fwd_bwd_workspace_size(p, ...) bytes).  This is
 * the layout of the paper's forward-plus-backward benchmark (Sec. 4, the
 * N sweep with B = 4 clouds). */
gs_status gauss_sum_fwd_bwd_batched(const gs_problem* p, const gs_batch* batch, const void* q,
                                    const void* k, const void* v, float tau, const void* dout,
                                    int dout_dtype, float* out, float* dq, float* dk, float* dv,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for gauss_sum_fwd_bwd_batched to run `count` problems in
 * one launch group (as gauss_sum_fwd_batched_workspace_size). */
size_t gauss_sum_fwd_bwd_batched_workspace_size(const gs_problem* p, int64_t count, int want_dq,
                                                int want_dk, int want_dv);

/* One MMD-flow evaluation (Sec. 3, the MMD and particle-flow paragraphs):
 * points x (N x D, qk_dtype) serve as both queries and keys, v (N x 1,
 * v_dtype) are the signed weights of sigma = mu - nu = sum_n v_n delta_{x_n}.
 * Writes, for m < N,
 *   s[m]       = sum_n Phi(x_m, x_n) v_n                      (fp32, N x 1)
 *   grad[m, :] = tau (sum_n Phi v_n x_n - x_m s[m])           (fp32, N x D)
 *              = the gradient of s_m with respect to its query point x_m
 *                (the MMD-flow / SVGD kernel-term velocity),
 *   *mmd2      = sum_m v_m s[m] = MMD_tau(mu, nu)^2            (fp64 scalar)
 * from one pass over the pairs (the forward sum is the gradient pass's own
 * row sum); the inner product is a fixed-order fp64 reduction, so *mmd2 is
 * bitwise reproducible.  Any of s, grad, mmd2 may be NULL (not wanted); at
 * least one must be given.  All pointers are device pointers; mmd2 points to
 * one double (8-byte aligned).  Requires p->M == p->N (GS_ERR_BAD_SHAPE) and
 * p->C == 1 (GS_ERR_UNSUPPORTED); other checks as gauss_sum_fwd_bwd.  N == 0
 * writes *mmd2 = 0.  Workspace: gauss_sum_mmd_flow_workspace_size. */
gs_status gauss_sum_mmd_flow(const gs_problem* p, const void* x, const void* v, float tau, float* s,
                             float* grad, double* mmd2, void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* Bytes of device workspace gauss_sum_mmd_flow needs (0 if p is invalid for it). */
size_t gauss_sum_mmd_flow_workspace_size(const gs_problem* p);

/* One Stein variational gradient descent update (Sec. 3, the MMD-flow and
 * SVGD paragraph: the kernel part of the SVGD direction has the same form as
 * the query gradient): particles x (N x D, qk_dtype) and the scores
 * score_n = grad log p(x_n) (N x D, v_dtype) give, for m < N,
 *   phi[m, :] = sum_n Phi(x_m, x_n) score_n + tau sum_n Phi(x_m, x_n) (x_m - x_n)
 * (fp32, N x D), the SVGD direction without its 1/N factor (the second sum is
 * the gradient of sum_n Phi(x_n, x_m) with respect to x_n, summed: the
 * repulsive term).  One pass over the pairs: the kernel values are formed
 * once and feed both the sum with values score and the query gradient with
 * unit weights (their difference is written).  Requires p->M == p->N and
 * p->C == p->D (GS_ERR_BAD_SHAPE); fp16 or bf16 points.  phi must not overlap
 * x, score or the workspace.  N == 0 is a no-op.  Workspace:
 * gauss_sum_svgd_workspace_size. */
gs_status gauss_sum_svgd(const gs_problem* p, const void* x, const void* score, float tau, float* phi,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for gauss_sum_svgd; 0 if p does not describe an SVGD
 * update (M != N, C != D, invalid, or fp32 points) or N == 0. */
size_t gauss_sum_svgd_workspace_size(const gs_problem* p);

/* Static, never-NULL description of a status code (any int: codes outside
 * gs_status give "unknown status"). */
const char* gauss_sum_status_string(int status);

/* GAUSS_SUM_ABI_VERSION of the built library. */
int gauss_sum_abi_version(void);

/* Kernel timing hook for benchmarks and profiling; not needed to compute.
 * gauss_sum_profile_start(capacity, kind) creates 2*capacity HIP events on
 * the current device; afterwards each launch of a main kernel selected by
 * `kind` (1 = forward-type kernels, 2 = gradient-type kernels, 3 = both),
 * across all following calls, is bracketed by a pair of events recorded on
 * the call's stream, until capacity launches are recorded.
 * gauss_sum_profile_stop(ms, max) waits for those events, writes up to `max`
 * per-launch durations in milliseconds (host array) and returns how many
 * launches were recorded (negative on a HIP error); it releases the events.
 * Status: GS_ERR_BAD_SHAPE for capacity < 1 or kind outside 1..3, GS_ERR_HIP
 * if events cannot be created.  The hook is process-global and not
 * thread-safe: use it from one thread while no other thread calls the
 * library. */
gs_status gauss_sum_profile_start(int capacity, int kind);
int gauss_sum_profile_stop(float* ms, int max);

#ifdef __cplusplus
}
#endif

#endif /* GAUSS_SUM_H */
