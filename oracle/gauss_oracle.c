/*
 * gauss_oracle.c -- plain, slow, obviously correct fp64 CPU oracle for the
 * exact Gauss sum and its gradients.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The GPU library never
 * links, calls or includes anything from here, and this file includes nothing
 * from the GPU library: the two share no code.
 *
 * What is computed (paper "Fast Gauss Sums via Flash Attention"):
 *
 *   Gauss kernel   Phi(q,k) = exp(-tau/2 * ||q - k||^2)            (Sec. 1, Eq. 1)
 *   Gauss sum      s_m      = sum_n Phi(q_m, k_n) v_n               (Sec. 1, Eq. 1)
 *   query gradient grad_{q_m} s_m = tau * sum_n Phi v_n (k_n - q_m)  (Sec. 3, MMD
 *                  flows / SVGD gradient equation)
 *
 * For a scalar loss L = sum_{m,c} g[m,c] s[m,c] (g = upstream gradient) the
 * chain rule applied to Eq. 1 gives, with w_mn = sum_c g[m,c] v[n,c]:
 *
 *   dq[m,:] = tau * sum_n Phi_mn w_mn (k_n - q_m)      (Sec. 3 gradient, C >= 1)
 *   dk[n,:] = tau * sum_m Phi_mn w_mn (q_m - k_n)      (same, differentiating k_n)
 *   dv[n,:] =       sum_m Phi_mn g_m                   (Eq. 1 is linear in v)
 *
 * Every function evaluates these definitions literally: a double loop, the
 * squared distance in difference form sum_d (q_d - k_d)^2, exp() from libm,
 * all arithmetic in fp64.  Alongside each result it returns the sum of the
 * absolute values of its terms, the scale against which a reduced-precision
 * result is judged: A = sum_n Phi |v_n| for the sum, and for the q and k
 * gradients, which are double sums over (n, c) of tau Phi g_c v_c (k - q),
 * tau sum Phi (sum_c |g_c v_c|) |k - q|.  The *_scales variants of the q and k
 * gradients also return the net scale tau sum Phi |sum_c g_c v_c| |k - q|, in
 * which the C terms of each w are summed before the magnitude is taken (the
 * other reading of the gradient tolerance, at most the first).
 *
 * Parallelism: output rows are independent; rows are split into contiguous
 * chunks over POSIX threads.  Each row is summed by one thread in index
 * order, so results do not depend on the thread count.
 *
 * Status codes: 0 ok, 1 bad argument (null pointer with nonzero size,
 * negative size), 2 thread creation failure.
 */
#include <math.h>
#include <pthread.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

#define ORACLE_MAX_THREADS 256

enum { OP_FWD = 0, OP_DQ = 1, OP_DK = 2, OP_DV = 3 };

typedef struct {
  int op;
  int64_t M, N, D, C;
  const double *q, *k, *v, *g;
  double tau;
  const int64_t* rows; /* selected output rows, or NULL for 0..nrows-1 */
  int64_t row_begin, row_end;
  double *out, *absout;
  double* netout; /* q / k gradients: tau sum Phi |w| |k - q|, or NULL */
} job_t;

/* Phi(a, b) = exp(-tau/2 * sum_d (a_d - b_d)^2): Eq. 1, difference form. */
static double phi(const double* a, const double* b, int64_t D, double tau) {
  double d2 = 0.0;
  for (int64_t d = 0; d < D; ++d) {
    double t = a[d] - b[d];
    d2 += t * t;
  }
  return exp(-0.5 * tau * d2);
}

/* w = sum_c g[m,c] v[n,c]: the upstream gradient contracted with a value. */
static double dotc(const double* gm, const double* vn, int64_t C) {
  double w = 0.0;
  for (int64_t c = 0; c < C; ++c) w += gm[c] * vn[c];
  return w;
}

/* sum_c |g[m,c] v[n,c]|: the magnitude of the C terms that make up w. */
static double absdotc(const double* gm, const double* vn, int64_t C) {
  double w = 0.0;
  for (int64_t c = 0; c < C; ++c) w += fabs(gm[c] * vn[c]);
  return w;
}

/* s_m and A_m = sum_n Phi |v_n| for one query row m (Eq. 1). */
static void fwd_row(const job_t* j, int64_t m, double* o, double* a) {
  const double* qm = j->q + m * j->D;
  for (int64_t c = 0; c < j->C; ++c) { o[c] = 0.0; a[c] = 0.0; }
  for (int64_t n = 0; n < j->N; ++n) {
    const double* vn = j->v + n * j->C;
    double p = phi(qm, j->k + n * j->D, j->D, j->tau);
    for (int64_t c = 0; c < j->C; ++c) {
      o[c] += p * vn[c];
      a[c] += p * fabs(vn[c]);
    }
  }
}

/* dq_m = tau sum_n Phi w (k_n - q_m) (Sec. 3 query-gradient equation with
 * values contracted against g_m).  As a double sum over (n, c) its terms are
 * tau Phi g_mc v_nc (k_n - q_m), so the scale is
 * Aq = tau sum_n Phi (sum_c |g_mc v_nc|) |k_n - q_m|. */
static void dq_row(const job_t* j, int64_t m, double* o, double* a, double* nt) {
  const double* qm = j->q + m * j->D;
  const double* gm = j->g + m * j->C;
  for (int64_t d = 0; d < j->D; ++d) { o[d] = 0.0; a[d] = 0.0; if (nt) nt[d] = 0.0; }
  for (int64_t n = 0; n < j->N; ++n) {
    const double* kn = j->k + n * j->D;
    double p = phi(qm, kn, j->D, j->tau);
    double w = dotc(gm, j->v + n * j->C, j->C);
    double wa = absdotc(gm, j->v + n * j->C, j->C);
    for (int64_t d = 0; d < j->D; ++d) {
      double diff = kn[d] - qm[d];
      o[d] += j->tau * p * w * diff;
      a[d] += j->tau * p * wa * fabs(diff);
      if (nt) nt[d] += j->tau * p * fabs(w) * fabs(diff);
    }
  }
}

/* dk_n = tau sum_m Phi w (q_m - k_n) and its scale
 * Ak = tau sum_m Phi (sum_c |g_mc v_nc|) |q_m - k_n|. */
static void dk_row(const job_t* j, int64_t n, double* o, double* a, double* nt) {
  const double* kn = j->k + n * j->D;
  const double* vn = j->v + n * j->C;
  for (int64_t d = 0; d < j->D; ++d) { o[d] = 0.0; a[d] = 0.0; if (nt) nt[d] = 0.0; }
  for (int64_t m = 0; m < j->M; ++m) {
    const double* qm = j->q + m * j->D;
    double p = phi(qm, kn, j->D, j->tau);
    double w = dotc(j->g + m * j->C, vn, j->C);
    double wa = absdotc(j->g + m * j->C, vn, j->C);
    for (int64_t d = 0; d < j->D; ++d) {
      double diff = qm[d] - kn[d];
      o[d] += j->tau * p * w * diff;
      a[d] += j->tau * p * wa * fabs(diff);
      if (nt) nt[d] += j->tau * p * fabs(w) * fabs(diff);
    }
  }
}

/* dv_n = sum_m Phi g_m and Av = sum_m Phi |g_m|. */
static void dv_row(const job_t* j, int64_t n, double* o, double* a) {
  const double* kn = j->k + n * j->D;
  for (int64_t c = 0; c < j->C; ++c) { o[c] = 0.0; a[c] = 0.0; }
  for (int64_t m = 0; m < j->M; ++m) {
    const double* gm = j->g + m * j->C;
    double p = phi(j->q + m * j->D, kn, j->D, j->tau);
    for (int64_t c = 0; c < j->C; ++c) {
      o[c] += p * gm[c];
      a[c] += p * fabs(gm[c]);
    }
  }
}

static void* run_job(void* arg) {
  const job_t* j = (const job_t*)arg;
  int64_t width = (j->op == OP_FWD || j->op == OP_DV) ? j->C : j->D;
  for (int64_t r = j->row_begin; r < j->row_end; ++r) {
    int64_t row = j->rows ? j->rows[r] : r;
    double* o = j->out + r * width;
    double* a = j->absout + r * width;
    double* nt = j->netout ? j->netout + r * width : NULL;
    switch (j->op) {
      case OP_FWD: fwd_row(j, row, o, a); break;
      case OP_DQ: dq_row(j, row, o, a, nt); break;
      case OP_DK: dk_row(j, row, o, a, nt); break;
      default: dv_row(j, row, o, a); break;
    }
  }
  return NULL;
}

static int dispatch(job_t base, int64_t nrows, int nthreads) {
  if (base.M < 0 || base.N < 0 || base.D < 1 || base.C < 1 || nrows < 0) return 1;
  if (!base.out || !base.absout) return nrows ? 1 : 0;
  if ((base.M && !base.q) || (base.N && (!base.k || !base.v))) return 1;
  if ((base.op != OP_FWD) && base.M && !base.g) return 1;
  if (nrows == 0) return 0;
  int64_t limit = (base.op == OP_FWD || base.op == OP_DQ) ? base.M : base.N;
  if (base.rows) {
    for (int64_t r = 0; r < nrows; ++r)
      if (base.rows[r] < 0 || base.rows[r] >= limit) return 1;
  } else if (nrows > limit) {
    return 1;
  }
  if (nthreads < 1) nthreads = 1;
  if (nthreads > ORACLE_MAX_THREADS) nthreads = ORACLE_MAX_THREADS;
  if ((int64_t)nthreads > nrows) nthreads = (int)nrows;

  job_t jobs[ORACLE_MAX_THREADS];
  pthread_t tids[ORACLE_MAX_THREADS];
  int64_t chunk = (nrows + nthreads - 1) / nthreads;
  int started = 0, rc = 0;
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = base;
    jobs[t].row_begin = t * chunk < nrows ? t * chunk : nrows;
    jobs[t].row_end = (t + 1) * chunk < nrows ? (t + 1) * chunk : nrows;
    if (t == 0) continue;
    if (pthread_create(&tids[t], NULL, run_job, &jobs[t]) != 0) { rc = 2; break; }
    started = t;
  }
  if (rc == 0) run_job(&jobs[0]);
  for (int t = 1; t <= started; ++t) pthread_join(tids[t], NULL);
  return rc;
}

/* Forward, Eq. 1: out[r,c] = s[rows[r], c], absout[r,c] = sum_n Phi |v[n,c]|.
 * q: M x D, k: N x D, v: N x C, row-major fp64; out, absout: nrows x C. */
int gs_oracle_fwd(int64_t M, int64_t N, int64_t D, int64_t C, const double* q, const double* k,
                  const double* v, double tau, const int64_t* rows, int64_t nrows, double* out,
                  double* absout, int nthreads) {
  job_t j = {OP_FWD, M, N, D, C, q, k, v, NULL, tau, rows, 0, 0, out, absout, NULL};
  return dispatch(j, nrows, nthreads);
}

/* Query gradient (Sec. 3): out[r,:] = dL/dq[rows[r],:] for L = sum g*s.
 * g: M x C; out, absout: nrows x D. */
int gs_oracle_dq(int64_t M, int64_t N, int64_t D, int64_t C, const double* q, const double* k,
                 const double* v, const double* g, double tau, const int64_t* rows, int64_t nrows,
                 double* out, double* absout, int nthreads) {
  job_t j = {OP_DQ, M, N, D, C, q, k, v, g, tau, rows, 0, 0, out, absout, NULL};
  return dispatch(j, nrows, nthreads);
}

/* Key gradient: out[r,:] = dL/dk[rows[r],:]; rows index keys. out: nrows x D. */
int gs_oracle_dk(int64_t M, int64_t N, int64_t D, int64_t C, const double* q, const double* k,
                 const double* v, const double* g, double tau, const int64_t* rows, int64_t nrows,
                 double* out, double* absout, int nthreads) {
  job_t j = {OP_DK, M, N, D, C, q, k, v, g, tau, rows, 0, 0, out, absout, NULL};
  return dispatch(j, nrows, nthreads);
}

/* gs_oracle_dq, also writing the net scale tau sum_n Phi |w| |k_n - q_m| to
 * netout (nrows x D). */
int gs_oracle_dq_scales(int64_t M, int64_t N, int64_t D, int64_t C, const double* q,
                        const double* k, const double* v, const double* g, double tau,
                        const int64_t* rows, int64_t nrows, double* out, double* absout,
                        double* netout, int nthreads) {
  job_t j = {OP_DQ, M, N, D, C, q, k, v, g, tau, rows, 0, 0, out, absout, netout};
  if (nrows && !netout) return 1;
  return dispatch(j, nrows, nthreads);
}

/* gs_oracle_dk, also writing the net scale tau sum_m Phi |w| |q_m - k_n|. */
int gs_oracle_dk_scales(int64_t M, int64_t N, int64_t D, int64_t C, const double* q,
                        const double* k, const double* v, const double* g, double tau,
                        const int64_t* rows, int64_t nrows, double* out, double* absout,
                        double* netout, int nthreads) {
  job_t j = {OP_DK, M, N, D, C, q, k, v, g, tau, rows, 0, 0, out, absout, netout};
  if (nrows && !netout) return 1;
  return dispatch(j, nrows, nthreads);
}

/* Value gradient: out[r,:] = dL/dv[rows[r],:]; rows index keys. out: nrows x C. */
int gs_oracle_dv(int64_t M, int64_t N, int64_t D, int64_t C, const double* q, const double* k,
                 const double* v, const double* g, double tau, const int64_t* rows, int64_t nrows,
                 double* out, double* absout, int nthreads) {
  job_t j = {OP_DV, M, N, D, C, q, k, v, g, tau, rows, 0, 0, out, absout, NULL};
  return dispatch(j, nrows, nthreads);
}
