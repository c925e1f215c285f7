/*
 * sw_oracle.c -- plain CPU reference for the affine-recurrence hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the oracle that the HIP path is
 * checked against.  Only tests/, __graft_entry__.smoke() and the cpu_baseline
 * leg of bench.py may load it.  The product library never links, includes or
 * calls anything here, and nothing here is shared with the HIP sources.
 *
 * Every routine is the plain definition written out, in the paper's order:
 *   - the recurrence h_t = a_t h_{t-1} + b_t x_t of Sec. 3.1, Eq. (3), run as
 *     a sequential loop over t in fp64 (or in Z/2^32 for the int32 mode);
 *   - the affine pair (A_t, U_t) = (a_t, b_t x_t) of Sec. 3.2, Eq. (6), and
 *     its composition (A2,U2) (+) (A1,U1) = (A2 A1, A2 U1 + U2), Eq. (7);
 *   - the inclusive prefix compositions of Sec. 3.2, from which the state is
 *     rebuilt as h_t = A_{1:t} h_0 + U_{1:t};
 *   - the Mamba-style fused form used as the motivating workload (Sec. 1,
 *     Sec. 3.1): a_{t,n} = exp(delta_t A_n), b_t x_t = delta_t B_{t,n} x_t,
 *     y_t = sum_n C_{t,n} h_{t,n} + Dskip x_t, zero initial state.
 *
 * Beside the state, the fp64 loops carry two bounds used by the tests to
 * judge fp32 results (Sec. 6.5 asks that parameterisation effects be told
 * apart from implementation error):
 *   mag_t  = |a_t| mag_{t-1} + |u_t|,  mag_0 = |h_0|: the sum of the absolute
 *            values of the terms of the unrolled form Eq. (5), so |h_t|<=mag_t;
 *   sens_t = |a_t| (sens_{t-1} + mag_{t-1}), sens_0 = 0: the sum over k of
 *            (t-k) |prod a| |u_k|, i.e. the first-order change of h_t when
 *            every a_i is perturbed by a relative amount of one.
 *
 * Rows are independent recurrences; they are split over POSIX threads.  Each
 * row stays a plain sequential loop.  No fast-math: build with -O2 and
 * -fno-fast-math.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include "sw_oracle.h"

/* ------------------------------------------------------------------------ */
/* threading helper: run fn(row_begin, row_end, ctx) over a static partition  */

typedef void (*row_fn)(int64_t r0, int64_t r1, const void* ctx);

typedef struct {
  row_fn fn;
  const void* ctx;
  int64_t r0, r1;
} worker_arg;

static void* worker_main(void* p) {
  worker_arg* w = (worker_arg*)p;
  w->fn(w->r0, w->r1, w->ctx);
  return NULL;
}

int swo_threads_used(int requested, int64_t rows) {
  long ncpu = sysconf(_SC_NPROCESSORS_ONLN);
  int t = requested > 0 ? requested : (int)(ncpu > 0 ? ncpu : 1);
  if (t > 256) t = 256;
  if (rows < t) t = (int)(rows > 0 ? rows : 1);
  return t;
}

static void run_rows(row_fn fn, const void* ctx, int64_t rows, int requested) {
  int t = swo_threads_used(requested, rows);
  if (t <= 1) {
    fn(0, rows, ctx);
    return;
  }
  pthread_t tid[256];
  worker_arg args[256];
  int64_t per = rows / t, extra = rows % t, r = 0;
  for (int i = 0; i < t; i++) {
    int64_t n = per + (i < extra ? 1 : 0);
    args[i].fn = fn;
    args[i].ctx = ctx;
    args[i].r0 = r;
    args[i].r1 = r + n;
    r += n;
    if (pthread_create(&tid[i], NULL, worker_main, &args[i]) != 0) {
      /* could not start a thread: do this share on the calling thread */
      fn(args[i].r0, args[i].r1, ctx);
      args[i].fn = NULL;
    }
  }
  for (int i = 0; i < t; i++)
    if (args[i].fn) pthread_join(tid[i], NULL);
}

/* ------------------------------------------------------------------------ */
/* Eq. (7): (A2,U2) (+) (A1,U1) = (A2*A1, A2*U1 + U2); the left operand is the
 * later segment. */

void swo_compose_f64(double A2, double U2, double A1, double U1, double* A, double* U) {
  *A = A2 * A1;
  *U = A2 * U1 + U2;
}

void swo_compose_u32(uint32_t A2, uint32_t U2, uint32_t A1, uint32_t U1, uint32_t* A, uint32_t* U) {
  *A = A2 * A1;      /* unsigned arithmetic wraps modulo 2^32 */
  *U = A2 * U1 + U2;
}

/* ------------------------------------------------------------------------ */
/* Bare recurrence, fp64: Eq. (3) with the output taken as every inclusive
 * state h_1..h_L of each row. */

typedef struct {
  const float *a, *bx, *h0;
  double *h, *mag, *sens;
  int64_t L;
} affine_f64_ctx;

static void affine_f64_rows(int64_t r0, int64_t r1, const void* vctx) {
  const affine_f64_ctx* c = (const affine_f64_ctx*)vctx;
  for (int64_t r = r0; r < r1; r++) {
    const float* a = c->a + r * c->L;
    const float* bx = c->bx + r * c->L;
    double h = c->h0 ? (double)c->h0[r] : 0.0;
    double m = fabs(h), s = 0.0;
    for (int64_t t = 0; t < c->L; t++) {
      double at = (double)a[t], ut = (double)bx[t];
      h = at * h + ut;
      s = fabs(at) * (s + m);
      m = fabs(at) * m + fabs(ut);
      c->h[r * c->L + t] = h;
      if (c->mag) c->mag[r * c->L + t] = m;
      if (c->sens) c->sens[r * c->L + t] = s;
    }
  }
}

int swo_affine_scan_f64(const float* a, const float* bx, const float* h0, double* h, double* mag,
                        double* sens, int64_t rows, int64_t L, int nthreads) {
  if (!a || !bx || !h || rows < 0 || L < 0) return 1;
  affine_f64_ctx c = {a, bx, h0, h, mag, sens, L};
  run_rows(affine_f64_rows, &c, rows, nthreads);
  return 0;
}

/* Bare recurrence in the int32 wraparound ring Z/2^32. */

typedef struct {
  const uint32_t *a, *bx, *h0;
  uint32_t* h;
  int64_t L;
} affine_u32_ctx;

static void affine_u32_rows(int64_t r0, int64_t r1, const void* vctx) {
  const affine_u32_ctx* c = (const affine_u32_ctx*)vctx;
  for (int64_t r = r0; r < r1; r++) {
    const uint32_t* a = c->a + r * c->L;
    const uint32_t* bx = c->bx + r * c->L;
    uint32_t h = c->h0 ? c->h0[r] : 0u;
    for (int64_t t = 0; t < c->L; t++) {
      h = a[t] * h + bx[t];
      c->h[r * c->L + t] = h;
    }
  }
}

int swo_affine_scan_u32(const uint32_t* a, const uint32_t* bx, const uint32_t* h0, uint32_t* h,
                        int64_t rows, int64_t L, int nthreads) {
  if (!a || !bx || !h || rows < 0 || L < 0) return 1;
  affine_u32_ctx c = {a, bx, h0, h, L};
  run_rows(affine_u32_rows, &c, rows, nthreads);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Eq. (3)-(4) with the input and output projections written out: per row,
 * h_t = a_t h_{t-1} + b_t x_t and y_t = c_t h_t, with x or c absent meaning
 * all ones (the weighted prefix of Eq. (10) is x = 1, c = 1).  fp64: the
 * products of two fp32 values are exact.  y_mag = |c_t| M_t and
 * y_sens = |c_t| M1_t, with M and M1 as for the bare recurrence. */

typedef struct {
  const float *a, *b, *x, *c, *h0;
  double *y, *h_last, *y_mag, *y_sens;
  int64_t L;
} proj_f64_ctx;

static void proj_f64_rows(int64_t r0, int64_t r1, const void* vctx) {
  const proj_f64_ctx* c = (const proj_f64_ctx*)vctx;
  const int64_t L = c->L;
  for (int64_t r = r0; r < r1; r++) {
    double h = c->h0 ? (double)c->h0[r] : 0.0;
    double m = fabs(h), s = 0.0;
    for (int64_t t = 0; t < L; t++) {
      const int64_t i = r * L + t;
      const double at = (double)c->a[i];
      const double ut = (double)c->b[i] * (c->x ? (double)c->x[i] : 1.0);
      const double ct = c->c ? (double)c->c[i] : 1.0;
      h = at * h + ut;
      s = fabs(at) * (s + m);
      m = fabs(at) * m + fabs(ut);
      c->y[i] = ct * h;
      if (c->y_mag) c->y_mag[i] = fabs(ct) * m;
      if (c->y_sens) c->y_sens[i] = fabs(ct) * s;
    }
    if (c->h_last) c->h_last[r] = h;
  }
}

int swo_affine_proj_f64(const float* a, const float* b, const float* x, const float* cc,
                        const float* h0, double* y, double* h_last, double* y_mag, double* y_sens,
                        int64_t rows, int64_t L, int nthreads) {
  if (!a || !b || !y || rows < 0 || L < 0) return 1;
  proj_f64_ctx c = {a, b, x, cc, h0, y, h_last, y_mag, y_sens, L};
  run_rows(proj_f64_rows, &c, rows, nthreads);
  return 0;
}

typedef struct {
  const uint32_t *a, *b, *x, *c, *h0;
  uint32_t *y, *h_last;
  int64_t L;
} proj_u32_ctx;

static void proj_u32_rows(int64_t r0, int64_t r1, const void* vctx) {
  const proj_u32_ctx* c = (const proj_u32_ctx*)vctx;
  const int64_t L = c->L;
  for (int64_t r = r0; r < r1; r++) {
    uint32_t h = c->h0 ? c->h0[r] : 0u;
    for (int64_t t = 0; t < L; t++) {
      const int64_t i = r * L + t;
      const uint32_t ut = c->b[i] * (c->x ? c->x[i] : 1u);
      h = c->a[i] * h + ut;
      c->y[i] = (c->c ? c->c[i] : 1u) * h;
    }
    if (c->h_last) c->h_last[r] = h;
  }
}

int swo_affine_proj_u32(const uint32_t* a, const uint32_t* b, const uint32_t* x,
                        const uint32_t* cc, const uint32_t* h0, uint32_t* y, uint32_t* h_last,
                        int64_t rows, int64_t L, int nthreads) {
  if (!a || !b || !y || rows < 0 || L < 0) return 1;
  proj_u32_ctx c = {a, b, x, cc, h0, y, h_last, L};
  run_rows(proj_u32_rows, &c, rows, nthreads);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Sec. 3.2: inclusive prefix compositions P_t = p_t (+) P_{t-1}, P_0 = the
 * identity pair (1, 0), p_t = (a_t, bx_t) of Eq. (6).  The state is rebuilt
 * from the prefix pair as h_t = A_{1:t} h_0 + U_{1:t}.  This is a second,
 * independent route to the states of the loop above. */

int swo_affine_prefix_f64(const float* a, const float* bx, const float* h0, double* Apre,
                          double* Upre, double* h, int64_t rows, int64_t L) {
  if (!a || !bx || rows < 0 || L < 0) return 1;
  for (int64_t r = 0; r < rows; r++) {
    double PA = 1.0, PU = 0.0;
    double hz = h0 ? (double)h0[r] : 0.0;
    for (int64_t t = 0; t < L; t++) {
      double nA, nU;
      swo_compose_f64((double)a[r * L + t], (double)bx[r * L + t], PA, PU, &nA, &nU);
      PA = nA;
      PU = nU;
      if (Apre) Apre[r * L + t] = PA;
      if (Upre) Upre[r * L + t] = PU;
      if (h) h[r * L + t] = PA * hz + PU;
    }
  }
  return 0;
}

int swo_affine_prefix_u32(const uint32_t* a, const uint32_t* bx, const uint32_t* h0,
                          uint32_t* Apre, uint32_t* Upre, uint32_t* h, int64_t rows, int64_t L) {
  if (!a || !bx || rows < 0 || L < 0) return 1;
  for (int64_t r = 0; r < rows; r++) {
    uint32_t PA = 1u, PU = 0u;
    uint32_t hz = h0 ? h0[r] : 0u;
    for (int64_t t = 0; t < L; t++) {
      uint32_t nA, nU;
      swo_compose_u32(a[r * L + t], bx[r * L + t], PA, PU, &nA, &nU);
      PA = nA;
      PU = nU;
      if (Apre) Apre[r * L + t] = PA;
      if (Upre) Upre[r * L + t] = PU;
      if (h) h[r * L + t] = PA * hz + PU;
    }
  }
  return 0;
}

/* softplus(v) = log(1 + e^v).  For v > 0 it is written v + log(1 + e^-v),
 * the same value, so that e^v is never formed where it would overflow. */
static double softplus_f64(double v) { return v > 0.0 ? v + log1p(exp(-v)) : log1p(exp(v)); }

/* ------------------------------------------------------------------------ */
/* Fused selective scan, fp64.  Rows are (batch, channel) pairs; row r reads
 * x[r,:], delta[r,:], A[r,:] (its channel's row of A), Dskip[r], and the
 * (L, N) slices Bm[row_b[r]], Cm[row_b[r]] shared by all channels of a batch.
 *
 *   for each n:  h = 0
 *     for each t: a = exp(delta_t * A_n)            (discretised transition)
 *                 u = delta_t * x_t * B_{t,n}       (discretised input)
 *                 h = a * h + u                     (Eq. (3))
 *                 y_t += C_{t,n} * h                (projection over n)
 *     h_last_n = h
 *   y_t += Dskip * x_t
 *
 * a_mode 0: a in fp64.  a_mode 1: a rounded to fp32 before use (isolates the
 * error that any fp32 implementation takes on by storing exp(delta A) in
 * fp32; used for the numerical characterisation of Sec. 6.5).
 *
 * The optional inputs of a Mamba block (the production kernel the paper
 * compares against fuses them; Sec. 1, Sec. 6.3), all NULL / 0 by default:
 *   delta_bias[d]:  delta' = delta + delta_bias[d];
 *   softplus:       delta' = log(1 + exp(delta')), evaluated in fp64 as
 *                   log1p(exp(v)) for v <= 0 and v + log1p(exp(-v)) above
 *                   (the same function; exp(v) would overflow for v > 709);
 *   h0[r, n]:       initial state h[-1] instead of zero (mag_0 = |h0|);
 *   z[r, t]:        y_t <- y_t * silu(z_t), silu(z) = z / (1 + exp(-z)); the
 *                   magnitude and sensitivity of y scale by |silu(z_t)|. */

typedef struct {
  const float *x, *delta, *A, *Bm, *Cm, *Dskip;
  const int64_t* row_b;
  double *y, *h_last, *y_mag, *y_sens, *h_mag, *h_sens;
  int64_t N, L;
  int a_mode;
  const float *z, *delta_bias, *h0;
  int softplus;
} sel_ctx;

static void sel_rows(int64_t r0, int64_t r1, const void* vctx) {
  const sel_ctx* c = (const sel_ctx*)vctx;
  const int64_t N = c->N, L = c->L;
  for (int64_t r = r0; r < r1; r++) {
    const float* x = c->x + r * L;
    const float* dl = c->delta + r * L;
    const float* Bm = c->Bm + c->row_b[r] * L * N;
    const float* Cm = c->Cm + c->row_b[r] * L * N;
    double* y = c->y + r * L;
    double* ym = c->y_mag ? c->y_mag + r * L : NULL;
    double* ys = c->y_sens ? c->y_sens + r * L : NULL;
    for (int64_t t = 0; t < L; t++) {
      y[t] = 0.0;
      if (ym) ym[t] = 0.0;
      if (ys) ys[t] = 0.0;
    }
    for (int64_t n = 0; n < N; n++) {
      const double An = (double)c->A[r * N + n];
      double h = c->h0 ? (double)c->h0[r * N + n] : 0.0;
      double m = fabs(h), s = 0.0;
      for (int64_t t = 0; t < L; t++) {
        double dv = (double)dl[t];
        if (c->delta_bias) dv += (double)c->delta_bias[r];
        if (c->softplus) dv = softplus_f64(dv);
        double a = exp(dv * An);
        if (c->a_mode == 1) a = (double)(float)a;
        const double u = dv * (double)x[t] * (double)Bm[t * N + n];
        const double cc = (double)Cm[t * N + n];
        h = a * h + u;
        s = fabs(a) * (s + m);
        m = fabs(a) * m + fabs(u);
        y[t] += cc * h;
        if (ym) ym[t] += fabs(cc) * m;
        if (ys) ys[t] += fabs(cc) * s;
      }
      if (c->h_last) c->h_last[r * N + n] = h;
      if (c->h_mag) c->h_mag[r * N + n] = m;
      if (c->h_sens) c->h_sens[r * N + n] = s;
    }
    if (c->Dskip) {
      const double Dr = (double)c->Dskip[r];
      for (int64_t t = 0; t < L; t++) {
        y[t] += Dr * (double)x[t];
        if (ym) ym[t] += fabs(Dr * (double)x[t]);
      }
    }
    if (c->z) {
      const float* z = c->z + r * L;
      for (int64_t t = 0; t < L; t++) {
        const double zv = (double)z[t];
        const double g = zv / (1.0 + exp(-zv));
        y[t] *= g;
        if (ym) ym[t] *= fabs(g);
        if (ys) ys[t] *= fabs(g);
      }
    }
  }
}

int swo_selective_scan_ex_f64(const float* x, const float* delta, const float* A, const float* Bm,
                              const float* Cm, const int64_t* row_b, const float* Dskip,
                              const float* z, const float* delta_bias, const float* h0,
                              int softplus, double* y, double* h_last, double* y_mag,
                              double* y_sens, double* h_mag, double* h_sens, int64_t R, int64_t N,
                              int64_t L, int a_mode, int nthreads) {
  if (!x || !delta || !A || !Bm || !Cm || !row_b || !y || R < 0 || N < 0 || L < 0) return 1;
  if (a_mode != 0 && a_mode != 1) return 1;
  sel_ctx c = {x, delta, A, Bm, Cm, Dskip, row_b, y, h_last, y_mag, y_sens, h_mag, h_sens,
               N, L, a_mode, z, delta_bias, h0, softplus != 0};
  run_rows(sel_rows, &c, R, nthreads);
  return 0;
}

int swo_selective_scan_f64(const float* x, const float* delta, const float* A, const float* Bm,
                           const float* Cm, const int64_t* row_b, const float* Dskip, double* y,
                           double* h_last, double* y_mag, double* y_sens, double* h_mag,
                           double* h_sens, int64_t R, int64_t N, int64_t L, int a_mode,
                           int nthreads) {
  if (!x || !delta || !A || !Bm || !Cm || !row_b || !y || R < 0 || N < 0 || L < 0) return 1;
  if (a_mode != 0 && a_mode != 1) return 1;
  return swo_selective_scan_ex_f64(x, delta, A, Bm, Cm, row_b, Dskip, NULL, NULL, NULL, 0, y,
                                   h_last, y_mag, y_sens, h_mag, h_sens, R, N, L, a_mode,
                                   nthreads);
}

/* ------------------------------------------------------------------------ */
/* Backward of the fused form (the gradient of a scalar loss
 * sum_t dy_t y_t + sum_n dh_last_n h_last_n with respect to every input),
 * by the chain rule through the forward loop above.  The paper gives the
 * forward only; the adjoint of Eq. (3) is the same kind of recurrence run
 * backwards in time:
 *   ds_t      = dy_t g_t                       (g_t = silu(z_t), or 1)
 *   lam_t     = ds_t C_{t,n} + a_{t+1,n} lam_{t+1},   lam_{L} term = dh_last_n
 *   dh0_n     = a_{0,n} lam_0
 *   dC_{t,n} += ds_t h_{t,n}                   (summed over the rows of a batch)
 *   dB_{t,n} += lam_t delta_t x_t              (summed over the rows of a batch)
 *   ddelta'_t = sum_n lam_t (a_t h_{t-1} A_n + B_{t,n} x_t)
 *   dx_t      = sum_n lam_t delta_t B_{t,n} + ds_t Dskip
 *   dA_n     += sum_t lam_t a_t h_{t-1} delta_t
 *   dDskip   += sum_t ds_t x_t
 *   dz_t      = dy_t s_t silu'(z_t),  s_t = sum_n C h + Dskip x (pre-gate y)
 *   ddelta_t  = ddelta'_t sigmoid(delta_t + bias) with softplus, else ddelta'_t
 *   dbias    += sum_t ddelta_t
 * where delta is the delta after bias and softplus.  Each row also gets the
 * magnitude of every output: the same expressions evaluated on absolute
 * values with |h| replaced by the forward magnitude M_t and lam by
 *   Mlam_t = |ds_t C_{t,n}| + |a_{t+1}| Mlam_{t+1},   Mlam_L = |dh_last|,
 * which bounds the sum of the absolute values of the terms of each output
 * (silu'(z) = sig + z sig (1 - sig) enters with |sig| + |z sig (1 - sig)|).
 * Per-row outputs: dx, ddelta, dz (R, L); dh0 (R, N); the row's share of dA
 * (R, N), dDskip and dbias (R).  dB and dC (nb, L, N) are summed over the
 * rows of each batch (each thread accumulates its own copy; the copies are
 * added in thread order). */

typedef struct {
  const float *x, *delta, *A, *Bm, *Cm, *Dskip, *z, *delta_bias, *h0, *dy, *dh_last;
  const int64_t* row_b;
  int softplus;
  double *dx, *ddelta, *dz, *dA, *dD, *dbias, *dh0;
  double *mdx, *mddelta, *mdz, *mdA, *mdD, *mdbias, *mdh0;
  double *accB, *accC, *accMB, *accMC; /* per thread: nthreads x (nb, L, N) */
  int64_t nb, N, L;
} bwd_ctx;

static void bwd_rows(int64_t r0, int64_t r1, int ti, const void* vctx) {
  const bwd_ctx* c = (const bwd_ctx*)vctx;
  const int64_t N = c->N, L = c->L;
  const int64_t per = c->nb * L * N;
  double* aB = c->accB + (int64_t)ti * per;
  double* aC = c->accC + (int64_t)ti * per;
  double* aMB = c->accMB ? c->accMB + (int64_t)ti * per : NULL;
  double* aMC = c->accMC ? c->accMC + (int64_t)ti * per : NULL;
  /* per-row work arrays */
  double* dl = (double*)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1) * 8);
  double* hs = (double*)malloc(sizeof(double) * (size_t)(L + 1) * 2);
  if (!dl || !hs) {
    free(dl);
    free(hs);
    return;
  }
  double* sg = dl + L;     /* d delta / d raw delta */
  double* g = dl + 2 * L;  /* gate */
  double* gp = dl + 3 * L; /* gate derivative */
  double* ds = dl + 4 * L;
  double* s = dl + 5 * L;  /* pre-gate y */
  double* ms = dl + 6 * L; /* its magnitude */
  double* mgp = dl + 7 * L; /* |sig| + |z sig (1 - sig)|: the terms of the gate derivative */
  double* mh = hs + (L + 1);
  for (int64_t r = r0; r < r1; r++) {
    const float* x = c->x + r * L;
    const float* dyr = c->dy + r * L;
    const int64_t b = c->row_b[r];
    const float* Bm = c->Bm + b * L * N;
    const float* Cm = c->Cm + b * L * N;
    const double Dr = c->Dskip ? (double)c->Dskip[r] : 0.0;
    for (int64_t t = 0; t < L; t++) {
      const double raw = (double)c->delta[r * L + t] + (c->delta_bias ? (double)c->delta_bias[r] : 0.0);
      if (c->softplus) {
        dl[t] = softplus_f64(raw);
        sg[t] = 1.0 / (1.0 + exp(-raw));
      } else {
        dl[t] = raw;
        sg[t] = 1.0;
      }
      if (c->z) {
        const double zv = (double)c->z[r * L + t];
        const double sig = 1.0 / (1.0 + exp(-zv));
        g[t] = zv * sig;
        gp[t] = sig * (1.0 + zv * (1.0 - sig));
        mgp[t] = sig + fabs(zv * sig * (1.0 - sig));
      } else {
        g[t] = 1.0;
        gp[t] = 0.0;
        mgp[t] = 0.0;
      }
      ds[t] = (double)dyr[t] * g[t];
      s[t] = Dr * (double)x[t];
      ms[t] = fabs(Dr * (double)x[t]);
      c->dx[r * L + t] = ds[t] * Dr;
      c->ddelta[r * L + t] = 0.0;
      if (c->mdx) c->mdx[r * L + t] = fabs(ds[t] * Dr);
      if (c->mddelta) c->mddelta[r * L + t] = 0.0;
    }
    double dD_sum = 0.0, mD_sum = 0.0;
    for (int64_t n = 0; n < N; n++) {
      const double An = (double)c->A[r * N + n];
      /* forward: hs[t+1] = h_t, hs[0] = h_{-1} */
      hs[0] = c->h0 ? (double)c->h0[r * N + n] : 0.0;
      mh[0] = fabs(hs[0]);
      for (int64_t t = 0; t < L; t++) {
        const double a = exp(dl[t] * An);
        const double u = dl[t] * (double)x[t] * (double)Bm[t * N + n];
        hs[t + 1] = a * hs[t] + u;
        mh[t + 1] = fabs(a) * mh[t] + fabs(u);
        s[t] += (double)Cm[t * N + n] * hs[t + 1];
        ms[t] += fabs((double)Cm[t * N + n]) * mh[t + 1];
      }
      /* backward */
      double lam_next = c->dh_last ? (double)c->dh_last[r * N + n] : 0.0;
      double mlam_next = fabs(lam_next);
      double dA_n = 0.0, mA_n = 0.0;
      for (int64_t t = L - 1; t >= 0; t--) {
        const double a = exp(dl[t] * An);
        const double Bt = (double)Bm[t * N + n], Ct = (double)Cm[t * N + n];
        const double lam = ds[t] * Ct + lam_next;
        const double mlam = fabs(ds[t] * Ct) + mlam_next;
        const double xb = (double)x[t] * Bt;
        c->ddelta[r * L + t] += lam * (a * hs[t] * An + xb);
        c->dx[r * L + t] += lam * dl[t] * Bt;
        if (c->mddelta) c->mddelta[r * L + t] += mlam * (fabs(a * An) * mh[t] + fabs(xb));
        if (c->mdx) c->mdx[r * L + t] += mlam * fabs(dl[t] * Bt);
        dA_n += lam * a * hs[t] * dl[t];
        mA_n += mlam * fabs(a * dl[t]) * mh[t];
        aB[(b * L + t) * N + n] += lam * dl[t] * (double)x[t];
        aC[(b * L + t) * N + n] += ds[t] * hs[t + 1];
        if (aMB) aMB[(b * L + t) * N + n] += mlam * fabs(dl[t] * (double)x[t]);
        if (aMC) aMC[(b * L + t) * N + n] += fabs(ds[t]) * mh[t + 1];
        lam_next = a * lam;
        mlam_next = fabs(a) * mlam;
      }
      c->dA[r * N + n] = dA_n;
      if (c->mdA) c->mdA[r * N + n] = mA_n;
      if (c->dh0) c->dh0[r * N + n] = lam_next;
      if (c->mdh0) c->mdh0[r * N + n] = mlam_next;
    }
    double dbias = 0.0, mbias = 0.0;
    for (int64_t t = 0; t < L; t++) {
      dD_sum += ds[t] * (double)x[t];
      mD_sum += fabs(ds[t] * (double)x[t]);
      c->ddelta[r * L + t] *= sg[t];
      if (c->mddelta) c->mddelta[r * L + t] *= fabs(sg[t]);
      dbias += c->ddelta[r * L + t];
      if (c->mddelta) mbias += c->mddelta[r * L + t];
      if (c->dz) {
        c->dz[r * L + t] = (double)dyr[t] * s[t] * gp[t];
        if (c->mdz) c->mdz[r * L + t] = fabs((double)dyr[t]) * mgp[t] * ms[t];
      }
    }
    c->dD[r] = dD_sum;
    if (c->mdD) c->mdD[r] = mD_sum;
    c->dbias[r] = dbias;
    if (c->mdbias) c->mdbias[r] = mbias;
  }
  free(dl);
  free(hs);
}

typedef void (*row_fn_i)(int64_t r0, int64_t r1, int ti, const void* ctx);

typedef struct {
  row_fn_i fn;
  const void* ctx;
  int64_t r0, r1;
  int ti;
} worker_arg_i;

static void* worker_main_i(void* p) {
  worker_arg_i* w = (worker_arg_i*)p;
  w->fn(w->r0, w->r1, w->ti, w->ctx);
  return NULL;
}

/* run_rows with the worker's index passed along (for per-thread buffers) */
static void run_rows_i(row_fn_i fn, const void* ctx, int64_t rows, int t) {
  if (t <= 1) {
    fn(0, rows, 0, ctx);
    return;
  }
  pthread_t tid[256];
  worker_arg_i args[256];
  int64_t per = rows / t, extra = rows % t, r = 0;
  for (int i = 0; i < t; i++) {
    int64_t n = per + (i < extra ? 1 : 0);
    args[i].fn = fn;
    args[i].ctx = ctx;
    args[i].r0 = r;
    args[i].r1 = r + n;
    args[i].ti = i;
    r += n;
    if (pthread_create(&tid[i], NULL, worker_main_i, &args[i]) != 0) {
      fn(args[i].r0, args[i].r1, i, ctx);
      args[i].fn = NULL;
    }
  }
  for (int i = 0; i < t; i++)
    if (args[i].fn) pthread_join(tid[i], NULL);
}

int swo_selective_scan_bwd_f64(const float* x, const float* delta, const float* A, const float* Bm,
                               const float* Cm, const int64_t* row_b, const float* Dskip,
                               const float* z, const float* delta_bias, const float* h0,
                               int softplus, const float* dy, const float* dh_last, double* dx,
                               double* ddelta, double* dz, double* dA, double* dD, double* dbias,
                               double* dh0, double* dB, double* dC, double* const* mags,
                               int64_t nb, int64_t R, int64_t N, int64_t L, int nthreads) {
  if (!x || !delta || !A || !Bm || !Cm || !row_b || !dy || !dx || !ddelta || !dA || !dD ||
      !dbias || !dB || !dC || nb < 0 || R < 0 || N < 0 || L < 0)
    return 1;
  if (z && !dz) return 1;
  for (int64_t r = 0; r < R; r++)
    if (row_b[r] < 0 || row_b[r] >= nb) return 1;
  const int t = swo_threads_used(nthreads, R);
  const int64_t per = nb * L * N;
  const int want_m = mags != NULL;
  double* acc = (double*)calloc((size_t)t * (size_t)per * (want_m ? 4 : 2) + 1, sizeof(double));
  if (!acc) return 1;
  bwd_ctx c;
  memset(&c, 0, sizeof(c));
  c.x = x; c.delta = delta; c.A = A; c.Bm = Bm; c.Cm = Cm; c.Dskip = Dskip; c.z = z;
  c.delta_bias = delta_bias; c.h0 = h0; c.dy = dy; c.dh_last = dh_last; c.row_b = row_b;
  c.softplus = softplus != 0;
  c.dx = dx; c.ddelta = ddelta; c.dz = dz; c.dA = dA; c.dD = dD; c.dbias = dbias; c.dh0 = dh0;
  if (want_m) {
    c.mdx = mags[0]; c.mddelta = mags[1]; c.mdz = mags[2]; c.mdA = mags[3]; c.mdD = mags[4];
    c.mdbias = mags[5]; c.mdh0 = mags[6];
  }
  c.accB = acc;
  c.accC = acc + (size_t)t * per;
  if (want_m) {
    c.accMB = acc + 2 * (size_t)t * per;
    c.accMC = acc + 3 * (size_t)t * per;
  }
  c.nb = nb; c.N = N; c.L = L;
  run_rows_i(bwd_rows, &c, R, t);
  for (int64_t i = 0; i < per; i++) {
    double sb = 0.0, sc = 0.0, mb = 0.0, mc = 0.0;
    for (int k = 0; k < t; k++) {
      sb += c.accB[(size_t)k * per + i];
      sc += c.accC[(size_t)k * per + i];
      if (want_m) {
        mb += c.accMB[(size_t)k * per + i];
        mc += c.accMC[(size_t)k * per + i];
      }
    }
    dB[i] = sb;
    dC[i] = sc;
    if (want_m) {
      if (mags[7]) mags[7][i] = mb;
      if (mags[8]) mags[8][i] = mc;
    }
  }
  free(acc);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* The fused form as a plain fp32 sequential loop: the same loop as above with
 * every quantity held and rounded in fp32, in the order written, with libm's
 * expf and no FMA contraction (ISO C, -std=c11):
 *
 *   a = expf(delta_t * A_n);  u = (delta_t * x_t) * B_{t,n};
 *   h = a * h + u;            y_t += C_{t,n} * h;   then y_t += Dskip * x_t.
 *
 * It is not a reference for the GPU result: it measures what a direct fp32
 * evaluation of the recurrence incurs against the fp64 loop (the numerical
 * characterisation of Sec. 6.5). */

typedef struct {
  const float *x, *delta, *A, *Bm, *Cm, *Dskip;
  const int64_t* row_b;
  float *y, *h_last;
  int64_t N, L;
} sel32_ctx;

static void sel32_rows(int64_t r0, int64_t r1, const void* vctx) {
  const sel32_ctx* c = (const sel32_ctx*)vctx;
  const int64_t N = c->N, L = c->L;
  for (int64_t r = r0; r < r1; r++) {
    const float* x = c->x + r * L;
    const float* dl = c->delta + r * L;
    const float* Bm = c->Bm + c->row_b[r] * L * N;
    const float* Cm = c->Cm + c->row_b[r] * L * N;
    float* y = c->y + r * L;
    for (int64_t t = 0; t < L; t++) y[t] = 0.0f;
    for (int64_t n = 0; n < N; n++) {
      const float An = c->A[r * N + n];
      float h = 0.0f;
      for (int64_t t = 0; t < L; t++) {
        const float a = expf(dl[t] * An);
        const float u = (dl[t] * x[t]) * Bm[t * N + n];
        const float ah = a * h;
        h = ah + u;
        const float ch = Cm[t * N + n] * h;
        y[t] = y[t] + ch;
      }
      if (c->h_last) c->h_last[r * N + n] = h;
    }
    if (c->Dskip) {
      const float Dr = c->Dskip[r];
      for (int64_t t = 0; t < L; t++) {
        const float dx = Dr * x[t];
        y[t] = y[t] + dx;
      }
    }
  }
}

int swo_selective_scan_f32seq(const float* x, const float* delta, const float* A,
                              const float* Bm, const float* Cm, const int64_t* row_b,
                              const float* Dskip, float* y, float* h_last, int64_t R, int64_t N,
                              int64_t L, int nthreads) {
  if (!x || !delta || !A || !Bm || !Cm || !row_b || !y || R < 0 || N < 0 || L < 0) return 1;
  sel32_ctx c = {x, delta, A, Bm, Cm, Dskip, row_b, y, h_last, N, L};
  run_rows(sel32_rows, &c, R, nthreads);
  return 0;
}
