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
 *   softplus:       delta' = log(1 + exp(delta'))  (log1p of exp in fp64);
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
        if (c->softplus) dv = log1p(exp(dv));
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
