/*
 * sw_oracle.h -- declarations of the plain CPU reference (test infrastructure
 * only; see sw_oracle.c).  Not included by, and sharing nothing with, the
 * HIP library.
 */
#ifndef SW_ORACLE_H
#define SW_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Number of threads a call with `requested` threads (<=0: all online CPUs)
 * over `rows` rows actually uses. */
int swo_threads_used(int requested, int64_t rows);

/* Eq. (7): (A2,U2) (+) (A1,U1); the left operand is the later segment. */
void swo_compose_f64(double A2, double U2, double A1, double U1, double* A, double* U);
void swo_compose_u32(uint32_t A2, uint32_t U2, uint32_t A1, uint32_t U1, uint32_t* A, uint32_t* U);

/* Eq. (3) per row, inclusive states h[r,t], t = 0..L-1 (h[r,-1] = h0[r] or 0).
 * mag / sens may be NULL.  Returns 0, or 1 on a bad argument. */
int swo_affine_scan_f64(const float* a, const float* bx, const float* h0, double* h, double* mag,
                        double* sens, int64_t rows, int64_t L, int nthreads);
int swo_affine_scan_u32(const uint32_t* a, const uint32_t* bx, const uint32_t* h0, uint32_t* h,
                        int64_t rows, int64_t L, int nthreads);

/* Eq. (3)-(4) with input and output projections: h_t = a_t h_{t-1} + b_t x_t,
 * y_t = c_t h_t per row (x, c NULL: ones); h_last[r] = h_{L-1} (h0 when L = 0).
 * Any of h0 / h_last / y_mag / y_sens may be NULL. */
int swo_affine_proj_f64(const float* a, const float* b, const float* x, const float* c,
                        const float* h0, double* y, double* h_last, double* y_mag, double* y_sens,
                        int64_t rows, int64_t L, int nthreads);
int swo_affine_proj_u32(const uint32_t* a, const uint32_t* b, const uint32_t* x,
                        const uint32_t* c, const uint32_t* h0, uint32_t* y, uint32_t* h_last,
                        int64_t rows, int64_t L, int nthreads);

/* Sec. 3.2 prefix compositions and the state rebuilt from them.  Any of
 * Apre / Upre / h may be NULL. */
int swo_affine_prefix_f64(const float* a, const float* bx, const float* h0, double* Apre,
                          double* Upre, double* h, int64_t rows, int64_t L);
int swo_affine_prefix_u32(const uint32_t* a, const uint32_t* bx, const uint32_t* h0,
                          uint32_t* Apre, uint32_t* Upre, uint32_t* h, int64_t rows, int64_t L);

/* Fused selective scan over R rows; see sw_oracle.c for the layout. */
int swo_selective_scan_f64(const float* x, const float* delta, const float* A, const float* Bm,
                           const float* Cm, const int64_t* row_b, const float* Dskip, double* y,
                           double* h_last, double* y_mag, double* y_sens, double* h_mag,
                           double* h_sens, int64_t R, int64_t N, int64_t L, int a_mode,
                           int nthreads);

/* The fused form with the optional Mamba-block inputs (z, delta_bias, h0,
 * softplus; any may be NULL / 0), per row; see sw_oracle.c. */
int swo_selective_scan_ex_f64(const float* x, const float* delta, const float* A, const float* Bm,
                              const float* Cm, const int64_t* row_b, const float* Dskip,
                              const float* z, const float* delta_bias, const float* h0,
                              int softplus, double* y, double* h_last, double* y_mag,
                              double* y_sens, double* h_mag, double* h_sens, int64_t R, int64_t N,
                              int64_t L, int a_mode, int nthreads);

/* Backward of the fused form (see sw_oracle.c).  Per-row outputs dx, ddelta,
 * dz (R, L), dh0 (R, N), the row's share of dA (R, N), dDskip and dbias (R);
 * dB, dC (nb, L, N) summed over the rows of each batch.  `mags`, if not NULL,
 * points to 9 arrays (any may be NULL) receiving the magnitudes of dx, ddelta,
 * dz, dA, dDskip, dbias, dh0, dB, dC in the same layouts. */
int swo_selective_scan_bwd_f64(const float* x, const float* delta, const float* A, const float* Bm,
                               const float* Cm, const int64_t* row_b, const float* Dskip,
                               const float* z, const float* delta_bias, const float* h0,
                               int softplus, const float* dy, const float* dh_last, double* dx,
                               double* ddelta, double* dz, double* dA, double* dD, double* dbias,
                               double* dh0, double* dB, double* dC, double* const* mags,
                               int64_t nb, int64_t R, int64_t N, int64_t L, int nthreads);

/* The fused form as a plain fp32 sequential loop (see sw_oracle.c). */
int swo_selective_scan_f32seq(const float* x, const float* delta, const float* A,
                              const float* Bm, const float* Cm, const int64_t* row_b,
                              const float* Dskip, float* y, float* h_last, int64_t R, int64_t N,
                              int64_t L, int nthreads);

#ifdef __cplusplus
}
#endif
#endif
