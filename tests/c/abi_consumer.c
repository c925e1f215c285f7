/*
 * A plain C program that uses libscanweaver through its C ABI only (no
 * Python, no torch): device memory from the HIP runtime, one call of each
 * kind, results checked against closed forms, and the error paths.
 *
 *   int32 bare scan with a = 1, bx = 1, h0[r] = 7 r  ->  h_t = 7 r + t + 1
 *     (exact in the int32 ring);
 *   fp32 fused scan with A = 0 (so a = exp(0) = 1), delta = 0.5, x = 1,
 *     B = C = 1, Dskip = 2, N = 1  ->  h_t = 0.5 (t + 1) and
 *     y_t = 0.5 (t + 1) + 2 (exact in fp32 at these lengths);
 *   a NULL output and a host pointer are rejected with SW_ERR_INVALID_ARG
 *     and a message.
 * Prints "abi consumer ok" and exits 0 on success.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "scanweaver.h"

#define HIPCHK(e)                                                             \
  do {                                                                        \
    hipError_t err_ = (e);                                                    \
    if (err_ != hipSuccess) {                                                 \
      fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, hipGetErrorString(err_)); \
      return 2;                                                               \
    }                                                                         \
  } while (0)

static int fail(const char* what) {
  fprintf(stderr, "abi consumer: %s (last error: %s)\n", what, sw_last_error());
  return 1;
}

static int check_affine_i32(void) {
  const int64_t B = 2, D = 3, L = 5000, n = B * D * L;
  int32_t* host = (int32_t*)malloc((size_t)n * sizeof(int32_t));
  int32_t h0h[6];
  int32_t *a, *bx, *h0, *h;
  int64_t i, r;
  if (!host) return fail("host allocation");
  HIPCHK(hipMalloc((void**)&a, (size_t)n * sizeof(int32_t)));
  HIPCHK(hipMalloc((void**)&bx, (size_t)n * sizeof(int32_t)));
  HIPCHK(hipMalloc((void**)&h, (size_t)n * sizeof(int32_t)));
  HIPCHK(hipMalloc((void**)&h0, sizeof(h0h)));
  for (i = 0; i < n; ++i) host[i] = 1;
  for (r = 0; r < B * D; ++r) h0h[r] = (int32_t)(7 * r);
  HIPCHK(hipMemcpy(a, host, (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(bx, host, (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(h0, h0h, sizeof(h0h), hipMemcpyHostToDevice));
  if (sw_affine_scan_i32(a, bx, h0, h, B, D, L) != SW_OK) return fail("sw_affine_scan_i32");
  HIPCHK(hipDeviceSynchronize());
  HIPCHK(hipMemcpy(host, h, (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost));
  for (r = 0; r < B * D; ++r)
    for (i = 0; i < L; ++i)
      if (host[r * L + i] != (int32_t)(7 * r + i + 1)) return fail("int32 scan value");
  /* error paths: NULL output, then a host pointer as input */
  if (sw_affine_scan_i32(a, bx, h0, NULL, B, D, L) != SW_ERR_INVALID_ARG)
    return fail("NULL output accepted");
  if (strlen(sw_last_error()) == 0) return fail("no message for the NULL output");
  if (sw_affine_scan_i32(host, bx, h0, h, B, D, L) != SW_ERR_INVALID_ARG)
    return fail("host pointer accepted");
  HIPCHK(hipFree(a));
  HIPCHK(hipFree(bx));
  HIPCHK(hipFree(h));
  HIPCHK(hipFree(h0));
  free(host);
  return 0;
}

static int check_selective_f32(void) {
  const int64_t B = 1, D = 2, N = 1, L = 3000, n = B * D * L;
  float* host = (float*)malloc((size_t)n * sizeof(float));
  float *x, *dl, *A, *Bm, *Cm, *Dk, *y, *hl;
  float hlh[2], zero[2] = {0.0f, 0.0f}, two[2] = {2.0f, 2.0f};
  int64_t i, r;
  if (!host) return fail("host allocation");
  HIPCHK(hipMalloc((void**)&x, (size_t)n * sizeof(float)));
  HIPCHK(hipMalloc((void**)&dl, (size_t)n * sizeof(float)));
  HIPCHK(hipMalloc((void**)&y, (size_t)n * sizeof(float)));
  HIPCHK(hipMalloc((void**)&Bm, (size_t)(B * L * N) * sizeof(float)));
  HIPCHK(hipMalloc((void**)&Cm, (size_t)(B * L * N) * sizeof(float)));
  HIPCHK(hipMalloc((void**)&A, (size_t)(D * N) * sizeof(float)));
  HIPCHK(hipMalloc((void**)&Dk, (size_t)D * sizeof(float)));
  HIPCHK(hipMalloc((void**)&hl, (size_t)(B * D * N) * sizeof(float)));
  for (i = 0; i < n; ++i) host[i] = 1.0f;
  HIPCHK(hipMemcpy(x, host, (size_t)n * sizeof(float), hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(Bm, host, (size_t)(B * L * N) * sizeof(float), hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(Cm, host, (size_t)(B * L * N) * sizeof(float), hipMemcpyHostToDevice));
  for (i = 0; i < n; ++i) host[i] = 0.5f;
  HIPCHK(hipMemcpy(dl, host, (size_t)n * sizeof(float), hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(A, zero, (size_t)(D * N) * sizeof(float), hipMemcpyHostToDevice));
  HIPCHK(hipMemcpy(Dk, two, (size_t)D * sizeof(float), hipMemcpyHostToDevice));
  if (sw_selective_scan_fwd(x, dl, A, Bm, Cm, Dk, y, hl, B, D, N, L) != SW_OK)
    return fail("sw_selective_scan_fwd");
  HIPCHK(hipDeviceSynchronize());
  HIPCHK(hipMemcpy(host, y, (size_t)n * sizeof(float), hipMemcpyDeviceToHost));
  HIPCHK(hipMemcpy(hlh, hl, sizeof(hlh), hipMemcpyDeviceToHost));
  for (r = 0; r < B * D; ++r) {
    for (i = 0; i < L; ++i)
      if (host[r * L + i] != 0.5f * (float)(i + 1) + 2.0f) return fail("fused scan y");
    if (hlh[r] != 0.5f * (float)L) return fail("fused scan h_last");
  }
  HIPCHK(hipFree(x));
  HIPCHK(hipFree(dl));
  HIPCHK(hipFree(y));
  HIPCHK(hipFree(Bm));
  HIPCHK(hipFree(Cm));
  HIPCHK(hipFree(A));
  HIPCHK(hipFree(Dk));
  HIPCHK(hipFree(hl));
  free(host);
  return 0;
}

int main(void) {
  int rc;
  printf("library version %d\n", sw_version());
  fflush(stdout);
  rc = check_affine_i32();
  if (rc) return rc;
  rc = check_selective_f32();
  if (rc) return rc;
  printf("abi consumer ok\n");
  return 0;
}
