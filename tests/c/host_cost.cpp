// Host cost of enqueuing the library's calls, through the C ABI alone.
//
// For each call: the best over 60 bursts of 20 back-to-back calls of the
// host time per call (the GPU is synchronised between bursts, so no burst
// waits on a full queue); then the same calls 2000 times back to back, whose
// wall time per call is the larger of the host and the GPU time.  Beside
// them, the HIP runtime calls a library call makes: a launch of an empty
// kernel, the pointer and device queries.  Inputs are zero (the values do
// not matter here; the tests check results).  Prints one line per figure.
#include <hip/hip_runtime.h>
#include <stdio.h>

#include <chrono>
#include <functional>

#include "scanweaver.h"

__global__ void empty_kernel(int* p) {
  if (p && threadIdx.x == 1u << 20) p[0] = 1;  // never true: the launch is all there is
}

static int burst_us(const char* name, const std::function<void()>& f) {
  double best = 1e30;
  for (int round = 0; round < 60; ++round) {
    const auto t0 = std::chrono::steady_clock::now();
    for (int i = 0; i < 20; ++i) f();
    const auto t1 = std::chrono::steady_clock::now();
    if (hipDeviceSynchronize() != hipSuccess) return 1;
    const double us = std::chrono::duration<double, std::micro>(t1 - t0).count() / 20;
    if (us < best) best = us;
  }
  printf("enqueue %-48s %7.3f us\n", name, best);
  return 0;
}

static int loop_us(const char* name, const std::function<void()>& f) {
  if (hipDeviceSynchronize() != hipSuccess) return 1;
  const auto t0 = std::chrono::steady_clock::now();
  for (int i = 0; i < 2000; ++i) f();
  if (hipDeviceSynchronize() != hipSuccess) return 1;
  const auto t1 = std::chrono::steady_clock::now();
  printf("back to back %-43s %7.3f us\n", name,
         std::chrono::duration<double, std::micro>(t1 - t0).count() / 2000);
  return 0;
}

int main() {
  const int64_t B = 2, D = 256, N = 16, L = 512, R1 = 64, L1 = 1024;
  const size_t nbare = (size_t)R1 * L1, nx = (size_t)B * D * L, nbc = (size_t)B * L * N;
  float *a, *bx, *h, *x, *dl, *A, *Bm, *Cm, *Ds, *y, *hl;
  float** bufs[] = {&a, &bx, &h, &x, &dl, &A, &Bm, &Cm, &Ds, &y, &hl};
  const size_t sizes[] = {nbare, nbare, nbare, nx, nx, (size_t)D * N, nbc, nbc, (size_t)D, nx,
                          (size_t)B * D * N};
  for (int i = 0; i < 11; ++i) {
    if (hipMalloc(bufs[i], sizes[i] * 4) != hipSuccess) return 2;
    if (hipMemset(*bufs[i], 0, sizes[i] * 4) != hipSuccess) return 2;
  }
  if (hipDeviceSynchronize() != hipSuccess) return 2;
  auto bare = [&] { (void)sw_affine_scan(a, bx, nullptr, h, 1, R1, L1); };
  auto bare_noalloc = [&] { (void)sw_affine_scan_noalloc(a, bx, nullptr, h, 1, R1, L1); };
  auto fused = [&] { (void)sw_selective_scan_fwd(x, dl, A, Bm, Cm, Ds, y, hl, B, D, N, L); };
  if (sw_affine_scan(a, bx, nullptr, h, 1, R1, L1) != SW_OK ||
      sw_affine_scan_noalloc(a, bx, nullptr, h, 1, R1, L1) != SW_OK ||
      sw_selective_scan_fwd(x, dl, A, Bm, Cm, Ds, y, hl, B, D, N, L) != SW_OK) {
    printf("call failed: %s\n", sw_last_error());
    return 1;
  }
  int rc = 0;
  rc |= burst_us("empty kernel launch", [] {
    hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, nullptr, nullptr);
  });
  rc |= burst_us("hipPointerGetAttributes", [&] {
    hipPointerAttribute_t at;
    (void)hipPointerGetAttributes(&at, x);
  });
  rc |= burst_us("hipGetDevice", [] {
    int d;
    (void)hipGetDevice(&d);
  });
  rc |= burst_us("sw_affine_scan B=1 D=64 L=1024", bare);
  rc |= burst_us("sw_affine_scan_noalloc B=1 D=64 L=1024", bare_noalloc);
  rc |= burst_us("sw_selective_scan_fwd B=2 D=256 N=16 L=512", fused);
  printf("fused launch: %s\n", sw_last_launch());
  rc |= loop_us("sw_affine_scan B=1 D=64 L=1024", bare);
  rc |= loop_us("sw_selective_scan_fwd B=2 D=256 N=16 L=512", fused);
  for (int i = 0; i < 11; ++i) (void)hipFree(*bufs[i]);
  if (rc) return 1;
  printf("host cost done\n");
  return 0;
}
