// sw_api.hip -- the C ABI of libscanweaver.so: argument validation, the
// per-thread stream, error reporting and dispatch to the kernels.
// Declarations and the full contract are in include/scanweaver.h.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <map>
#include <mutex>
#include <utility>

#include "sw_internal.h"

namespace sw {

int affine_scan_f32(const float* a, const float* bx, const float* h0, float* h, int64_t R,
                    int64_t L, bool vec);
int affine_scan_u32(const uint32_t* a, const uint32_t* bx, const uint32_t* h0, uint32_t* h,
                    int64_t R, int64_t L, bool vec);
int affine_scan_f32_noalloc(const float* a, const float* bx, const float* h0, float* h,
                            int64_t R, int64_t L, bool vec);
int affine_blelloch_f32(const float* a, const float* bx, const float* h0, float* h, int64_t R,
                        int64_t L, bool vec);
int affine_blelloch_u32(const uint32_t* a, const uint32_t* bx, const uint32_t* h0, uint32_t* h,
                        int64_t R, int64_t L, bool vec);
int affine_scan_io_f32(const float* a, const float* b, const float* x, const float* c,
                       const float* h0, float* y, float* h_last, int64_t R, int64_t L, bool vec);
int affine_scan_io_u32(const uint32_t* a, const uint32_t* b, const uint32_t* x, const uint32_t* c,
                       const uint32_t* h0, uint32_t* y, uint32_t* h_last, int64_t R, int64_t L,
                       bool vec);

namespace {
thread_local hipStream_t tls_stream = nullptr;
thread_local char tls_msg[512] = "";
thread_local char tls_launch[256] = "";
bool pool_ready[64] = {};  // guarded by scratch_mu

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = 0u;
}

// ------------------------------------------------------------ validation

struct Span {
  const void* p;
  size_t bytes;
  const char* name;
};

bool overlaps(const Span& a, const Span& b) {
  if (!a.p || !b.p || a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = (uintptr_t)a.p, b0 = (uintptr_t)b.p;
  return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

// Multiply non-negative sizes; false on overflow of int64.
bool mul_ok(int64_t a, int64_t b, int64_t* out) { return !__builtin_mul_overflow(a, b, out); }

int check_ptr(const void* p, size_t align, const char* name, bool required, int device) {
  if (!p) {
    if (required) return fail(SW_ERR_INVALID_ARG, "%s is NULL", name);
    return SW_OK;
  }
  if ((uintptr_t)p % align != 0)
    return fail(SW_ERR_INVALID_ARG, "%s is not %zu-byte aligned", name, align);
  hipPointerAttribute_t attr;
  memset(&attr, 0, sizeof(attr));
  hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();  // the query failure is not a sticky launch error
    return fail(SW_ERR_INVALID_ARG, "%s is not device memory (%s)", name, hipGetErrorString(e));
  }
  if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged &&
      attr.type != hipMemoryTypeUnified)
    return fail(SW_ERR_INVALID_ARG, "%s is not device memory (memory type %d)", name,
                (int)attr.type);
  if (attr.device != device)
    return fail(SW_ERR_INVALID_ARG, "%s lives on device %d, current device is %d", name,
                attr.device, device);
  return SW_OK;
}

int current_device(int* dev) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return fail(SW_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  return SW_OK;
}

int check_spans(const Span* outs, int nout, const Span* ins, int nin) {
  for (int i = 0; i < nout; ++i) {
    for (int j = 0; j < nin; ++j)
      if (overlaps(outs[i], ins[j]))
        return fail(SW_ERR_INVALID_ARG, "output %s overlaps input %s", outs[i].name,
                    ins[j].name);
    for (int j = i + 1; j < nout; ++j)
      if (overlaps(outs[i], outs[j]))
        return fail(SW_ERR_INVALID_ARG, "outputs %s and %s overlap", outs[i].name,
                    outs[j].name);
  }
  return SW_OK;
}

bool all_aligned16(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (p && (uintptr_t)p % 16 != 0) return false;
  return true;
}

template <typename T>
int affine_common(const T* a, const T* bx, const T* h0, T* h_out, int64_t B, int64_t D,
                  int64_t L, int (*run)(const T*, const T*, const T*, T*, int64_t, int64_t, bool)) {
  if (B < 0 || D < 0 || L < 0)
    return fail(SW_ERR_INVALID_ARG, "negative size (B=%lld D=%lld L=%lld)", (long long)B,
                (long long)D, (long long)L);
  int64_t R, n;
  if (!mul_ok(B, D, &R) || !mul_ok(R, L, &n) || !mul_ok(n, (int64_t)sizeof(T), &n))
    return fail(SW_ERR_UNSUPPORTED, "B*D*L overflows");
  if (R == 0 || L == 0) return SW_OK;
  int dev, st;
  if ((st = current_device(&dev)) != SW_OK) return st;
  if ((st = check_ptr(a, sizeof(T), "a", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(bx, sizeof(T), "bx", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(h0, sizeof(T), "h0", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(h_out, sizeof(T), "h_out", true, dev)) != SW_OK) return st;
  const size_t big = (size_t)n, small = (size_t)R * sizeof(T);
  Span outs[] = {{h_out, big, "h_out"}};
  Span ins[] = {{a, big, "a"}, {bx, big, "bx"}, {h0, small, "h0"}};
  if ((st = check_spans(outs, 1, ins, 3)) != SW_OK) return st;
  const bool vec = L % 4 == 0 && all_aligned16({a, bx, h_out});
  return run(a, bx, h0, h_out, R, L, vec);
}

// Validation of the output-projection form (Eq. (3)-(4)); see include/scanweaver.h.
template <typename T>
int affine_proj_common(const T* a, const T* b, const T* x, const T* c, const T* h0, T* y,
                       T* h_last, int64_t B, int64_t D, int64_t L,
                       int (*run)(const T*, const T*, const T*, const T*, const T*, T*, T*,
                                  int64_t, int64_t, bool)) {
  if (B < 0 || D < 0 || L < 0)
    return fail(SW_ERR_INVALID_ARG, "negative size (B=%lld D=%lld L=%lld)", (long long)B,
                (long long)D, (long long)L);
  int64_t R, n;
  if (!mul_ok(B, D, &R) || !mul_ok(R, L, &n) || !mul_ok(n, (int64_t)sizeof(T), &n))
    return fail(SW_ERR_UNSUPPORTED, "B*D*L overflows");
  if (R == 0) return SW_OK;
  int dev, st;
  if ((st = current_device(&dev)) != SW_OK) return st;
  const size_t big = (size_t)n, small = (size_t)R * sizeof(T);
  if ((st = check_ptr(h0, sizeof(T), "h0", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(h_last, sizeof(T), "h_last", false, dev)) != SW_OK) return st;
  if (L == 0) {
    if (!h_last) return SW_OK;
    Span o[] = {{h_last, small, "h_last"}};
    Span i[] = {{h0, small, "h0"}};
    if ((st = check_spans(o, 1, i, 1)) != SW_OK) return st;
    if (!h0) return zero_words(reinterpret_cast<uint32_t*>(h_last), (size_t)R, current_stream());
    // the final state of an empty sequence is the initial one
    hipError_t e = hipMemcpyAsync(h_last, h0, small, hipMemcpyDeviceToDevice, current_stream());
    if (e != hipSuccess) return fail(SW_ERR_HIP, "h_last copy: %s", hipGetErrorString(e));
    return SW_OK;
  }
  if ((st = check_ptr(a, sizeof(T), "a", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(b, sizeof(T), "b", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(x, sizeof(T), "x", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(c, sizeof(T), "c", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(y, sizeof(T), "y", true, dev)) != SW_OK) return st;
  Span outs[] = {{y, big, "y"}, {h_last, small, "h_last"}};
  Span ins[] = {{a, big, "a"}, {b, big, "b"}, {x, big, "x"}, {c, big, "c"}, {h0, small, "h0"}};
  if ((st = check_spans(outs, 2, ins, 5)) != SW_OK) return st;
  const bool vec = L % 4 == 0 && all_aligned16({a, b, x, c, y});
  return run(a, b, x, c, h0, y, h_last, R, L, vec);
}

// Validation shared by the fused entry points; see include/scanweaver.h.
int selective_common(SelArgs a) {
  const int64_t B = a.B, D = a.D, N = a.N, L = a.L;
  if (B < 0 || D < 0 || L < 0 || N < 0)
    return fail(SW_ERR_INVALID_ARG, "negative size (B=%lld D=%lld N=%lld L=%lld)",
                (long long)B, (long long)D, (long long)N, (long long)L);
  if (N < 1 || N > 64) return fail(SW_ERR_UNSUPPORTED, "N=%lld outside [1, 64]", (long long)N);
  int64_t R, nx, nbc, nh, tmp;
  if (!mul_ok(B, D, &R) || !mul_ok(R, L, &nx) || !mul_ok(nx, 4, &tmp) || !mul_ok(B, L, &nbc) ||
      !mul_ok(nbc, N, &nbc) || !mul_ok(nbc, 4, &tmp) || !mul_ok(R, N, &nh))
    return fail(SW_ERR_UNSUPPORTED, "sizes overflow");
  if (R == 0) return SW_OK;
  const int64_t blocks = B * ((D + 31) / 32);
  if (blocks >= ((int64_t)1 << 24))
    return fail(SW_ERR_UNSUPPORTED, "B*ceil(D/32)=%lld workgroups exceed the launch limit",
                (long long)blocks);
  int dev, st;
  if ((st = current_device(&dev)) != SW_OK) return st;
  if (L == 0) {
    if (!a.h_last) return SW_OK;
    if ((st = check_ptr(a.h_last, 4, "h_last", true, dev)) != SW_OK) return st;
    if ((st = check_ptr(a.h0, 4, "h0", false, dev)) != SW_OK) return st;
    if (a.h0) {
      // the final state of an empty sequence is the initial one
      Span o[] = {{a.h_last, (size_t)nh * 4, "h_last"}};
      Span i[] = {{a.h0, (size_t)nh * 4, "h0"}};
      if ((st = check_spans(o, 1, i, 1)) != SW_OK) return st;
      hipError_t e = hipMemcpyAsync(a.h_last, a.h0, (size_t)nh * 4, hipMemcpyDeviceToDevice,
                                    current_stream());
      if (e != hipSuccess) return fail(SW_ERR_HIP, "h_last copy: %s", hipGetErrorString(e));
      return SW_OK;
    }
    return zero_words(reinterpret_cast<uint32_t*>(a.h_last), (size_t)nh, current_stream());
  }
  const size_t es = a.bf16_in ? 2 : 4, ys = a.y_bf16 ? 2 : 4;
  if ((st = check_ptr(a.x, es, "x", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.delta, es, "delta", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.A, 4, "A", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.Bm, es, "Bm", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.Cm, es, "Cm", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.Dskip, 4, "Dskip", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.z, es, "z", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.delta_bias, 4, "delta_bias", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.h0, 4, "h0", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.y, ys, "y", true, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.h_last, 4, "h_last", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.ckpt, 4, "ckpt", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.s_out, 4, "s_pre", false, dev)) != SW_OK) return st;
  if (a.ckpt && N > 16)
    return fail(SW_ERR_UNSUPPORTED, "checkpoints need N <= 16 (got %lld)", (long long)N);
  const size_t nck = (size_t)R * (size_t)((L + 7) / 8) * 16;
  Span outs[] = {{a.y, (size_t)nx * ys, "y"}, {a.h_last, (size_t)nh * 4, "h_last"},
                 {a.ckpt, nck * 4, "ckpt"}, {a.s_out, (size_t)nx * 4, "s_pre"}};
  Span ins[] = {{a.x, (size_t)nx * es, "x"},          {a.delta, (size_t)nx * es, "delta"},
                {a.A, (size_t)(D * N) * 4, "A"},      {a.Bm, (size_t)nbc * es, "Bm"},
                {a.Cm, (size_t)nbc * es, "Cm"},       {a.Dskip, (size_t)D * 4, "Dskip"},
                {a.z, (size_t)nx * es, "z"},          {a.delta_bias, (size_t)D * 4, "delta_bias"},
                {a.h0, (size_t)nh * 4, "h0"}};
  if ((st = check_spans(outs, 4, ins, 9)) != SW_OK) return st;
  a.vec = L % 4 == 0 && all_aligned16({a.x, a.delta, a.y, a.z, a.s_out});
  return a.blelloch ? selective_blelloch_fwd(a) : selective_fwd(a);
}

// Validation of the backward entry point; see include/scanweaver.h.
int selective_bwd_common(BwdArgs a) {
  const int64_t B = a.B, D = a.D, N = a.N, L = a.L;
  if (B < 0 || D < 0 || L < 0 || N < 0)
    return fail(SW_ERR_INVALID_ARG, "negative size (B=%lld D=%lld N=%lld L=%lld)",
                (long long)B, (long long)D, (long long)N, (long long)L);
  if (N < 1 || N > 64) return fail(SW_ERR_UNSUPPORTED, "N=%lld outside [1, 64]", (long long)N);
  int64_t R, nx, nbc, nh, nan, tmp;
  if (!mul_ok(B, D, &R) || !mul_ok(R, L, &nx) || !mul_ok(nx, 4, &tmp) || !mul_ok(B, L, &nbc) ||
      !mul_ok(nbc, N, &nbc) || !mul_ok(nbc, 4, &tmp) || !mul_ok(R, N, &nh) ||
      !mul_ok(D, N, &nan) || !mul_ok(R, 16 * ((L + 7) / 8 + 1), &tmp) || !mul_ok(tmp, 8, &tmp))
    return fail(SW_ERR_UNSUPPORTED, "sizes overflow");
  if (a.dz && !a.z) return fail(SW_ERR_INVALID_ARG, "dz requires z");
  if (a.s_pre && !a.z) return fail(SW_ERR_INVALID_ARG, "s_pre requires z");
  if (a.ckpt && N > 16)
    return fail(SW_ERR_UNSUPPORTED, "checkpoints hold 16 states (got N=%lld)", (long long)N);
  int dev, st;
  if ((st = current_device(&dev)) != SW_OK) return st;
  const size_t es = a.bf16_in ? 2 : 4, dys = a.dy_bf16 ? 2 : 4;
  const bool empty = R == 0 || L == 0;
  // inputs
  if ((st = check_ptr(a.x, es, "x", !empty, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.delta, es, "delta", !empty, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.A, 4, "A", !empty, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.Bm, es, "Bm", !empty, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.Cm, es, "Cm", !empty, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.Dskip, 4, "Dskip", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.z, es, "z", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.delta_bias, 4, "delta_bias", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.h0, 4, "h0", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.dy, dys, "dy", !empty, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.dh_last, 4, "dh_last", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.ckpt, 4, "ckpt", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.s_pre, 4, "s_pre", false, dev)) != SW_OK) return st;
  // outputs
  if ((st = check_ptr(a.dx, 4, "dx", nx > 0, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.ddelta, 4, "ddelta", nx > 0, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.dA, 4, "dA", nan > 0, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.dB, 4, "dB", nbc > 0, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.dC, 4, "dC", nbc > 0, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.dDskip, 4, "dDskip", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.dz, 4, "dz", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.ddelta_bias, 4, "ddelta_bias", false, dev)) != SW_OK) return st;
  if ((st = check_ptr(a.dh0, 4, "dh0", false, dev)) != SW_OK) return st;
  Span outs[] = {{a.dx, (size_t)nx * 4, "dx"},         {a.ddelta, (size_t)nx * 4, "ddelta"},
                 {a.dA, (size_t)nan * 4, "dA"},        {a.dB, (size_t)nbc * 4, "dB"},
                 {a.dC, (size_t)nbc * 4, "dC"},        {a.dDskip, (size_t)D * 4, "dDskip"},
                 {a.dz, (size_t)nx * 4, "dz"},         {a.ddelta_bias, (size_t)D * 4, "ddelta_bias"},
                 {a.dh0, (size_t)nh * 4, "dh0"}};
  Span ins[] = {{a.x, (size_t)nx * es, "x"},           {a.delta, (size_t)nx * es, "delta"},
                {a.A, (size_t)nan * 4, "A"},            {a.Bm, (size_t)nbc * es, "Bm"},
                {a.Cm, (size_t)nbc * es, "Cm"},         {a.Dskip, (size_t)D * 4, "Dskip"},
                {a.z, (size_t)nx * es, "z"},            {a.delta_bias, (size_t)D * 4, "delta_bias"},
                {a.h0, (size_t)nh * 4, "h0"},           {a.dy, (size_t)nx * dys, "dy"},
                {a.dh_last, (size_t)nh * 4, "dh_last"},
                {a.ckpt, (size_t)R * (size_t)((L + 7) / 8) * 64, "ckpt"},
                {a.s_pre, (size_t)nx * 4, "s_pre"}};
  if ((st = check_spans(outs, 9, ins, 13)) != SW_OK) return st;
  hipStream_t s = current_stream();
  if (empty) {
    // no step: every sum is empty, and the initial state's gradient is dh_last
    uint32_t* zs[] = {reinterpret_cast<uint32_t*>(a.dA), reinterpret_cast<uint32_t*>(a.dB),
                      reinterpret_cast<uint32_t*>(a.dC), reinterpret_cast<uint32_t*>(a.dDskip),
                      reinterpret_cast<uint32_t*>(a.ddelta_bias)};
    const size_t nw[] = {(size_t)nan, (size_t)nbc, (size_t)nbc, (size_t)D, (size_t)D};
    for (int i = 0; i < 5; ++i)
      if (zs[i] && (st = zero_words(zs[i], nw[i], s)) != SW_OK) return st;
    if (a.dh0 && nh > 0) {
      if (!a.dh_last) return zero_words(reinterpret_cast<uint32_t*>(a.dh0), (size_t)nh, s);
      hipError_t e = hipMemcpyAsync(a.dh0, a.dh_last, (size_t)nh * 4, hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return fail(SW_ERR_HIP, "dh0 copy: %s", hipGetErrorString(e));
    }
    return SW_OK;
  }
  a.vec = L % 4 == 0 && all_aligned16({a.x, a.delta});
  return selective_bwd(a);
}

SelArgs sel_args(const void* x, const void* delta, const float* A, const void* Bm, const void* Cm,
                 const float* Dskip, void* y, float* h_last, int64_t B, int64_t D, int64_t N,
                 int64_t L, bool bf16_in) {
  SelArgs a{};
  a.x = x;
  a.delta = delta;
  a.A = A;
  a.Bm = Bm;
  a.Cm = Cm;
  a.Dskip = Dskip;
  a.y = y;
  a.h_last = h_last;
  a.B = B;
  a.D = D;
  a.N = N;
  a.L = L;
  a.bf16_in = bf16_in;
  return a;
}

}  // namespace

// ------------------------------------------------------------ host helpers

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(tls_msg, sizeof(tls_msg), fmt, ap);
  va_end(ap);
  return status;
}

void note_launch(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(tls_launch, sizeof(tls_launch), fmt, ap);
  va_end(ap);
}

hipStream_t current_stream() { return tls_stream; }

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SW_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return SW_OK;
}

namespace {

struct StreamScratch {
  void* base = nullptr;   // [0, 256): ticket counter; [256, bytes): carry words
  size_t bytes = 0;
  uint32_t next_ticket = 0;
  uint32_t epoch = 0;
};

std::mutex scratch_mu;
std::map<std::pair<int, hipStream_t>, StreamScratch> scratch_map;

void keep_pool_memory(int dev) {
  if (dev < 0 || dev >= 64 || pool_ready[dev]) return;
  // keep freed blocks in the stream-ordered pool instead of returning them at every sync
  hipMemPool_t pool;
  if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
    uint64_t keep = UINT64_MAX;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
  }
  (void)hipGetLastError();
  pool_ready[dev] = true;
}

// A call that needs the per-stream scratch or a workspace cannot be captured
// into a HIP graph: a replay would repeat the ticket range and epoch the host
// handed out (the tickets are spent, so the replayed kernel writes nothing),
// and a workspace allocated per call would become a graph allocation.  Refuse
// it while `s` is capturing instead of recording a graph that replays wrongly.
int refuse_capture(hipStream_t s, const char* what) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(s, &cs);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(SW_ERR_HIP, "hipStreamIsCapturing: %s", hipGetErrorString(e));
  }
  if (cs != hipStreamCaptureStatusNone)
    return fail(SW_ERR_UNSUPPORTED,
                "this call uses %s and cannot be captured into a HIP graph (stream capture "
                "is active)", what);
  return SW_OK;
}

}  // namespace

ScratchSession::ScratchSession() {}

void ScratchSession::invalidate() {
  if (!locked_ || dev_ < 0) return;
  StreamScratch& ws = scratch_map[std::make_pair(dev_, stream_)];
  ws.bytes = 0;  // the next reserve() reallocates and zeroes
}

ScratchSession::~ScratchSession() {
  if (locked_) scratch_mu.unlock();
}

int ScratchSession::reserve(size_t carry_words, uint32_t tickets, hipStream_t s) {
  int st = refuse_capture(s, "the per-stream scratch (tickets and carries)");
  if (st != SW_OK) return st;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SW_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (!locked_) {
    scratch_mu.lock();
    locked_ = true;
  }
  dev_ = dev;
  stream_ = s;
  StreamScratch& ws = scratch_map[std::make_pair(dev, s)];
  const size_t need = 256 + carry_words * 8;
  if (ws.bytes < need || ws.epoch + 1 >= (1u << 30)) {
    if (ws.base) (void)hipFreeAsync(ws.base, s);
    ws = StreamScratch();
    keep_pool_memory(dev);
    size_t bytes = need < ((size_t)1 << 20) ? ((size_t)1 << 20) : need + need / 4;
    e = hipMallocAsync(&ws.base, bytes, s);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      ws.base = nullptr;
      return fail(SW_ERR_ALLOC, "hipMallocAsync(%zu bytes): %s", bytes, hipGetErrorString(e));
    }
    st = zero_words(reinterpret_cast<uint32_t*>(ws.base), bytes / 4, s);
    if (st != SW_OK) return st;
    ws.bytes = bytes;
  }
  ws.epoch += 1;
  epoch = ws.epoch;
  ticket = reinterpret_cast<uint32_t*>(ws.base);
  ticket_base = ws.next_ticket;
  ws.next_ticket += tickets;  // wraps modulo 2^32 together with the device counter
  carry = reinterpret_cast<unsigned long long*>(reinterpret_cast<char*>(ws.base) + 256);
  return SW_OK;
}

int workspace_alloc(void** p, size_t bytes, hipStream_t s) {
  *p = nullptr;
  int st = refuse_capture(s, "a workspace allocated per call");
  if (st != SW_OK) return st;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SW_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  {
    std::lock_guard<std::mutex> g(scratch_mu);
    keep_pool_memory(dev);
  }
  *p = nullptr;
  e = hipMallocAsync(p, bytes < 256 ? 256 : bytes, s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    *p = nullptr;
    return fail(SW_ERR_ALLOC, "hipMallocAsync(%zu bytes): %s", bytes, hipGetErrorString(e));
  }
  return SW_OK;
}

void workspace_free(void* p, hipStream_t s) {
  if (p) (void)hipFreeAsync(p, s);
}

int device_cus(int* cus) {
  static std::atomic<int> cache[64];
  *cus = 0;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(SW_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  }
  int n = (dev >= 0 && dev < 64) ? cache[dev].load(std::memory_order_relaxed) : 0;
  if (n <= 0) {
    e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess || n <= 0) {
      (void)hipGetLastError();
      return fail(SW_ERR_HIP, "compute unit count of device %d: %s", dev, hipGetErrorString(e));
    }
    if (dev >= 0 && dev < 64) cache[dev].store(n, std::memory_order_relaxed);
  }
  *cus = n;
  return SW_OK;
}

int zero_words(uint32_t* p, size_t words, hipStream_t s) {
  if (words == 0) return SW_OK;
  size_t blocks = (words + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, words);
  return check_launch("fill_zero_kernel");
}

}  // namespace sw

// ------------------------------------------------------------------ C ABI

SW_API int sw_version(void) { return 200; }

SW_API int sw_affine_scan(const float* a, const float* bx, const float* h0, float* h_out,
                          int64_t B, int64_t D, int64_t L) {
  return sw::affine_common<float>(a, bx, h0, h_out, B, D, L, sw::affine_scan_f32);
}

SW_API int sw_affine_scan_i32(const int32_t* a, const int32_t* bx, const int32_t* h0,
                              int32_t* h_out, int64_t B, int64_t D, int64_t L) {
  return sw::affine_common<uint32_t>(reinterpret_cast<const uint32_t*>(a),
                                     reinterpret_cast<const uint32_t*>(bx),
                                     reinterpret_cast<const uint32_t*>(h0),
                                     reinterpret_cast<uint32_t*>(h_out), B, D, L,
                                     sw::affine_scan_u32);
}

SW_API int sw_affine_scan_noalloc(const float* a, const float* bx, const float* h0,
                                  float* h_out, int64_t B, int64_t D, int64_t L) {
  return sw::affine_common<float>(a, bx, h0, h_out, B, D, L, sw::affine_scan_f32_noalloc);
}

SW_API int sw_affine_scan_schedule(const float* a, const float* bx, const float* h0,
                                  float* h_out, int64_t B, int64_t D, int64_t L, int schedule) {
  if (schedule == SW_SCHED_DEFAULT) return sw_affine_scan(a, bx, h0, h_out, B, D, L);
  if (schedule != SW_SCHED_BLELLOCH)
    return sw::fail(SW_ERR_INVALID_ARG, "unknown schedule %d", schedule);
  return sw::affine_common<float>(a, bx, h0, h_out, B, D, L, sw::affine_blelloch_f32);
}

SW_API int sw_affine_scan_schedule_i32(const int32_t* a, const int32_t* bx, const int32_t* h0,
                                      int32_t* h_out, int64_t B, int64_t D, int64_t L,
                                      int schedule) {
  if (schedule == SW_SCHED_DEFAULT) return sw_affine_scan_i32(a, bx, h0, h_out, B, D, L);
  if (schedule != SW_SCHED_BLELLOCH)
    return sw::fail(SW_ERR_INVALID_ARG, "unknown schedule %d", schedule);
  return sw::affine_common<uint32_t>(reinterpret_cast<const uint32_t*>(a),
                                     reinterpret_cast<const uint32_t*>(bx),
                                     reinterpret_cast<const uint32_t*>(h0),
                                     reinterpret_cast<uint32_t*>(h_out), B, D, L,
                                     sw::affine_blelloch_u32);
}

SW_API int sw_selective_scan_fwd_schedule(const void* x, const void* delta, const float* A,
                                          const void* Bm, const void* Cm, const float* Dskip,
                                          float* y, float* h_last, int64_t B, int64_t D, int64_t N,
                                          int64_t L, int in_dtype, int schedule) {
  if (in_dtype != SW_DTYPE_F32 && in_dtype != SW_DTYPE_BF16)
    return sw::fail(SW_ERR_INVALID_ARG, "unknown dtype %d", in_dtype);
  if (schedule != SW_SCHED_DEFAULT && schedule != SW_SCHED_BLELLOCH)
    return sw::fail(SW_ERR_INVALID_ARG, "unknown schedule %d", schedule);
  sw::SelArgs a = sw::sel_args(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, N, L,
                               in_dtype == SW_DTYPE_BF16);
  a.blelloch = schedule == SW_SCHED_BLELLOCH;
  return sw::selective_common(a);
}

SW_API int sw_affine_scan_proj(const float* a, const float* b, const float* x, const float* c,
                               const float* h0, float* y, float* h_last, int64_t B, int64_t D,
                               int64_t L) {
  return sw::affine_proj_common<float>(a, b, x, c, h0, y, h_last, B, D, L, sw::affine_scan_io_f32);
}

SW_API int sw_affine_scan_proj_i32(const int32_t* a, const int32_t* b, const int32_t* x,
                                   const int32_t* c, const int32_t* h0, int32_t* y,
                                   int32_t* h_last, int64_t B, int64_t D, int64_t L) {
  using U = const uint32_t*;
  return sw::affine_proj_common<uint32_t>(U(a), U(b), U(x), U(c), U(h0),
                                          reinterpret_cast<uint32_t*>(y),
                                          reinterpret_cast<uint32_t*>(h_last), B, D, L,
                                          sw::affine_scan_io_u32);
}

SW_API int sw_selective_scan_bwd(const void* x, const void* delta, const float* A,
                                 const void* Bm, const void* Cm, const float* Dskip,
                                 const void* z, const float* delta_bias, const float* h0,
                                 const void* dy, const float* dh_last, const float* ckpt,
                                 const float* s_pre, float* dx, float* ddelta,
                                 float* dA, float* dB, float* dC, float* dDskip, float* dz,
                                 float* ddelta_bias, float* dh0, int64_t B, int64_t D, int64_t N,
                                 int64_t L, int in_dtype, int dy_dtype, int flags) {
  if ((in_dtype != SW_DTYPE_F32 && in_dtype != SW_DTYPE_BF16) ||
      (dy_dtype != SW_DTYPE_F32 && dy_dtype != SW_DTYPE_BF16))
    return sw::fail(SW_ERR_INVALID_ARG, "unknown dtype (in %d, dy %d)", in_dtype, dy_dtype);
  if (flags & ~(int)SW_DELTA_SOFTPLUS)
    return sw::fail(SW_ERR_INVALID_ARG, "unknown flags 0x%x", (unsigned)flags);
  sw::BwdArgs a{};
  a.x = x;
  a.delta = delta;
  a.Bm = Bm;
  a.Cm = Cm;
  a.z = z;
  a.dy = dy;
  a.A = A;
  a.Dskip = Dskip;
  a.delta_bias = delta_bias;
  a.h0 = h0;
  a.dh_last = dh_last;
  a.ckpt = ckpt;
  a.s_pre = s_pre;
  a.dx = dx;
  a.ddelta = ddelta;
  a.dA = dA;
  a.dB = dB;
  a.dC = dC;
  a.dDskip = dDskip;
  a.dz = dz;
  a.ddelta_bias = ddelta_bias;
  a.dh0 = dh0;
  a.B = B;
  a.D = D;
  a.N = N;
  a.L = L;
  a.bf16_in = in_dtype == SW_DTYPE_BF16;
  a.dy_bf16 = dy_dtype == SW_DTYPE_BF16;
  a.softplus = (flags & SW_DELTA_SOFTPLUS) != 0;
  return sw::selective_bwd_common(a);
}

SW_API int sw_selective_scan_fwd(const float* x, const float* delta, const float* A,
                                 const float* Bm, const float* Cm, const float* Dskip, float* y,
                                 float* h_last, int64_t B, int64_t D, int64_t N, int64_t L) {
  return sw::selective_common(
      sw::sel_args(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, N, L, false));
}

SW_API int sw_selective_scan_fwd_bf16(const uint16_t* x, const uint16_t* delta, const float* A,
                                      const uint16_t* Bm, const uint16_t* Cm, const float* Dskip,
                                      float* y, float* h_last, int64_t B, int64_t D, int64_t N,
                                      int64_t L) {
  return sw::selective_common(
      sw::sel_args(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, N, L, true));
}

SW_API int sw_selective_scan_fwd_ex(const void* x, const void* delta, const float* A,
                                    const void* Bm, const void* Cm, const float* Dskip,
                                    const void* z, const float* delta_bias, const float* h0,
                                    void* y, float* h_last, int64_t B, int64_t D, int64_t N,
                                    int64_t L, int in_dtype, int out_dtype, int flags) {
  if ((in_dtype != SW_DTYPE_F32 && in_dtype != SW_DTYPE_BF16) ||
      (out_dtype != SW_DTYPE_F32 && out_dtype != SW_DTYPE_BF16))
    return sw::fail(SW_ERR_INVALID_ARG, "unknown dtype (in=%d out=%d)", in_dtype, out_dtype);
  if (flags & ~SW_DELTA_SOFTPLUS)
    return sw::fail(SW_ERR_INVALID_ARG, "unknown flags 0x%x", (unsigned)flags);
  sw::SelArgs a = sw::sel_args(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, N, L,
                               in_dtype == SW_DTYPE_BF16);
  a.z = z;
  a.delta_bias = delta_bias;
  a.h0 = h0;
  a.y_bf16 = out_dtype == SW_DTYPE_BF16;
  a.softplus = (flags & SW_DELTA_SOFTPLUS) != 0;
  return sw::selective_common(a);
}

SW_API int sw_selective_scan_plan(int64_t B, int64_t D, int64_t N, int64_t L, int in_dtype,
                                  int out_dtype, int train, int cus, int* layout, int64_t* nseg,
                                  int64_t* lseg, int* form) {
  if (!layout || !nseg || !lseg || !form)
    return sw::fail(SW_ERR_INVALID_ARG, "an output pointer is NULL");
  if ((in_dtype != SW_DTYPE_F32 && in_dtype != SW_DTYPE_BF16) ||
      (out_dtype != SW_DTYPE_F32 && out_dtype != SW_DTYPE_BF16))
    return sw::fail(SW_ERR_INVALID_ARG, "unknown dtype (in=%d out=%d)", in_dtype, out_dtype);
  if (B < 0 || D < 0 || L < 0 || N < 0)
    return sw::fail(SW_ERR_INVALID_ARG, "negative size (B=%lld D=%lld N=%lld L=%lld)",
                    (long long)B, (long long)D, (long long)N, (long long)L);
  if (N < 1 || N > 64)
    return sw::fail(SW_ERR_UNSUPPORTED, "N=%lld outside [1, 64]", (long long)N);
  if (train && N > 16)
    return sw::fail(SW_ERR_UNSUPPORTED, "checkpoints need N <= 16 (got %lld)", (long long)N);
  int64_t R, nx;
  if (!sw::mul_ok(B, D, &R) || !sw::mul_ok(R, L, &nx) || !sw::mul_ok(nx, 4, &nx))
    return sw::fail(SW_ERR_UNSUPPORTED, "sizes overflow");
  if (B * ((D + 31) / 32) >= ((int64_t)1 << 24))
    return sw::fail(SW_ERR_UNSUPPORTED, "B*ceil(D/32)=%lld workgroups exceed the launch limit",
                    (long long)(B * ((D + 31) / 32)));
  if (cus <= 0) {
    int st = sw::device_cus(&cus);
    if (st != SW_OK) return st;
  }
  // arrays as the library's own allocations would be: 16-byte aligned (the
  // pointers stand in for them and are never dereferenced)
  alignas(16) static const float stand_in[4] = {0.f, 0.f, 0.f, 0.f};
  sw::SelArgs a = sw::sel_args(stand_in, stand_in, stand_in, stand_in, stand_in, nullptr,
                               const_cast<float*>(stand_in), nullptr, B, D, N, L,
                               in_dtype == SW_DTYPE_BF16);
  a.y_bf16 = out_dtype == SW_DTYPE_BF16;
  if (train) a.ckpt = const_cast<float*>(stand_in);
  a.vec = L % 4 == 0;
  const sw::SelPlan p = sw::selective_plan(a, cus);
  *layout = p.layout;
  *nseg = p.nseg;
  *lseg = p.lseg;
  *form = p.form;
  return SW_OK;
}

SW_API int sw_selective_scan_fwd_train(const void* x, const void* delta, const float* A,
                                       const void* Bm, const void* Cm, const float* Dskip,
                                       const void* z, const float* delta_bias, const float* h0,
                                       void* y, float* h_last, float* ckpt, float* s_pre,
                                       int64_t B, int64_t D, int64_t N, int64_t L, int in_dtype,
                                       int out_dtype, int flags) {
  if (!ckpt) return sw::fail(SW_ERR_INVALID_ARG, "ckpt is NULL");
  if ((in_dtype != SW_DTYPE_F32 && in_dtype != SW_DTYPE_BF16) ||
      (out_dtype != SW_DTYPE_F32 && out_dtype != SW_DTYPE_BF16))
    return sw::fail(SW_ERR_INVALID_ARG, "unknown dtype (in=%d out=%d)", in_dtype, out_dtype);
  if (flags & ~SW_DELTA_SOFTPLUS)
    return sw::fail(SW_ERR_INVALID_ARG, "unknown flags 0x%x", (unsigned)flags);
  sw::SelArgs a = sw::sel_args(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, N, L,
                               in_dtype == SW_DTYPE_BF16);
  a.z = z;
  a.delta_bias = delta_bias;
  a.h0 = h0;
  a.y_bf16 = out_dtype == SW_DTYPE_BF16;
  a.softplus = (flags & SW_DELTA_SOFTPLUS) != 0;
  a.ckpt = ckpt;
  a.s_out = s_pre;
  return sw::selective_common(a);
}

SW_API int sw_set_stream(void* hip_stream) {
  sw::tls_stream = reinterpret_cast<hipStream_t>(hip_stream);
  return SW_OK;
}

SW_API void* sw_get_stream(void) { return reinterpret_cast<void*>(sw::tls_stream); }

SW_API const char* sw_status_string(int status) {
  switch (status) {
    case SW_OK: return "SW_OK";
    case SW_ERR_INVALID_ARG: return "SW_ERR_INVALID_ARG";
    case SW_ERR_UNSUPPORTED: return "SW_ERR_UNSUPPORTED";
    case SW_ERR_HIP: return "SW_ERR_HIP";
    case SW_ERR_ALLOC: return "SW_ERR_ALLOC";
    default: return "SW_ERR_UNKNOWN";
  }
}

SW_API const char* sw_last_error(void) { return sw::tls_msg; }

SW_API const char* sw_last_launch(void) { return sw::tls_launch; }
