// sw_internal.h -- shared host/device helpers of libscanweaver (not installed).
//
// Holds: error bookkeeping and the per-thread stream of the C ABI, the exact
// bf16 -> fp32 widening, the affine-pair arithmetic of Eq. (7) for fp32 and
// for Z/2^32, the wavefront-level inclusive scan of pairs built on DPP, and
// the status words used to pass chunk carries between workgroups.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scanweaver.h"

#define SW_API extern "C" __attribute__((visibility("default")))

namespace sw {

// ---------------------------------------------------------------- host side
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
hipStream_t current_stream();
int check_launch(const char* what);  // hipGetLastError -> SW_ERR_HIP with a message
// Records, for sw_last_launch(), which kernels the calling thread's last
// fused forward or backward call enqueued.
void note_launch(const char* fmt, ...) __attribute__((format(printf, 1, 2)));

// Compute units of the current device (looked up once per device), written
// to *cus; returns SW_OK or SW_ERR_HIP with the message set.
int device_cus(int* cus);

// Zero `words` 32-bit words with a plain kernel (no memset node).
int zero_words(uint32_t* p, size_t words, hipStream_t s);

// Persistent scratch of one (device, stream): carry words passed between
// workgroups and a ticket counter.  It is zeroed once when (re)allocated and
// never again: each launch tags the carry words it writes with a fresh
// epoch, so words left by earlier launches never match, and the ticket
// counter only grows (a launch knows the value it starts from).  The session
// holds a lock from reserve() until it is destroyed, so the order in which
// launches are enqueued on the stream is the order in which epochs and ticket
// ranges were handed out.
struct ScratchSession {
  ScratchSession();
  ~ScratchSession();
  ScratchSession(const ScratchSession&) = delete;
  ScratchSession& operator=(const ScratchSession&) = delete;
  // Make room for `carry_words` 64-bit words on stream `s`; the launch will
  // consume exactly `tickets` tickets.  Fills carry / ticket / ticket_base /
  // epoch.  Returns SW_OK or an error status.
  int reserve(size_t carry_words, uint32_t tickets, hipStream_t s);
  // The launch that reserved could not be enqueued: the ticket count handed
  // out no longer matches the device counter, so start afresh next time.
  void invalidate();
  unsigned long long* carry = nullptr;
  uint32_t* ticket = nullptr;
  uint32_t ticket_base = 0;
  uint32_t epoch = 0;  // in [1, 2^30)
 private:
  bool locked_ = false;
  int dev_ = -1;
  hipStream_t stream_ = nullptr;
};

// Arguments of one fused selective scan call, already validated.  x, delta,
// Bm, Cm and z are fp32 or bf16 (raw bits) as `bf16_in` says; y is fp32 or
// bf16 bits as `y_bf16` says.  z, delta_bias, h0, Dskip and h_last may be NULL.
struct SelArgs {
  const void *x, *delta, *Bm, *Cm, *z;
  const float *A, *Dskip, *delta_bias, *h0;
  void* y;
  float* h_last;
  int64_t B, D, N, L;
  bool bf16_in, y_bf16, softplus, vec;
  bool blelloch = false;  // the paper's schedule (plain form only)
  float* ckpt = nullptr;  // (B*D, ceil(L/8), 16): states at 8-step boundaries (N <= 16)
  float* s_out = nullptr;  // (B, D, L) fp32: y before the output gate (with the options)
};
int selective_fwd(const SelArgs& a);
int selective_blelloch_fwd(const SelArgs& a);
// The kernels a forward call takes: layout 16 (one lane per state), 4 (four
// lanes per row, four states each) or 8 (the 8-lane kernel of any N, which
// chains its own sequence chunks); nseg segments of lseg steps (the last
// the rest; 1 and L for whole rows); form 0 whole rows, 1 records, 2
// correction.  Layout 0, nseg 0: nothing to launch (B*D or L zero).
struct SelPlan {
  int layout = 0;
  int64_t nseg = 0, lseg = 0;
  int form = 0;
};
// The plan of selective_fwd for `a` priced for `cus` compute units (the
// pointers of `a` are only tested for alignment; nothing is launched).
SelPlan selective_plan(const SelArgs& a, int cus);
// The states of the forward walk without y: the 8-step checkpoints (a.ckpt,
// required) and h_last if given, for a backward call without the forward's
// checkpoints.  Enqueues (*taken = true) only where the forward takes its
// 16-lane layout and no gate, bf16 y or pre-gate output is asked for;
// otherwise returns SW_OK with nothing enqueued.
int selective_states_fwd(const SelArgs& a, bool* taken);

// Arguments of one backward call of the fused form, already validated.
// x, delta, Bm, Cm, z are fp32 or bf16 as `bf16_in` says, dy as `dy_bf16`
// says; gradients are fp32.  Optional inputs (NULL: absent): Dskip, z,
// delta_bias, h0, dh_last; optional outputs: dDskip (with Dskip), dz (with z),
// ddelta_bias (with delta_bias), dh0.
struct BwdArgs {
  const void *x, *delta, *Bm, *Cm, *z, *dy;
  const float *A, *Dskip, *delta_bias, *h0, *dh_last;
  const float* ckpt;  // the forward's states at 8-step boundaries, or NULL (recomputed)
  const float* s_pre;  // the forward's output before the gate, or NULL (recomputed)
  float *dx, *ddelta, *dA, *dB, *dC, *dDskip, *dz, *ddelta_bias, *dh0;
  int64_t B, D, N, L;
  bool bf16_in, dy_bf16, softplus, vec;  // vec: x and delta allow the forward's vector path
};
int selective_bwd(const BwdArgs& a);

// Stream-ordered workspace (hipMallocAsync / hipFreeAsync on `s`; freed
// blocks stay in the device's pool).
int workspace_alloc(void** p, size_t bytes, hipStream_t s);
void workspace_free(void* p, hipStream_t s);

// Flags of the fused kernels (runtime, wave-uniform).
enum : uint32_t { SEL_SOFTPLUS = 1u, SEL_Y_BF16 = 2u, SEL_GATED = 4u };

// ---------------------------------------------------------------- device side

// bf16 bits -> fp32, exact.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_one(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN), two at a time:
// gfx950 converts a pair in one instruction (v_cvt_pk_bf16_f32); lo goes to
// bits 0-15, hi to bits 16-31.
typedef __bf16 sw_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  const sw_bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint32_t bf16_rne(float v) { return bf16x2_rne(v, 0.0f) & 0xffffu; }

// softplus(v) = log(1 + e^v) in fp32 from the hardware exp2/log2/rcp, a few
// ulps: e^-v is negligible past v = 16; log1p(u) = log(w) * u / (w - 1) with
// w = 1 + u keeps the small-u end accurate (w == 1 means log1p(u) = u).
__device__ __forceinline__ float softplus_f32(float v) {
  constexpr float LOG2E_ = 1.4426950408889634f, LN2_ = 0.6931471805599453f;
  if (v > 16.0f) return v + __builtin_amdgcn_exp2f(-v * LOG2E_);
  const float u = __builtin_amdgcn_exp2f(v * LOG2E_);
  const float w = 1.0f + u;
  if (w == 1.0f) return u;
  return __builtin_amdgcn_logf(w) * LN2_ * (u * __builtin_amdgcn_rcpf(w - 1.0f));
}

// silu(z) = z / (1 + e^-z) in fp32 (exp2 and rcp; 0 for z -> -inf).
__device__ __forceinline__ float silu_f32(float z) {
  constexpr float LOG2E_ = 1.4426950408889634f;
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-z * LOG2E_));
}

// Affine-pair arithmetic.  combine(later, earlier) is Eq. (7):
//   (A2,U2) (+) (A1,U1) = (A2*A1, A2*U1 + U2).
template <typename T>
struct Ring;

template <>
struct Ring<float> {
  static constexpr float one() { return 1.0f; }
  static constexpr float zero() { return 0.0f; }
  static __device__ __forceinline__ float mul(float a, float b) { return a * b; }
  static __device__ __forceinline__ float mad(float a, float b, float c) {
    return __builtin_fmaf(a, b, c);
  }
  static __device__ __forceinline__ uint32_t bits(float v) { return __float_as_uint(v); }
  static __device__ __forceinline__ float from_bits(uint32_t v) { return __uint_as_float(v); }
};

template <>
struct Ring<uint32_t> {
  static constexpr uint32_t one() { return 1u; }
  static constexpr uint32_t zero() { return 0u; }
  static __device__ __forceinline__ uint32_t mul(uint32_t a, uint32_t b) { return a * b; }
  static __device__ __forceinline__ uint32_t mad(uint32_t a, uint32_t b, uint32_t c) {
    return a * b + c;  // unsigned: wraps modulo 2^32
  }
  static __device__ __forceinline__ uint32_t bits(uint32_t v) { return v; }
  static __device__ __forceinline__ uint32_t from_bits(uint32_t v) { return v; }
};

// (A,U) <- (A,U) (+) (Ap,Up)   where (Ap,Up) is the earlier segment.
template <typename T>
__device__ __forceinline__ void absorb_earlier(T& A, T& U, T Ap, T Up) {
  U = Ring<T>::mad(A, Up, U);
  A = Ring<T>::mul(A, Ap);
}

// DPP controls (GFX9 encoding).
enum : int {
  DPP_ROW_SHR1 = 0x111,
  DPP_ROW_SHR2 = 0x112,
  DPP_ROW_SHR4 = 0x114,
  DPP_ROW_SHR8 = 0x118,
  DPP_WAVE_SHR1 = 0x138,
  DPP_ROW_BCAST15 = 0x142,
  DPP_ROW_BCAST31 = 0x143,
};

// Move `v` across lanes with DPP; lanes without a valid source, or outside
// row_mask, receive `ident`.
template <int CTRL, int ROW_MASK, typename T>
__device__ __forceinline__ T dpp_or(T v, T ident) {
  uint32_t r = (uint32_t)__builtin_amdgcn_update_dpp((int)Ring<T>::bits(ident),
                                                     (int)Ring<T>::bits(v), CTRL, ROW_MASK, 0xf,
                                                     false);
  return Ring<T>::from_bits(r);
}

template <int CTRL, int ROW_MASK, typename T>
__device__ __forceinline__ void scan_step(T& A, T& U) {
  T Ap = dpp_or<CTRL, ROW_MASK>(A, Ring<T>::one());
  T Up = dpp_or<CTRL, ROW_MASK>(U, Ring<T>::zero());
  absorb_earlier(A, U, Ap, Up);
}

// Inclusive scan of one affine pair per lane across the 64 lanes of a
// wavefront (lane i ends with p_i (+) ... (+) p_0).  Kogge-Stone within each
// 16-lane row (shifts 1, 2, 4, 8), then the row carries via row_bcast:15 and
// row_bcast:31.  Lanes with no source keep the identity pair (1, 0).
template <typename T>
__device__ __forceinline__ void wave_inclusive_scan(T& A, T& U) {
  scan_step<DPP_ROW_SHR1, 0xf>(A, U);
  scan_step<DPP_ROW_SHR2, 0xf>(A, U);
  scan_step<DPP_ROW_SHR4, 0xf>(A, U);
  scan_step<DPP_ROW_SHR8, 0xf>(A, U);
  scan_step<DPP_ROW_BCAST15, 0xa>(A, U);
  scan_step<DPP_ROW_BCAST31, 0xc>(A, U);
}

// Inclusive -> exclusive: lane i receives lane i-1's pair, lane 0 the identity.
template <typename T>
__device__ __forceinline__ void wave_shift_exclusive(T& A, T& U) {
  A = dpp_or<DPP_WAVE_SHR1, 0xf>(A, Ring<T>::one());
  U = dpp_or<DPP_WAVE_SHR1, 0xf>(U, Ring<T>::zero());
}

// ------------------------------------------------------- workgroup order
// The dispatcher deals a launch's workgroups to the 8 XCDs in turn
// (workgroup i to XCD i % 8), and each XCD has its own L2.  This renumbers
// the first 8 * floor(n / 8) workgroups so that XCD x takes the contiguous
// range [x * n/8, (x + 1) * n/8) of logical workgroups: neighbours in the
// logical order (the row blocks of one batch, which read the same B and C;
// the row blocks of one segment) then share an L2.  A bijection on [0, n);
// the tail keeps its place.
__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t i, uint32_t n) {
  const uint32_t per = n / 8;
  if (i >= 8 * per) return i;
  return (i % 8) * per + i / 8;
}

// ------------------------------------------------------------- carry words
// A carry word is 64 bits: status in the high half, a 32-bit payload in the
// low half, written and read with single relaxed device-scope atomics, so a
// reader either sees the whole word or the previous one, and no fence is
// needed between payload and flag.  Status encodes the launch's epoch and a
// kind; words from earlier launches carry older epochs and never match.
enum : uint32_t { CARRY_EMPTY = 0, CARRY_AGG = 1, CARRY_INC = 2 };

__device__ __forceinline__ uint32_t carry_status(uint32_t epoch, uint32_t kind) {
  return (epoch << 2) | kind;
}

__device__ __forceinline__ void carry_put(unsigned long long* w, uint32_t status, uint32_t payload) {
  unsigned long long v = ((unsigned long long)status << 32) | payload;
  __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned long long carry_get(const unsigned long long* w) {
  return __hip_atomic_load(const_cast<unsigned long long*>(w), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace sw
