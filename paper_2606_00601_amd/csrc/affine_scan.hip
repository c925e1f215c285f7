// affine_scan.hip -- bare affine scan h_t = a_t h_{t-1} + bx_t (Eq. (3)) on
// gfx950, as a prefix scan over the affine pairs of Eq. (6) under the
// composition of Eq. (7), for fp32 and for the int32 wraparound ring.
//
// One workgroup (4 wavefronts, 256 lanes) owns one chunk of K*256 consecutive
// steps of one (b,d) row:
//   1. each lane loads K consecutive (a, bx) with 16-byte vector loads
//      (consecutive lanes read consecutive 16-byte pieces: fully coalesced) and
//      composes them sequentially into its local inclusive prefixes;
//   2. the 64 lane totals of a wavefront are scanned with DPP lane moves
//      (wave_inclusive_scan) and shifted to exclusive prefixes;
//   3. the four wavefront totals go through LDS and every lane folds the
//      totals of the wavefronts before it;
//   4. rows longer than one chunk pass carries between workgroups by
//      decoupled look-back: a chunk publishes its aggregate pair, walks back
//      over its predecessors' published aggregates until it meets a published
//      inclusive state, and then publishes its own inclusive state;
//   5. every lane rebuilds its states as h = A_pre * h_in + U_pre (Sec. 3.2)
//      and stores them with 16-byte vector stores.
// The elementwise form of Eq. (3)-(4) (IO variant) forms bx = b * x at the
// load, stores y = c * h instead of h and can write the final state h_last.
// Chunks are handed out through an atomic ticket in chunk-major order (all
// rows' chunk 0 first), so a chunk only ever waits on chunks that already
// hold a ticket, which guarantees forward progress.  When the rows alone fill
// the GPU, affine_rows_kernel below walks each row in one workgroup instead
// and no carry leaves the chip.
#include <mutex>

#include "sw_internal.h"

// Scratch of the entry point that allocates nothing (sw_affine_scan_noalloc):
// the ticket counter in the first 256 bytes, then three carry words per chunk
// for at most SW_NOALLOC_MAX_CHUNKS chunks.  Each GPU holds its own copy,
// found by hipGetSymbolAddress once per device; host code uses only that
// address, never the array's name.
static __device__ __align__(256) unsigned long long scratch[32 + 3 * (int64_t)SW_NOALLOC_MAX_CHUNKS];

namespace sw {
namespace {

constexpr int AS_THREADS = 256;
constexpr int AS_WAVES = AS_THREADS / 64;

// Operands of one call.  The plain scan has b = bx, y = h and no x, c or
// h_last; the IO variant reads x (NULL: 1) and c (NULL: 1) and writes h_last
// (NULL: not written).
template <typename T>
struct AffIO {
  const T *a, *b, *x, *c, *h0;
  T *y, *h_last;
};

// y element of state hv at step t (IO: times c_t; the final state goes to h_last)
template <bool IO, typename T>
__device__ __forceinline__ T out_elem(const AffIO<T>& io, const T* __restrict__ cr, T hv,
                                      int64_t t, int64_t L, int64_t row) {
  if constexpr (IO) {
    if (io.h_last && t == L - 1) io.h_last[row] = hv;
    if (cr) return Ring<T>::mul(cr[t], hv);
  }
  return hv;
}

template <typename T, int K, bool VEC, bool IO>
__global__ __launch_bounds__(AS_THREADS) void affine_scan_kernel(
    const AffIO<T> io, int64_t R, int64_t L, int64_t nchunks, int64_t total,
    unsigned long long* __restrict__ carry, uint32_t* __restrict__ ticket, uint32_t tbase,
    uint32_t epoch) {
  static_assert(K % 4 == 0, "K must be a multiple of 4");
  constexpr int64_t CH = (int64_t)AS_THREADS * K;
  using Rg = Ring<T>;
  __shared__ T sA[AS_WAVES], sU[AS_WAVES];
  __shared__ T s_hin;
  __shared__ uint32_t s_id;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint32_t st_agg = carry_status(epoch, CARRY_AGG);
  const uint32_t st_inc = carry_status(epoch, CARRY_INC);
  int64_t id = blockIdx.x;

  for (;;) {
    if (nchunks > 1) {
      if (tid == 0) s_id = atomicAdd(ticket, 1u) - tbase;
      __syncthreads();
      id = s_id;
    }
    if (id >= total) break;  // uniform across the workgroup
    const int64_t c = id / R;
    const int64_t row = id - c * R;
    const int64_t t0 = c * CH + (int64_t)tid * K;
    const T* __restrict__ ar = io.a + row * L;
    const T* __restrict__ br = io.b + row * L;
    const T* __restrict__ xr = (IO && io.x) ? io.x + row * L : nullptr;
    const T* __restrict__ cr = (IO && io.c) ? io.c + row * L : nullptr;
    T* __restrict__ hr = io.y + row * L;

    // 1. load and local inclusive prefixes
    T pa[K], pu[K];
    if (VEC && t0 + K <= L) {
#pragma unroll
      for (int q = 0; q < K / 4; ++q) {
        uint4 va = *reinterpret_cast<const uint4*>(ar + t0 + 4 * q);
        uint4 vb = *reinterpret_cast<const uint4*>(br + t0 + 4 * q);
        pa[4 * q + 0] = Rg::from_bits(va.x);
        pa[4 * q + 1] = Rg::from_bits(va.y);
        pa[4 * q + 2] = Rg::from_bits(va.z);
        pa[4 * q + 3] = Rg::from_bits(va.w);
        pu[4 * q + 0] = Rg::from_bits(vb.x);
        pu[4 * q + 1] = Rg::from_bits(vb.y);
        pu[4 * q + 2] = Rg::from_bits(vb.z);
        pu[4 * q + 3] = Rg::from_bits(vb.w);
        if (xr) {
          const uint4 vx = *reinterpret_cast<const uint4*>(xr + t0 + 4 * q);
          pu[4 * q + 0] = Rg::mul(pu[4 * q + 0], Rg::from_bits(vx.x));
          pu[4 * q + 1] = Rg::mul(pu[4 * q + 1], Rg::from_bits(vx.y));
          pu[4 * q + 2] = Rg::mul(pu[4 * q + 2], Rg::from_bits(vx.z));
          pu[4 * q + 3] = Rg::mul(pu[4 * q + 3], Rg::from_bits(vx.w));
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const bool ok = t0 + k < L;
        pa[k] = ok ? ar[t0 + k] : Rg::one();
        pu[k] = ok ? (xr ? Rg::mul(br[t0 + k], xr[t0 + k]) : br[t0 + k]) : Rg::zero();
      }
    }
#pragma unroll
    for (int k = 1; k < K; ++k) absorb_earlier(pa[k], pu[k], pa[k - 1], pu[k - 1]);

    // 2. wavefront scan of the lane totals
    T wA = pa[K - 1], wU = pu[K - 1];
    wave_inclusive_scan(wA, wU);
    if (lane == 63) {
      sA[wave] = wA;
      sU[wave] = wU;
    }
    wave_shift_exclusive(wA, wU);
    __syncthreads();

    // 3. fold the totals of earlier wavefronts; chunk total
    T pA = Rg::one(), pU = Rg::zero();  // prefix of waves before this one
    T cA = Rg::one(), cU = Rg::zero();  // running chunk total
#pragma unroll
    for (int w = 0; w < AS_WAVES; ++w) {
      if (w == wave) {
        pA = cA;
        pU = cU;
      }
      T nA = sA[w], nU = sU[w];
      absorb_earlier(nA, nU, cA, cU);
      cA = nA;
      cU = nU;
    }
    absorb_earlier(wA, wU, pA, pU);  // lane's exclusive prefix within the chunk

    // 4. carry into the chunk
    T hin;
    if (c == 0) {
      hin = io.h0 ? io.h0[row] : Rg::zero();
      if (nchunks > 1 && tid == 0)
        carry_put(carry + (row * nchunks) * 3, st_inc, Rg::bits(Rg::mad(cA, hin, cU)));
    } else {
      if (tid == 0) {
        unsigned long long* base = carry + (row * nchunks) * 3;
        if (c + 1 < nchunks) {
          carry_put(base + c * 3 + 1, st_agg, Rg::bits(cA));
          carry_put(base + c * 3 + 2, st_agg, Rg::bits(cU));
        }
        T accA = Rg::one(), accU = Rg::zero();
        int64_t p = c - 1;
        for (;;) {
          const unsigned long long wi = carry_get(base + p * 3);
          if ((uint32_t)(wi >> 32) == st_inc) {
            hin = Rg::mad(accA, Rg::from_bits((uint32_t)wi), accU);
            break;
          }
          const unsigned long long wa = carry_get(base + p * 3 + 1);
          const unsigned long long wu = carry_get(base + p * 3 + 2);
          if ((uint32_t)(wa >> 32) == st_agg && (uint32_t)(wu >> 32) == st_agg) {
            absorb_earlier(accA, accU, Rg::from_bits((uint32_t)wa), Rg::from_bits((uint32_t)wu));
            --p;  // chunk 0 always publishes an inclusive state, so p stays >= 0
            continue;
          }
          __builtin_amdgcn_s_sleep(1);
        }
        if (c + 1 < nchunks) carry_put(base + c * 3, st_inc, Rg::bits(Rg::mad(cA, hin, cU)));
        s_hin = hin;
      }
      __syncthreads();
      hin = s_hin;
    }

    // 5. rebuild the states and store
    const T hs = Rg::mad(wA, hin, wU);
    if (VEC && !IO && t0 + K <= L) {
#pragma unroll
      for (int q = 0; q < K / 4; ++q) {
        uint4 o;
        o.x = Rg::bits(Rg::mad(pa[4 * q + 0], hs, pu[4 * q + 0]));
        o.y = Rg::bits(Rg::mad(pa[4 * q + 1], hs, pu[4 * q + 1]));
        o.z = Rg::bits(Rg::mad(pa[4 * q + 2], hs, pu[4 * q + 2]));
        o.w = Rg::bits(Rg::mad(pa[4 * q + 3], hs, pu[4 * q + 3]));
        *reinterpret_cast<uint4*>(hr + t0 + 4 * q) = o;
      }
    } else if (VEC && t0 + K <= L) {
#pragma unroll
      for (int q = 0; q < K / 4; ++q) {
        uint4 vc = make_uint4(0u, 0u, 0u, 0u);
        if (cr) vc = *reinterpret_cast<const uint4*>(cr + t0 + 4 * q);
        const uint32_t cb[4] = {vc.x, vc.y, vc.z, vc.w};
        T v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int k = 4 * q + e;
          v[e] = Rg::mad(pa[k], hs, pu[k]);
          if (io.h_last && t0 + k == L - 1) io.h_last[row] = v[e];
          if (cr) v[e] = Rg::mul(Rg::from_bits(cb[e]), v[e]);
        }
        *reinterpret_cast<uint4*>(hr + t0 + 4 * q) =
            make_uint4(Rg::bits(v[0]), Rg::bits(v[1]), Rg::bits(v[2]), Rg::bits(v[3]));
      }
    } else {
#pragma unroll
      for (int k = 0; k < K; ++k)
        if (t0 + k < L) hr[t0 + k] = out_elem<IO>(io, cr, Rg::mad(pa[k], hs, pu[k]), t0 + k, L, row);
    }
    if (nchunks <= 1) {
      id += gridDim.x;
    }
    __syncthreads();  // LDS is reused by the next chunk
  }
}

constexpr int AS_K = 8;

// Row-serial variant for many rows: one workgroup owns one (b,d) row and walks
// it chunk by chunk, keeping the carry in registers (every lane folds the four
// wavefront totals, so every lane knows the state leaving the chunk).  No
// cross-workgroup traffic, no scratch; the next chunk's loads are in flight
// while the current one is scanned.  Used when the rows alone fill the GPU.
template <typename T, int K, bool VEC>
struct ChunkRegs {
  T a[K], u[K];
};

// In the IO variant the c of the chunk is prefetched with it.
template <typename T, int K>
struct ChunkC {
  T c[K];
};

// Branch-free loads (clamped addresses, identity pairs past the end): the
// prefetch then never forces a wait, and the register buffer is never written
// from two control-flow paths.  Requires L >= 4; with VEC, L is a multiple of
// 4, so every 4-element piece is wholly inside or wholly outside the row.
// IO: u = b * x (x row `xr`, or 1 when NULL), and c (row `cr`, or 1) into `rc`.
template <bool IO, typename T, int K, bool VEC>
__device__ __forceinline__ void load_chunk(ChunkRegs<T, K, VEC>& r, ChunkC<T, K>& rc,
                                           const T* __restrict__ ar, const T* __restrict__ br,
                                           const T* __restrict__ xr, const T* __restrict__ cr,
                                           int64_t t0, int64_t L) {
  using Rg = Ring<T>;
  if (VEC) {
#pragma unroll
    for (int q = 0; q < K / 4; ++q) {
      const int64_t tq = t0 + 4 * q;
      const bool ok = tq < L;
      const int64_t at = ok ? tq : L - 4;
      const uint4 va = *reinterpret_cast<const uint4*>(ar + at);
      uint4 vb = *reinterpret_cast<const uint4*>(br + at);
      if (IO && xr) {
        const uint4 vx = *reinterpret_cast<const uint4*>(xr + at);
        vb = make_uint4(Rg::bits(Rg::mul(Rg::from_bits(vb.x), Rg::from_bits(vx.x))),
                        Rg::bits(Rg::mul(Rg::from_bits(vb.y), Rg::from_bits(vx.y))),
                        Rg::bits(Rg::mul(Rg::from_bits(vb.z), Rg::from_bits(vx.z))),
                        Rg::bits(Rg::mul(Rg::from_bits(vb.w), Rg::from_bits(vx.w))));
      }
      if (IO && cr) {
        const uint4 vc = *reinterpret_cast<const uint4*>(cr + at);
        rc.c[4 * q + 0] = Rg::from_bits(vc.x);
        rc.c[4 * q + 1] = Rg::from_bits(vc.y);
        rc.c[4 * q + 2] = Rg::from_bits(vc.z);
        rc.c[4 * q + 3] = Rg::from_bits(vc.w);
      }
      r.a[4 * q + 0] = ok ? Rg::from_bits(va.x) : Rg::one();
      r.a[4 * q + 1] = ok ? Rg::from_bits(va.y) : Rg::one();
      r.a[4 * q + 2] = ok ? Rg::from_bits(va.z) : Rg::one();
      r.a[4 * q + 3] = ok ? Rg::from_bits(va.w) : Rg::one();
      r.u[4 * q + 0] = ok ? Rg::from_bits(vb.x) : Rg::zero();
      r.u[4 * q + 1] = ok ? Rg::from_bits(vb.y) : Rg::zero();
      r.u[4 * q + 2] = ok ? Rg::from_bits(vb.z) : Rg::zero();
      r.u[4 * q + 3] = ok ? Rg::from_bits(vb.w) : Rg::zero();
    }
  } else {
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const bool ok = t0 + k < L;
      const int64_t at = ok ? t0 + k : L - 1;
      const T va = ar[at];
      T vb = br[at];
      if (IO && xr) vb = Rg::mul(vb, xr[at]);
      if (IO && cr) rc.c[k] = cr[at];
      r.a[k] = ok ? va : Rg::one();
      r.u[k] = ok ? vb : Rg::zero();
    }
  }
}

template <typename T, int K, bool VEC, bool IO>
__global__ __launch_bounds__(AS_THREADS) void affine_rows_kernel(const AffIO<T> io, int64_t R,
                                                                 int64_t L) {
  constexpr int64_t CH = (int64_t)AS_THREADS * K;
  using Rg = Ring<T>;
  __shared__ T sA[2][AS_WAVES], sU[2][AS_WAVES];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t nch = (L + CH - 1) / CH;

  for (int64_t row = blockIdx.x; row < R; row += gridDim.x) {
    const T* __restrict__ ar = io.a + row * L;
    const T* __restrict__ br = io.b + row * L;
    const T* __restrict__ xr = (IO && io.x) ? io.x + row * L : nullptr;
    const T* __restrict__ cr = (IO && io.c) ? io.c + row * L : nullptr;
    T* __restrict__ hr = io.y + row * L;
    T carry = io.h0 ? io.h0[row] : Rg::zero();
    ChunkRegs<T, K, VEC> cur, nxt;
    ChunkC<T, K> ccur, cnxt;
    load_chunk<IO>(cur, ccur, ar, br, xr, cr, (int64_t)tid * K, L);
    for (int64_t c = 0; c < nch; ++c) {
      const int64_t t0 = c * CH + (int64_t)tid * K;
      if (c + 1 < nch)  // in flight during the scan
        load_chunk<IO>(nxt, cnxt, ar, br, xr, cr, t0 + CH, L);
      T pa[K], pu[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        pa[k] = cur.a[k];
        pu[k] = cur.u[k];
      }
#pragma unroll
      for (int k = 1; k < K; ++k) absorb_earlier(pa[k], pu[k], pa[k - 1], pu[k - 1]);
      T wA = pa[K - 1], wU = pu[K - 1];
      wave_inclusive_scan(wA, wU);
      const int buf = (int)(c & 1);
      if (lane == 63) {
        sA[buf][wave] = wA;
        sU[buf][wave] = wU;
      }
      wave_shift_exclusive(wA, wU);
      __syncthreads();  // one barrier per chunk: the totals alternate between two buffers
      T pA = Rg::one(), pU = Rg::zero(), cA = Rg::one(), cU = Rg::zero();
#pragma unroll
      for (int w = 0; w < AS_WAVES; ++w) {
        if (w == wave) {
          pA = cA;
          pU = cU;
        }
        T nA = sA[buf][w], nU = sU[buf][w];
        absorb_earlier(nA, nU, cA, cU);
        cA = nA;
        cU = nU;
      }
      absorb_earlier(wA, wU, pA, pU);
      const T hs = Rg::mad(wA, carry, wU);
      // y = c * h (IO with c), else h; the state of step L-1 also goes to h_last
      auto outv = [&](int k) {
        const T hv = Rg::mad(pa[k], hs, pu[k]);
        if constexpr (IO) {
          if (io.h_last && t0 + k == L - 1) io.h_last[row] = hv;
          if (cr) return Rg::mul(ccur.c[k], hv);
        }
        return hv;
      };
      if (VEC) {
#pragma unroll
        for (int q = 0; q < K / 4; ++q) {
          uint4 o;
          o.x = Rg::bits(outv(4 * q + 0));
          o.y = Rg::bits(outv(4 * q + 1));
          o.z = Rg::bits(outv(4 * q + 2));
          o.w = Rg::bits(outv(4 * q + 3));
          if (t0 + 4 * q < L) *reinterpret_cast<uint4*>(hr + t0 + 4 * q) = o;
        }
      } else {
#pragma unroll
        for (int k = 0; k < K; ++k)
          if (t0 + k < L) hr[t0 + k] = outv(k);
      }
      carry = Rg::mad(cA, carry, cU);
      cur = nxt;
      if constexpr (IO) ccur = cnxt;
    }
    __syncthreads();  // the totals buffers are reused by the next row
  }
}

std::mutex scratch_addr_mu;
unsigned long long* scratch_addr[64] = {};  // per device, guarded by scratch_addr_mu

// The device address of `scratch` on device `dev` (the current device).
int static_scratch(int dev, unsigned long long** out) {
  *out = nullptr;
  if (dev < 0 || dev >= 64)
    return fail(SW_ERR_UNSUPPORTED, "device %d: the static scratch table holds 64 devices", dev);
  std::lock_guard<std::mutex> g(scratch_addr_mu);
  if (!scratch_addr[dev]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(SW_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                  hipGetErrorString(e));
    }
    scratch_addr[dev] = static_cast<unsigned long long*>(p);
  }
  *out = scratch_addr[dev];
  return SW_OK;
}

// `fixed`: take the look-back scratch from the static array instead of the
// per-stream allocation, clearing the ticket and this call's carry words with
// a fill kernel first (so every call starts from epoch 1 and ticket 0).
template <typename T, bool IO>
int launch_affine(const AffIO<T>& io, int64_t R, int64_t L, bool vec, bool fixed = false) {
  hipStream_t s = current_stream();
  constexpr int64_t CH = (int64_t)AS_THREADS * AS_K;
  int cus = 0;
  int st0 = device_cus(&cus);
  if (st0 != SW_OK) return st0;
  if (L > CH && R >= 8 * (int64_t)cus) {
    // enough rows to fill the machine: one workgroup per row, carries stay on chip
    const int64_t grid = R < ((int64_t)1 << 30) ? R : ((int64_t)1 << 30);
    auto kern = vec ? affine_rows_kernel<T, AS_K, true, IO> : affine_rows_kernel<T, AS_K, false, IO>;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(AS_THREADS), 0, s, io, R, L);
    return check_launch("affine_rows_kernel");
  }
  const int64_t nchunks = (L + CH - 1) / CH;
  const int64_t total = R * nchunks;
  const int64_t grid = total < 65536 ? total : 65536;
  auto kern = vec ? affine_scan_kernel<T, AS_K, true, IO> : affine_scan_kernel<T, AS_K, false, IO>;
  if (fixed) {
    unsigned long long* base = nullptr;
    if (nchunks > 1) {
      if (total > (int64_t)SW_NOALLOC_MAX_CHUNKS)
        return fail(SW_ERR_UNSUPPORTED,
                    "%lld look-back chunks of %lld steps exceed the %d the static scratch holds",
                    (long long)total, (long long)CH, (int)SW_NOALLOC_MAX_CHUNKS);
      int cur = 0;
      hipError_t e = hipGetDevice(&cur);
      if (e != hipSuccess) return fail(SW_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
      int st = static_scratch(cur, &base);
      if (st != SW_OK) return st;
      // 64 words of ticket area, then 2 words per 64-bit carry word
      st = zero_words(reinterpret_cast<uint32_t*>(base), (size_t)(64 + 6 * total), s);
      if (st != SW_OK) return st;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(AS_THREADS), 0, s, io, R, L, nchunks,
                       total, base ? base + 32 : nullptr, reinterpret_cast<uint32_t*>(base), 0u,
                       1u);
    return check_launch("affine_scan_kernel");
  }
  ScratchSession ss;
  if (nchunks > 1) {
    if (total >= ((int64_t)1 << 31))
      return fail(SW_ERR_UNSUPPORTED, "%lld chunks exceed the ticket range", (long long)total);
    // 3 carry words per chunk; every workgroup takes one ticket past the end
    int st = ss.reserve((size_t)total * 3, (uint32_t)(total + grid), s);
    if (st != SW_OK) return st;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(AS_THREADS), 0, s, io, R, L, nchunks, total,
                     ss.carry, ss.ticket, ss.ticket_base, ss.epoch);
  int st = check_launch("affine_scan_kernel");
  if (st != SW_OK) ss.invalidate();
  return st;
}

}  // namespace

int affine_scan_f32(const float* a, const float* bx, const float* h0, float* h, int64_t R,
                    int64_t L, bool vec) {
  return launch_affine<float, false>(AffIO<float>{a, bx, nullptr, nullptr, h0, h, nullptr}, R, L,
                                     vec);
}

int affine_scan_f32_noalloc(const float* a, const float* bx, const float* h0, float* h,
                            int64_t R, int64_t L, bool vec) {
  return launch_affine<float, false>(AffIO<float>{a, bx, nullptr, nullptr, h0, h, nullptr}, R, L,
                                     vec, true);
}

int affine_scan_u32(const uint32_t* a, const uint32_t* bx, const uint32_t* h0, uint32_t* h,
                    int64_t R, int64_t L, bool vec) {
  return launch_affine<uint32_t, false>(
      AffIO<uint32_t>{a, bx, nullptr, nullptr, h0, h, nullptr}, R, L, vec);
}

int affine_scan_io_f32(const float* a, const float* b, const float* x, const float* c,
                       const float* h0, float* y, float* h_last, int64_t R, int64_t L, bool vec) {
  return launch_affine<float, true>(AffIO<float>{a, b, x, c, h0, y, h_last}, R, L, vec);
}

int affine_scan_io_u32(const uint32_t* a, const uint32_t* b, const uint32_t* x, const uint32_t* c,
                       const uint32_t* h0, uint32_t* y, uint32_t* h_last, int64_t R, int64_t L,
                       bool vec) {
  return launch_affine<uint32_t, true>(AffIO<uint32_t>{a, b, x, c, h0, y, h_last}, R, L, vec);
}

}  // namespace sw
