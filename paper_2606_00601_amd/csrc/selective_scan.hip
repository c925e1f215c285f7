// selective_scan.hip -- fused selective scan, forward, on gfx950.
//
// The Mamba-style instance of the affine recurrence (Sec. 1, Sec. 3.1):
//   a_{t,n} = exp(delta_t A_n),  u_{t,n} = delta_t B_{t,n} x_t,
//   h_{t,n} = a_{t,n} h_{t-1,n} + u_{t,n}                       Eq. (3)
//   y_t     = sum_n C_{t,n} h_{t,n} + Dskip x_t
// computed as a sequential traversal over t of the independent (b,d,n)
// recurrences, which reconstructs the same states as any associative
// evaluation of Eq. (6)-(7) (Sec. 3.2).
//
// Work per (b,d,t,n) is one exp2 plus four fp32 VALU operations against about
// half a byte of HBM traffic, so the kernel is bound by the VALU issue rate,
// not by HBM.  The layout is chosen to spend as few VALU slots per element
// as possible:
//   * G = 8 lanes share one (b,d) row, each lane owning NPL = N/8 states, so
//     a workgroup of 256 lanes covers 32 rows and all N states;
//   * per tile of T steps the workgroup stages delta, delta*x and Dskip*x
//     (fp32, widened once from bf16 when needed) and B_t, C_t in LDS; lanes
//     read them with LDS broadcast loads;
//   * the per-lane loop does exp2(delta * A*log2e), delta*x*B, the state
//     FMA and the C FMA into a per-lane partial of y_t;
//   * the G partials of each y_t meet in LDS and are summed by the lane that
//     stores y, together with Dskip*x (coalesced 16-byte stores along t);
//   * the next tile's global loads are issued before the current tile is
//     computed, so HBM latency hides behind the VALU work.
#include "sw_internal.h"

namespace sw {
namespace {

constexpr int SS_THREADS = 256;
constexpr int SS_G = 8;                     // lanes per (b,d) row
constexpr int SS_RPB = SS_THREADS / SS_G;   // rows per workgroup
constexpr int SS_T = 32;                    // time steps per tile
constexpr float LOG2E = 1.4426950408889634f;

template <typename IN>
struct In;

template <>
struct In<float> {
  static __device__ __forceinline__ float get(const float* p, int64_t i) { return p[i]; }
  // four consecutive values from a 16-byte aligned address
  static __device__ __forceinline__ void get4(const float* p, int64_t i, float* v) {
    float4 q = *reinterpret_cast<const float4*>(p + i);
    v[0] = q.x;
    v[1] = q.y;
    v[2] = q.z;
    v[3] = q.w;
  }
};

template <>
struct In<uint16_t> {
  static __device__ __forceinline__ float get(const uint16_t* p, int64_t i) {
    return bf16_one(p[i]);
  }
  // four consecutive bf16 from an 8-byte aligned address
  static __device__ __forceinline__ void get4(const uint16_t* p, int64_t i, float* v) {
    uint2 q = *reinterpret_cast<const uint2*>(p + i);
    v[0] = bf16_lo(q.x);
    v[1] = bf16_hi(q.x);
    v[2] = bf16_lo(q.y);
    v[3] = bf16_hi(q.y);
  }
};

// Registers holding one tile's worth of global inputs for one thread.
template <int NPL>
struct TileRegs {
  float dl[4], xv[4];
  float bv[NPL], cv[NPL];
};

template <typename IN, int NPL, bool VEC>
__device__ __forceinline__ void load_tile(TileRegs<NPL>& r, const IN* __restrict__ x,
                                          const IN* __restrict__ delta,
                                          const IN* __restrict__ Bm, const IN* __restrict__ Cm,
                                          int64_t b, int64_t d0, int64_t D, int N, int64_t L,
                                          int64_t t0, int tid) {
  // delta and x: row tid/8, steps (tid%8)*4 .. +3 of the tile
  const int rr = tid / 8;
  const int tq = (tid % 8) * 4;
  const int64_t d = d0 + rr;
  const int64_t t = t0 + tq;
  if (d < D) {
    const int64_t base = (b * D + d) * L + t;
    if (VEC && t + 4 <= L) {
      In<IN>::get4(delta, base, r.dl);
      In<IN>::get4(x, base, r.xv);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const bool ok = t + k < L;
        r.dl[k] = ok ? In<IN>::get(delta, base + k) : 0.0f;
        r.xv[k] = ok ? In<IN>::get(x, base + k) : 0.0f;
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      r.dl[k] = 0.0f;
      r.xv[k] = 0.0f;
    }
  }
  // B and C: element e = tid + 256*m of the (T, G*NPL) tile
  constexpr int NPAD = SS_G * NPL;
#pragma unroll
  for (int m = 0; m < NPL; ++m) {
    const int e = tid + SS_THREADS * m;
    const int tt = e / NPAD;
    const int n = e % NPAD;
    const int64_t tg = t0 + tt;
    const bool ok = n < N && tg < L;
    const int64_t off = (b * L + tg) * N + n;
    r.bv[m] = ok ? In<IN>::get(Bm, off) : 0.0f;
    r.cv[m] = ok ? In<IN>::get(Cm, off) : 0.0f;
  }
}

template <typename IN, int NPL, bool VEC>
__global__ __launch_bounds__(SS_THREADS) void selective_fwd_kernel(
    const IN* __restrict__ x, const IN* __restrict__ delta, const float* __restrict__ A,
    const IN* __restrict__ Bm, const IN* __restrict__ Cm, const float* __restrict__ Dskip,
    float* __restrict__ y, float* __restrict__ h_last, int64_t D, int N, int64_t L) {
  constexpr int NPAD = SS_G * NPL;
  constexpr int T = SS_T;
  __shared__ float sDl[SS_RPB][T + 1];
  __shared__ float sDx[SS_RPB][T + 1];
  __shared__ float sYd[SS_RPB][T + 1];
  __shared__ __align__(16) float sBC[T][SS_G][2 * NPL];
  __shared__ float sP[SS_RPB][SS_G][T + 1];  // +1: lanes of 4 rows x 8 groups hit 32 banks

  const int tid = threadIdx.x;
  const int64_t ndb = (D + SS_RPB - 1) / SS_RPB;  // row blocks per batch
  const int64_t b = (int64_t)blockIdx.x / ndb;
  const int64_t d0 = ((int64_t)blockIdx.x - b * ndb) * SS_RPB;

  // compute-phase identity of this lane: row r, lane-group g, states g*NPL+j
  const int r = tid / SS_G;
  const int g = tid % SS_G;
  const int64_t d = d0 + r;
  float Al[NPL], hs[NPL];
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int n = g * NPL + j;
    Al[j] = (d < D && n < N) ? A[d * N + n] * LOG2E : 0.0f;
    hs[j] = 0.0f;
  }
  // staging identity: row tid/8, steps (tid%8)*4..+3
  const int rr = tid / 8;
  const int tq = (tid % 8) * 4;
  const float dsk = (Dskip && d0 + rr < D) ? Dskip[d0 + rr] : 0.0f;

  TileRegs<NPL> cur;
  load_tile<IN, NPL, VEC>(cur, x, delta, Bm, Cm, b, d0, D, N, L, 0, tid);

  for (int64_t t0 = 0; t0 < L; t0 += T) {
    // stage the tile held in registers
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      sDl[rr][tq + k] = cur.dl[k];
      sDx[rr][tq + k] = cur.dl[k] * cur.xv[k];
      sYd[rr][tq + k] = dsk * cur.xv[k];
    }
#pragma unroll
    for (int m = 0; m < NPL; ++m) {
      const int e = tid + SS_THREADS * m;
      const int tt = e / NPAD;
      const int n = e % NPAD;
      sBC[tt][n / NPL][n % NPL] = cur.bv[m];
      sBC[tt][n / NPL][NPL + n % NPL] = cur.cv[m];
    }
    __syncthreads();
    // prefetch the next tile while this one is computed
    if (t0 + T < L) load_tile<IN, NPL, VEC>(cur, x, delta, Bm, Cm, b, d0, D, N, L, t0 + T, tid);

    // recurrence over the tile
#pragma unroll 4
    for (int t = 0; t < T; ++t) {
      const float dl = sDl[r][t];
      const float dx = sDx[r][t];
      float bc[2 * NPL];
#pragma unroll
      for (int j = 0; j < 2 * NPL; ++j) bc[j] = sBC[t][g][j];
      float p = 0.0f;
#pragma unroll
      for (int j = 0; j < NPL; ++j) {
        const float a = __builtin_amdgcn_exp2f(dl * Al[j]);
        hs[j] = __builtin_fmaf(a, hs[j], dx * bc[j]);
        p = __builtin_fmaf(bc[NPL + j], hs[j], p);
      }
      sP[r][g][t] = p;
    }
    __syncthreads();

    // y = Dskip*x + sum of the G partials, stored along t
    {
      const int64_t dd = d0 + rr;
      const int64_t tt = t0 + tq;
      float yv[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        float s = sYd[rr][tq + k];
#pragma unroll
        for (int gg = 0; gg < SS_G; ++gg) s += sP[rr][gg][tq + k];
        yv[k] = s;
      }
      if (dd < D) {
        float* yr = y + (b * D + dd) * L;
        if (VEC && tt + 4 <= L) {
          *reinterpret_cast<float4*>(yr + tt) = make_float4(yv[0], yv[1], yv[2], yv[3]);
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (tt + k < L) yr[tt + k] = yv[k];
        }
      }
    }
    __syncthreads();
  }

  if (h_last && d < D) {
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int n = g * NPL + j;
      if (n < N) h_last[(b * D + d) * N + n] = hs[j];
    }
  }
}

template <typename IN, int NPL>
int launch_npl(const IN* x, const IN* delta, const float* A, const IN* Bm, const IN* Cm,
               const float* Dskip, float* y, float* h_last, int64_t B, int64_t D, int N,
               int64_t L, bool vec, hipStream_t s) {
  dim3 grid((unsigned)(B * ((D + SS_RPB - 1) / SS_RPB)));
  if (vec)
    hipLaunchKernelGGL((selective_fwd_kernel<IN, NPL, true>), grid, dim3(SS_THREADS), 0, s, x,
                       delta, A, Bm, Cm, Dskip, y, h_last, D, N, L);
  else
    hipLaunchKernelGGL((selective_fwd_kernel<IN, NPL, false>), grid, dim3(SS_THREADS), 0, s, x,
                       delta, A, Bm, Cm, Dskip, y, h_last, D, N, L);
  return check_launch("selective_fwd_kernel");
}

template <typename IN>
int launch_selective(const IN* x, const IN* delta, const float* A, const IN* Bm, const IN* Cm,
                     const float* Dskip, float* y, float* h_last, int64_t B, int64_t D,
                     int64_t N, int64_t L, bool vec) {
  hipStream_t s = current_stream();
  const int n = (int)N;
  if (n <= 8) return launch_npl<IN, 1>(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, n, L, vec, s);
  if (n <= 16) return launch_npl<IN, 2>(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, n, L, vec, s);
  if (n <= 32) return launch_npl<IN, 4>(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, n, L, vec, s);
  return launch_npl<IN, 8>(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, n, L, vec, s);
}

}  // namespace

int selective_fwd_f32(const float* x, const float* delta, const float* A, const float* Bm,
                      const float* Cm, const float* Dskip, float* y, float* h_last, int64_t B,
                      int64_t D, int64_t N, int64_t L, bool vec) {
  return launch_selective<float>(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, N, L, vec);
}

int selective_fwd_bf16(const uint16_t* x, const uint16_t* delta, const float* A,
                       const uint16_t* Bm, const uint16_t* Cm, const float* Dskip, float* y,
                       float* h_last, int64_t B, int64_t D, int64_t N, int64_t L, bool vec) {
  return launch_selective<uint16_t>(x, delta, A, Bm, Cm, Dskip, y, h_last, B, D, N, L, vec);
}

}  // namespace sw
