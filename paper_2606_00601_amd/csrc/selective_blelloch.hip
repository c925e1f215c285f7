// selective_blelloch.hip -- the fused selective scan with the paper's schedule
// (Sec. 3.3): every (b,d,n) recurrence scanned over t by a Blelloch tree of
// affine pairs in LDS.  Kept as the reference point of the schedule ablation
// against selective_scan16.hip / selective_scan.hip, which walk t
// sequentially per lane.
//
// One workgroup (256 lanes) owns one (b,d) row and walks it in chunks of 2048
// steps; lane i holds steps 8i .. 8i+7 of the chunk.  For each state n in
// turn:
//   1. the lane forms its pairs (a_t, u_t) = (exp(delta_t A_n),
//      delta_t B_{t,n} x_t) and writes them to LDS;
//   2. upsweep (11 levels), root set to the identity, downsweep (11 levels),
//      as in affine_blelloch.hip, leaving the exclusive prefix compositions;
//   3. affine-prefix reconstruction h_t = a_t (E_A h_in + E_U) + u_t, with
//      h_in the state n carried from the previous chunk, and y_t += C_{t,n} h_t
//      in the lane's registers; the carry becomes A_tot h_in + U_tot.
// After the 16 states, y_t + Dskip x_t is stored.  The same row's B and C
// values come from L2 (they are shared by all rows of the batch).
#include "selective_common.h"

namespace sw {
namespace {

constexpr int SB_THREADS = 256;
constexpr int SB_K = 8;                    // steps per lane
constexpr int SB_C = SB_THREADS * SB_K;    // steps per chunk (2048)
constexpr int SB_LEVELS = 11;
constexpr int SB_PAD = SB_C + SB_C / 32;
constexpr int SB_MAXN = 64;
constexpr float SB_LOG2E = 1.4426950408889634f;

__device__ __forceinline__ int sb_pos(int i) { return i + (i >> 5); }

template <typename IN>
__device__ __forceinline__ float sb_ld(const IN* __restrict__ p, int64_t i) {
  if constexpr (sizeof(IN) == 4)
    return p[i];
  else
    return bf16_one(p[i]);
}

template <typename IN>
__global__ __launch_bounds__(SB_THREADS) void selective_blelloch_kernel(
    const IN* __restrict__ x, const IN* __restrict__ delta, const float* __restrict__ A,
    const IN* __restrict__ Bm, const IN* __restrict__ Cm, const float* __restrict__ Dskip,
    float* __restrict__ y, float* __restrict__ h_last, int64_t R, int64_t D, int N, int64_t L) {
  __shared__ float sA[SB_PAD], sU[SB_PAD];
  __shared__ float s_carry[SB_MAXN];
  const int tid = threadIdx.x;
  const int64_t nch = (L + SB_C - 1) / SB_C;

  for (int64_t row = blockIdx.x; row < R; row += gridDim.x) {
    const int64_t b = row / D, d = row - b * D;
    const IN* __restrict__ xr = x + row * L;
    const IN* __restrict__ dr = delta + row * L;
    const IN* __restrict__ Bb = Bm + b * L * N;
    const IN* __restrict__ Cb = Cm + b * L * N;
    if (tid < N) s_carry[tid] = 0.0f;
    __syncthreads();
    for (int64_t c = 0; c < nch; ++c) {
      const int64_t t0 = c * SB_C + (int64_t)tid * SB_K;
      float dl[SB_K], xv[SB_K], yv[SB_K];
#pragma unroll
      for (int k = 0; k < SB_K; ++k) {
        const bool ok = t0 + k < L;
        const int64_t t = ok ? t0 + k : L - 1;
        dl[k] = ok ? sb_ld<IN>(dr, t) : 0.0f;  // identity steps past L: a = 1, u = 0
        xv[k] = ok ? sb_ld<IN>(xr, t) : 0.0f;
        yv[k] = 0.0f;
      }
      for (int n = 0; n < N; ++n) {
        const float Al = A[d * N + n] * SB_LOG2E;
        float av[SB_K], uv[SB_K];
#pragma unroll
        for (int k = 0; k < SB_K; ++k) {
          const int64_t t = t0 + k < L ? t0 + k : L - 1;
          av[k] = __builtin_amdgcn_exp2f(dl[k] * Al);
          uv[k] = dl[k] * xv[k] * sb_ld<IN>(Bb, t * N + n);
          sA[sb_pos(tid * SB_K + k)] = av[k];
          sU[sb_pos(tid * SB_K + k)] = uv[k];
        }
        __syncthreads();
        // upsweep
#pragma unroll
        for (int lv = 0; lv < SB_LEVELS; ++lv) {
          const int s = 2 << lv, nodes = SB_C >> (lv + 1);
          for (int j = tid; j < nodes; j += SB_THREADS) {
            const int ri = sb_pos((j + 1) * s - 1), li = sb_pos((j + 1) * s - 1 - s / 2);
            float Ar = sA[ri], Ur = sU[ri];
            absorb_earlier(Ar, Ur, sA[li], sU[li]);
            sA[ri] = Ar;
            sU[ri] = Ur;
          }
          __syncthreads();
        }
        const float totA = sA[sb_pos(SB_C - 1)], totU = sU[sb_pos(SB_C - 1)];
        const float hin = s_carry[n];
        __syncthreads();
        if (tid == 0) {
          sA[sb_pos(SB_C - 1)] = 1.0f;
          sU[sb_pos(SB_C - 1)] = 0.0f;
          s_carry[n] = __builtin_fmaf(totA, hin, totU);
        }
        __syncthreads();
        // downsweep
#pragma unroll
        for (int lv = SB_LEVELS - 1; lv >= 0; --lv) {
          const int s = 2 << lv, nodes = SB_C >> (lv + 1);
          for (int j = tid; j < nodes; j += SB_THREADS) {
            const int ri = sb_pos((j + 1) * s - 1), li = sb_pos((j + 1) * s - 1 - s / 2);
            const float lA = sA[li], lU = sU[li];
            const float pA = sA[ri], pU = sU[ri];
            sA[li] = pA;
            sU[li] = pU;
            float Ar = lA, Ur = lU;
            absorb_earlier(Ar, Ur, pA, pU);
            sA[ri] = Ar;
            sU[ri] = Ur;
          }
          __syncthreads();
        }
        // reconstruction and the C contraction
#pragma unroll
        for (int k = 0; k < SB_K; ++k) {
          const int e = sb_pos(tid * SB_K + k);
          const float hp = __builtin_fmaf(sA[e], hin, sU[e]);
          const float hv = __builtin_fmaf(av[k], hp, uv[k]);
          const int64_t t = t0 + k < L ? t0 + k : L - 1;
          yv[k] = __builtin_fmaf(sb_ld<IN>(Cb, t * N + n), hv, yv[k]);
        }
        __syncthreads();  // LDS is rewritten by the next state
      }
      const float dsk = Dskip ? Dskip[d] : 0.0f;
#pragma unroll
      for (int k = 0; k < SB_K; ++k)
        if (t0 + k < L) y[row * L + t0 + k] = __builtin_fmaf(dsk, xv[k], yv[k]);
    }
    if (h_last && tid < N) h_last[row * N + tid] = s_carry[tid];
    __syncthreads();  // s_carry is reset by the next row
  }
}

}  // namespace

int selective_blelloch_fwd(const SelArgs& a) {
  hipStream_t s = current_stream();
  const int64_t R = a.B * a.D;
  if (a.N > SB_MAXN) return fail(SW_ERR_UNSUPPORTED, "N=%lld above %d", (long long)a.N, SB_MAXN);
  if (a.z || a.delta_bias || a.h0 || a.softplus || a.y_bf16)
    return fail(SW_ERR_UNSUPPORTED, "the Blelloch schedule runs the plain form only");
  const int64_t grid = R < ((int64_t)1 << 30) ? R : ((int64_t)1 << 30);
  if (a.bf16_in)
    hipLaunchKernelGGL((selective_blelloch_kernel<uint16_t>), dim3((unsigned)grid),
                       dim3(SB_THREADS), 0, s, static_cast<const uint16_t*>(a.x),
                       static_cast<const uint16_t*>(a.delta), a.A,
                       static_cast<const uint16_t*>(a.Bm), static_cast<const uint16_t*>(a.Cm),
                       a.Dskip, static_cast<float*>(a.y), a.h_last, R, a.D, (int)a.N, a.L);
  else
    hipLaunchKernelGGL((selective_blelloch_kernel<float>), dim3((unsigned)grid), dim3(SB_THREADS),
                       0, s, static_cast<const float*>(a.x), static_cast<const float*>(a.delta),
                       a.A, static_cast<const float*>(a.Bm), static_cast<const float*>(a.Cm),
                       a.Dskip, static_cast<float*>(a.y), a.h_last, R, a.D, (int)a.N, a.L);
  note_launch("selective_blelloch_kernel: the Blelloch tree, whole rows");
  return check_launch("selective_blelloch_kernel");
}

}  // namespace sw
