// affine_blelloch.hip -- the bare affine scan with the paper's schedule: a
// Blelloch tree over the affine pairs of Eq. (6) in LDS (Sec. 3.3), kept as
// the reference point of the schedule ablation against the lane-sequential /
// DPP / look-back schedule of affine_scan.hip.
//
// One workgroup (256 lanes) owns one (b,d) row and walks it in chunks of
// 2048 steps, the carry held in registers (the hierarchical level above the
// tree).  Per chunk:
//   1. the 2048 pairs (a_t, bx_t) are loaded with 16-byte loads (the next
//      chunk's loads are issued before the tree runs) and written to LDS;
//   2. upsweep: 11 levels of the tree; at stride s the node ending at i
//      absorbs the one ending at i - s/2, (A,U)[i] <- (A,U)[i] (+) (A,U)[i-s/2]
//      (the later segment on the left, Eq. (7)); one barrier per level;
//   3. root initialisation: the root's pair is the chunk's total; it is
//      replaced by the identity (1, 0);
//   4. downsweep: 11 levels back down; the left child takes the parent's
//      prefix and the right child the left subtree's total composed after it;
//      at the end every position holds its exclusive prefix composition;
//   5. affine-prefix reconstruction: h_t = a_t (E_A h_in + E_U) + bx_t from
//      the exclusive prefix (E_A, E_U) and the chunk's incoming state h_in,
//      stored with 16-byte stores; the carry becomes A_tot h_in + U_tot.
// LDS positions are padded by one word per 32 so that the power-of-two
// strides of the tree do not all land in one bank.
#include "sw_internal.h"

namespace sw {
namespace {

constexpr int BL_THREADS = 256;
constexpr int BL_K = 8;                       // pairs per lane
constexpr int BL_C = BL_THREADS * BL_K;       // pairs per chunk (2048)
constexpr int BL_LEVELS = 11;                 // log2(BL_C)
constexpr int BL_PAD = BL_C + BL_C / 32;      // padded LDS length

__device__ __forceinline__ int bl_pos(int i) { return i + (i >> 5); }

template <typename T, bool VEC>
struct BlRegs {
  T a[BL_K], u[BL_K];
};

// Branch-free loads of the lane's BL_K pairs at t0 (clamped addresses;
// identity pairs past the end).  VEC: L is a multiple of 4 and the rows are
// 16-byte aligned.
template <typename T, bool VEC>
__device__ __forceinline__ void bl_load(BlRegs<T, VEC>& r, const T* __restrict__ ar,
                                        const T* __restrict__ br, int64_t t0, int64_t L) {
  using Rg = Ring<T>;
  if constexpr (VEC) {
#pragma unroll
    for (int q = 0; q < BL_K / 4; ++q) {
      const int64_t tq = t0 + 4 * q;
      const bool ok = tq < L;
      const int64_t at = ok ? tq : L - 4;
      const uint4 va = *reinterpret_cast<const uint4*>(ar + at);
      const uint4 vb = *reinterpret_cast<const uint4*>(br + at);
      const uint32_t aw[4] = {va.x, va.y, va.z, va.w};
      const uint32_t bw[4] = {vb.x, vb.y, vb.z, vb.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        r.a[4 * q + e] = ok ? Rg::from_bits(aw[e]) : Rg::one();
        r.u[4 * q + e] = ok ? Rg::from_bits(bw[e]) : Rg::zero();
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < BL_K; ++k) {
      const bool ok = t0 + k < L;
      const int64_t at = ok ? t0 + k : L - 1;
      const T va = ar[at], vb = br[at];
      r.a[k] = ok ? va : Rg::one();
      r.u[k] = ok ? vb : Rg::zero();
    }
  }
}

template <typename T, bool VEC>
__global__ __launch_bounds__(BL_THREADS) void affine_blelloch_kernel(
    const T* __restrict__ a, const T* __restrict__ bx, const T* __restrict__ h0,
    T* __restrict__ h, int64_t R, int64_t L) {
  using Rg = Ring<T>;
  __shared__ T sA[BL_PAD], sU[BL_PAD];
  const int tid = threadIdx.x;
  const int64_t nch = (L + BL_C - 1) / BL_C;

  for (int64_t row = blockIdx.x; row < R; row += gridDim.x) {
    const T* __restrict__ ar = a + row * L;
    const T* __restrict__ br = bx + row * L;
    T* __restrict__ hr = h + row * L;
    T carry = h0 ? h0[row] : Rg::zero();
    BlRegs<T, VEC> cur, nxt;
    bl_load(cur, ar, br, (int64_t)tid * BL_K, L);
    for (int64_t c = 0; c < nch; ++c) {
      const int64_t t0 = c * BL_C + (int64_t)tid * BL_K;
      if (c + 1 < nch) bl_load(nxt, ar, br, t0 + BL_C, L);  // in flight during the tree

      // 1. pairs into LDS
#pragma unroll
      for (int k = 0; k < BL_K; ++k) {
        sA[bl_pos(tid * BL_K + k)] = cur.a[k];
        sU[bl_pos(tid * BL_K + k)] = cur.u[k];
      }
      __syncthreads();

      // 2. upsweep
#pragma unroll
      for (int d = 0; d < BL_LEVELS; ++d) {
        const int s = 2 << d, nodes = BL_C >> (d + 1);
        for (int j = tid; j < nodes; j += BL_THREADS) {
          const int ri = bl_pos((j + 1) * s - 1), li = bl_pos((j + 1) * s - 1 - s / 2);
          T A = sA[ri], U = sU[ri];
          absorb_earlier(A, U, sA[li], sU[li]);
          sA[ri] = A;
          sU[ri] = U;
        }
        __syncthreads();
      }

      // 3. root: the chunk total, then the identity
      const T totA = sA[bl_pos(BL_C - 1)], totU = sU[bl_pos(BL_C - 1)];
      __syncthreads();
      if (tid == 0) {
        sA[bl_pos(BL_C - 1)] = Rg::one();
        sU[bl_pos(BL_C - 1)] = Rg::zero();
      }
      __syncthreads();

      // 4. downsweep
#pragma unroll
      for (int d = BL_LEVELS - 1; d >= 0; --d) {
        const int s = 2 << d, nodes = BL_C >> (d + 1);
        for (int j = tid; j < nodes; j += BL_THREADS) {
          const int ri = bl_pos((j + 1) * s - 1), li = bl_pos((j + 1) * s - 1 - s / 2);
          const T lA = sA[li], lU = sU[li];  // the left subtree's total
          const T pA = sA[ri], pU = sU[ri];  // the parent's prefix
          sA[li] = pA;
          sU[li] = pU;
          T A = lA, U = lU;
          absorb_earlier(A, U, pA, pU);
          sA[ri] = A;
          sU[ri] = U;
        }
        __syncthreads();
      }

      // 5. affine-prefix reconstruction of the inclusive states
      T hv[BL_K];
#pragma unroll
      for (int k = 0; k < BL_K; ++k) {
        const int e = bl_pos(tid * BL_K + k);
        const T hp = Rg::mad(sA[e], carry, sU[e]);  // state before step t
        hv[k] = Rg::mad(cur.a[k], hp, cur.u[k]);
      }
      if constexpr (VEC) {
#pragma unroll
        for (int q = 0; q < BL_K / 4; ++q)
          if (t0 + 4 * q < L)
            *reinterpret_cast<uint4*>(hr + t0 + 4 * q) =
                make_uint4(Rg::bits(hv[4 * q]), Rg::bits(hv[4 * q + 1]), Rg::bits(hv[4 * q + 2]),
                           Rg::bits(hv[4 * q + 3]));
      } else {
#pragma unroll
        for (int k = 0; k < BL_K; ++k)
          if (t0 + k < L) hr[t0 + k] = hv[k];
      }
      carry = Rg::mad(totA, carry, totU);
      cur = nxt;
      __syncthreads();  // LDS is rewritten by the next chunk
    }
  }
}

template <typename T>
int launch_blelloch(const T* a, const T* bx, const T* h0, T* h, int64_t R, int64_t L, bool vec) {
  hipStream_t s = current_stream();
  const int64_t grid = R < ((int64_t)1 << 30) ? R : ((int64_t)1 << 30);
  if (vec)
    hipLaunchKernelGGL((affine_blelloch_kernel<T, true>), dim3((unsigned)grid), dim3(BL_THREADS),
                       0, s, a, bx, h0, h, R, L);
  else
    hipLaunchKernelGGL((affine_blelloch_kernel<T, false>), dim3((unsigned)grid), dim3(BL_THREADS),
                       0, s, a, bx, h0, h, R, L);
  return check_launch("affine_blelloch_kernel");
}

}  // namespace

int affine_blelloch_f32(const float* a, const float* bx, const float* h0, float* h, int64_t R,
                        int64_t L, bool vec) {
  return launch_blelloch<float>(a, bx, h0, h, R, L, vec);
}

int affine_blelloch_u32(const uint32_t* a, const uint32_t* bx, const uint32_t* h0, uint32_t* h,
                        int64_t R, int64_t L, bool vec) {
  return launch_blelloch<uint32_t>(a, bx, h0, h, R, L, vec);
}

}  // namespace sw
