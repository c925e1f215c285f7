// selective_scan.hip -- fused selective scan, forward, on gfx950.
//
// The Mamba-style instance of the affine recurrence (Sec. 1, Sec. 3.1):
//   a_{t,n} = exp(delta_t A_n),  u_{t,n} = delta_t B_{t,n} x_t,
//   h_{t,n} = a_{t,n} h_{t-1,n} + u_{t,n}                       Eq. (3)
//   y_t     = sum_n C_{t,n} h_{t,n} + Dskip x_t
// evaluated as a sequential traversal over t of the independent (b,d,n)
// recurrences inside each chunk of the sequence; chunks of a row are chained
// through the exact inclusive state (the Eq. (7) composition of the chunk
// with its carry, Sec. 3.2), so the result is the sequential one.
//
// Work per (b,d,t,n) is one exp2 plus four fp32 VALU operations against about
// half a byte of HBM traffic: the kernel is bound by the VALU issue rate, not
// by HBM.  With at most two states per lane there are only about 1.5
// wavefronts of independent work per SIMD at Mamba shapes, so every
// wavefront has to keep its own SIMD issuing: the kernel is a software
// pipeline in which nothing waits on a load issued shortly before.
//   * one wavefront is one independent unit of work: 8 (b,d) rows x 8 lanes,
//     each lane owning NPL = N/8 states of its row; there is no workgroup
//     barrier anywhere;
//   * a tile is T = 32 steps.  The wavefront widens the tile's delta, x, B
//     and C (bf16 -> fp32 by a 16-bit shift, exact) and writes delta,
//     delta*x and the [B, C] slot of every state group into its own LDS, in
//     two alternating buffers: tile k+1 is staged while tile k is computed;
//   * global loads run three tiles ahead (two raw register sets), so a load
//     has two tiles of compute to arrive;
//   * the compute runs over 4-step blocks and reads the operands of the
//     block LA blocks ahead (across the tile boundary into the other
//     buffer), so LDS latency is hidden behind the current block;
//   * per step a lane does exp2(delta * A*log2e), (delta*x)*B, the state FMA
//     and the C FMA into a per-lane partial of y_t, written to LDS per block;
//   * the 8 partials of each y_t are summed, with Dskip*x, by the lane that
//     stores y (16-byte stores along t) one tile later: the reads are issued
//     before the next tile's first block and consumed after it.
// LDS instructions of one wavefront execute in order, so the cross-lane
// hand-offs through LDS need no hardware wait; compiler fences keep the
// compiler from reordering them.
// Load balance: the work is cut into tasks (8-row block, sequence chunk)
// handed out by an atomic ticket in chunk-major order to a persistent grid of
// wavefronts.  A task waits for the final state of the same rows' previous
// chunk, published as self-validating 64-bit words; that chunk holds an
// earlier ticket, so it is running or done, which guarantees forward
// progress.
#include <stdlib.h>

#include <type_traits>

#include "selective_common.h"

namespace sw {

namespace {

constexpr int SS_G = 8;            // lanes per (b,d) row
constexpr int SS_RPW = 64 / SS_G;  // rows per wavefront: 8
constexpr int SS_T = 32;           // steps per tile
constexpr int SS_TS = SS_T + 4;    // padded LDS row stride (16-byte aligned)
constexpr int SS_NB = SS_T / 4;    // 4-step blocks per tile
// B/C tile in LDS: per step t a row of 8 slots [B_{g*NPL..}, C_{g*NPL..}] of
// 2*NPL floats, rows padded by 4 floats so that the staging writes of the 64
// lanes (2 lanes per step) spread over all banks; a row itself is contiguous,
// so the compute-loop reads (8 slots of one step) are conflict-free too.
template <int NPL>
constexpr int bc_stride() { return SS_G * 2 * NPL + 4; }
constexpr float LOG2E = 1.4426950408889634f;

// One lane's share of one tile's global inputs.
template <typename IN, int NPL>
struct TileRaw {
  RawVec<IN, 4> dl, xv, zv;    // its row, steps tq .. tq+3 (zv: z, or x when not gated)
  RawVec<IN, 4 * NPL> bb, cc;  // elements lane*4*NPL .. +4*NPL-1 of the (T, 8*NPL) tile
};

// Per-task, per-lane addressing of one wavefront's inputs and outputs.
template <typename IN>
struct LanePtrs {
  const IN* dl;  // delta row of this lane's staging row, at step tq
  const IN* xv;  // x row, at step tq
  const IN* zsrc;  // z (or x) base, element path
  int64_t bc;    // element offset of this lane's B/C slice in tile 0 (vector path)
  int64_t row;   // element offset of the staging row (element path)
};

// Fill `r` with tile [t0, t0+T).  FULL (uniform): the tile lies inside the
// sequence and vector loads are allowed, so addresses need no clamping.
// Otherwise elements are gathered one by one with steps clamped to L-1 and
// padded states to N-1; the caller masks them when staging.
template <bool FULL, bool NPADDED, bool OPT, typename IN, int NPL>
__device__ __forceinline__ void load_tile(TileRaw<IN, NPL>& r, const LanePtrs<IN>& lp,
                                          const IN* __restrict__ x, const IN* __restrict__ delta,
                                          const IN* __restrict__ Bm, const IN* __restrict__ Cm,
                                          int64_t bc_off, int N, int64_t L, int64_t t0,
                                          int lane) {
  constexpr int NPAD = SS_G * NPL;
  constexpr int PER = 4 * NPL;  // B (and C) elements per lane per tile
  if constexpr (FULL) {
    r.dl.load_vec(lp.dl + t0);
    r.xv.load_vec(lp.xv + t0);
  } else {
    const int tq = (lane % 8) * 4;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t t = imin(t0 + tq + k, L - 1);
      r.dl.set(k, Elt<IN>::raw(delta, lp.row + t));
      r.xv.set(k, Elt<IN>::raw(x, lp.row + t));
      if constexpr (OPT) r.zv.set(k, Elt<IN>::raw(lp.zsrc, lp.row + t));
    }
  }
  if constexpr (FULL && !NPADDED) {
    // N == NPAD: the tile is T*N consecutive elements starting at (b, t0, 0)
    r.bb.load_vec(Bm + lp.bc + t0 * N);
    r.cc.load_vec(Cm + lp.bc + t0 * N);
  } else {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = lane * PER + i;
      const int64_t t = imin(t0 + e / NPAD, L - 1);
      const int n = (e % NPAD) < N ? (e % NPAD) : N - 1;
      r.bb.set(i, Elt<IN>::raw(Bm, bc_off + t * N + n));
      r.cc.set(i, Elt<IN>::raw(Cm, bc_off + t * N + n));
    }
  }
}

// Per-task buffer resources of the vector path: the 8 rows of x and delta
// of the row block, and B and C of its batch.  Every tile, including a
// sequence tail and the dummy tiles fetched past the end, is loaded with the
// same vector loads: lanes past the range read zeros (masked when staging).
// Equal load counts on every path let the compiler wait for exactly the
// loads of the tile being staged and leave the later tiles in flight.
struct TaskRsrc {
  __amdgpu_buffer_rsrc_t x, dl, bm, cm, z;
  int32_t row_off;  // byte offset of this lane's staging row and step tq in x / delta
  int32_t bc_off;   // byte offset of this lane's B/C slice of tile 0
};

// B and C are read as T*N consecutive elements: only for N == 8*NPL.
template <bool OPT, typename IN, int NPL>
__device__ __forceinline__ void load_tile_buf(TileRaw<IN, NPL>& r, const TaskRsrc& rs, int N,
                                              int64_t t0rel) {
  constexpr int ES = (int)sizeof(IN);
  const int32_t ts = (int32_t)t0rel * ES;
  r.dl.load_buf(rs.dl, rs.row_off + ts);
  r.xv.load_buf(rs.x, rs.row_off + ts);
  if constexpr (OPT) r.zv.load_buf(rs.z, rs.row_off + ts);
  r.bb.load_buf(rs.bm, rs.bc_off + ts * N);
  r.cc.load_buf(rs.cm, rs.bc_off + ts * N);
}

// Compiler-level ordering point for the cross-lane hand-offs through LDS.
// LDS instructions of a wavefront complete in issue order, so no hardware
// wait is needed; the wavefront-scope fences only keep the compiler from
// moving memory operations across this point.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <bool B_>
using Flag = std::integral_constant<bool, B_>;
template <int I_>
using Int = std::integral_constant<int, I_>;

// LDS of one wavefront.
template <int NPL>
struct Smem {
  float dl[2][SS_RPW * SS_TS];            // delta, two tile buffers
  float dx[2][SS_RPW * SS_TS];            // delta * x
  float bc[2][SS_T * bc_stride<NPL>()];   // per step: [B_g.., C_g..] slot of every group g
  float p[SS_RPW * SS_G * SS_TS];         // per-lane partials of y, one tile
};

// Read-ahead depth (4-step blocks) and number of rotating operand sets.
template <int NPL>
struct Pipe {
  static constexpr int LA = NPL <= 2 ? 2 : 1;
  static constexpr int NS = NPL <= 2 ? 4 : 2;
  static_assert(SS_NB % NS == 0 && LA < NS, "operand sets must rotate evenly over a tile");
};

// Operands of one 4-step block for one lane.
template <int NPL>
struct Blk {
  float dl[4], dx[4];
  float bc[4][2 * NPL];  // B of the lane's states, then C
};

template <int NPL>
__device__ __forceinline__ void read_blk(Blk<NPL>& k, const Smem<NPL>& sm, int buf, int r, int g,
                                         int bi) {
  const float4 a = *reinterpret_cast<const float4*>(&sm.dl[buf][r * SS_TS + 4 * bi]);
  const float4 b = *reinterpret_cast<const float4*>(&sm.dx[buf][r * SS_TS + 4 * bi]);
  k.dl[0] = a.x;
  k.dl[1] = a.y;
  k.dl[2] = a.z;
  k.dl[3] = a.w;
  k.dx[0] = b.x;
  k.dx[1] = b.y;
  k.dx[2] = b.z;
  k.dx[3] = b.w;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float* src = &sm.bc[buf][(4 * bi + q) * bc_stride<NPL>() + g * (2 * NPL)];
    if constexpr (NPL == 1) {
      const float2 v = *reinterpret_cast<const float2*>(src);
      k.bc[q][0] = v.x;
      k.bc[q][1] = v.y;
    } else {
#pragma unroll
      for (int j = 0; j < 2 * NPL; j += 4) {
        const float4 v = *reinterpret_cast<const float4*>(src + j);
        k.bc[q][j] = v.x;
        k.bc[q][j + 1] = v.y;
        k.bc[q][j + 2] = v.z;
        k.bc[q][j + 3] = v.w;
      }
    }
  }
}

// Four steps of the recurrence for the lane's NPL states; the partial
// sum_j C h of each step goes to LDS.
template <int NPL>
__device__ __forceinline__ void compute_blk(const Blk<NPL>& k, const float (&Al)[NPL],
                                            float (&hs)[NPL], float* __restrict__ pdst) {
  float p4[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float p = 0.0f;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const float a = __builtin_amdgcn_exp2f(k.dl[q] * Al[j]);
      hs[j] = __builtin_fmaf(a, hs[j], k.dx[q] * k.bc[q][j]);
      p = j == 0 ? k.bc[q][NPL] * hs[0] : __builtin_fmaf(k.bc[q][NPL + j], hs[j], p);
    }
    p4[q] = p;
  }
  *reinterpret_cast<float4*>(pdst) = make_float4(p4[0], p4[1], p4[2], p4[3]);
}

// OPT: the optional Mamba-block inputs (flags, z, delta bias) are read;
// without it the kernel is the plain form (an initial state is always taken).
// CK (N <= 16): the state at every 8-step boundary goes to ck,
// laid out as (B*D, nT8, 16), for the backward pass.
template <typename IN, int NPL, bool VEC, bool NPADDED, bool OPT, bool CK>
__global__ __launch_bounds__(64) void selective_fwd_kernel(
    const IN* __restrict__ x, const IN* __restrict__ delta, const float* __restrict__ A,
    const IN* __restrict__ Bm, const IN* __restrict__ Cm, const float* __restrict__ Dskip,
    const IN* __restrict__ z, const float* __restrict__ dbias, const float* __restrict__ h0,
    void* __restrict__ yv, float* __restrict__ h_last, int64_t D, int N, int64_t L, int64_t ndb,
    int64_t nrb, int64_t Lc, int64_t nchunks, uint32_t ntasks,
    unsigned long long* __restrict__ carry, uint32_t* __restrict__ ticket, uint32_t tbase,
    uint32_t epoch, uint32_t flags_in, float* __restrict__ ck, int64_t nT8,
    float* __restrict__ s_out) {
  static_assert(!CK || NPL <= 2, "checkpoints hold 16 states per row");
  constexpr int T = SS_T;
  const uint32_t flags = OPT ? flags_in : 0u;
  constexpr int TS = SS_TS;
  constexpr int PER = 4 * NPL;
  constexpr int LA = Pipe<NPL>::LA;
  constexpr int NS = Pipe<NPL>::NS;
  __shared__ __align__(16) Smem<NPL> sm;

  const int lane = threadIdx.x;
  const int r = lane / SS_G;      // row of this lane within the wavefront
  const int g = lane % SS_G;      // state group: states g*NPL .. g*NPL+NPL-1
  const int tq = (lane % 8) * 4;  // staging and reduce: steps tq .. tq+3 of a tile
  const int btt = lane / 2;       // staging of B/C: step btt of a tile, slots 4*(lane%2)..+3
  const uint32_t st_inc = carry_status(epoch, CARRY_INC);
  float* const p_w = &sm.p[(r * SS_G + g) * TS];
  const float* const p_r = &sm.p[(r * SS_G) * TS + tq];

  for (;;) {
    uint32_t tk = 0;
    if (lane == 0) tk = atomicAdd(ticket, 1u) - tbase;
    const uint32_t id = __builtin_amdgcn_readfirstlane(tk);
    if (id >= ntasks) break;
    const int64_t c = (int64_t)id / nrb;
    const int64_t rb = (int64_t)id - c * nrb;
    const int64_t b = rb / ndb;
    const int64_t d0 = (rb - b * ndb) * SS_RPW;
    const int64_t tb = c * Lc;
    const int64_t te = imin(L, tb + Lc);
    const int ntile = (int)((te - tb + T - 1) / T);

    const int64_t d = d0 + r;
    const bool dok = d < D;
    const int64_t dcl = dok ? d : D - 1;  // rows past D compute a copy of row D-1, never stored
    const int64_t bc_off = b * L * N;
    LanePtrs<IN> lp;
    lp.row = (b * D + dcl) * L;
    lp.dl = delta + lp.row + tq;
    lp.xv = x + lp.row + tq;
    lp.zsrc = (flags & SEL_GATED) ? z : x;
    lp.bc = bc_off + lane * PER;
    const bool ybf = (flags & SEL_Y_BF16) != 0;
    float* const y_row = static_cast<float*>(yv) + (b * D + dcl) * L + tq;
    uint16_t* const y16_row = static_cast<uint16_t*>(yv) + (b * D + dcl) * L + tq;
    // OPT: y before the output gate, for the backward of a gated call (or NULL)
    float* const s_row = (OPT && s_out) ? s_out + (b * D + dcl) * L + tq : nullptr;
    float Al[NPL], hs[NPL];
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int n = g * NPL + j;
      const float av = A[dcl * N + (n < N ? n : N - 1)];
      Al[j] = n < N ? av * LOG2E : 0.0f;  // padded states: a = 1, u = 0 (B masked to 0)
      hs[j] = (c == 0 && h0 && n < N) ? h0[(b * D + dcl) * N + n] : 0.0f;
    }
    const float dsk = Dskip ? Dskip[dcl] : 0.0f;
    const float dbv = (OPT && dbias) ? dbias[dcl] : 0.0f;

    if (c > 0) {  // state entering the chunk: the previous chunk's final state
      const unsigned long long* cw = carry + ((c - 1) * nrb + rb) * (64 * NPL) + lane * NPL;
#pragma unroll
      for (int j = 0; j < NPL; ++j) {
        unsigned long long w;
        while ((uint32_t)((w = carry_get(cw + j)) >> 32) != st_inc) __builtin_amdgcn_s_sleep(2);
        hs[j] = __uint_as_float((uint32_t)w);
      }
    }

    TaskRsrc rs;
    if constexpr (VEC) {
      const int64_t rows = imin(SS_RPW, D - d0);
      const int64_t row0 = b * D + d0;
      rs.x = buffer_rsrc(x + row0 * L, (uint32_t)(rows * L * (int64_t)sizeof(IN)));
      rs.dl = buffer_rsrc(delta + row0 * L, (uint32_t)(rows * L * (int64_t)sizeof(IN)));
      rs.bm = buffer_rsrc(Bm + bc_off, (uint32_t)(L * N * (int64_t)sizeof(IN)));
      rs.cm = buffer_rsrc(Cm + bc_off, (uint32_t)(L * N * (int64_t)sizeof(IN)));
      rs.z = buffer_rsrc(((flags & SEL_GATED) ? z : x) + row0 * L,
                         (uint32_t)(rows * L * (int64_t)sizeof(IN)));
      rs.row_off = (int32_t)(((dcl - d0) * L + tq) * (int64_t)sizeof(IN));
      rs.bc_off = (int32_t)(lane * PER * (int)sizeof(IN));
    }

    // a tile is full when it lies inside both the chunk and the sequence
    auto is_full = [&](int kt) { return tb + (int64_t)(kt + 1) * T <= te; };
    // Load tile kt.  The vector path loads every tile, including those past
    // the end of the chunk, so that each call issues the same loads.
    auto fetch = [&](TileRaw<IN, NPL>& rr, int kt) {
      const int64_t t0 = tb + (int64_t)kt * T;
      if constexpr (VEC)
        load_tile_buf<OPT>(rr, rs, N, t0);
      else if (kt < ntile)
        load_tile<false, NPADDED, OPT>(rr, lp, x, delta, Bm, Cm, bc_off, N, L, t0, lane);
    };

    // Widen (and, in a tail tile, mask) tile kt from `rr` into LDS buffer
    // `buf`; yd gets Dskip*x of this lane's four staging steps.
    auto stage = [&](const TileRaw<IN, NPL>& rr, int kt, int buf, float (&yd)[4],
                     float (&gt)[4], auto full) {
      constexpr bool FULL = decltype(full)::value;
      const int64_t t0 = tb + (int64_t)kt * T;
      float dl4[4], dx4[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float dv = rr.dl.get(q), xv = rr.xv.get(q);
        gt[q] = 1.0f;
        if constexpr (OPT) {
          dv += dbv;
          if (flags & SEL_SOFTPLUS) dv = softplus_f32(dv);
          if (flags & SEL_GATED) gt[q] = silu_f32(rr.zv.get(q));
        }
        if constexpr (!FULL) {
          if (t0 + tq + q >= te) dv = xv = 0.0f;  // identity step: a = 1, u = 0
        }
        dl4[q] = dv;
        dx4[q] = dv * xv;
        yd[q] = dsk * xv;
      }
      *reinterpret_cast<float4*>(&sm.dl[buf][r * TS + tq]) =
          make_float4(dl4[0], dl4[1], dl4[2], dl4[3]);
      *reinterpret_cast<float4*>(&sm.dx[buf][r * TS + tq]) =
          make_float4(dx4[0], dx4[1], dx4[2], dx4[3]);
      // this lane holds step btt = lane/2, states (lane%2)*4*NPL .. +4*NPL-1,
      // i.e. slots 4*(lane%2) .. +3; one slot [B.., C..] is written at a time
      const bool tmask = !FULL && t0 + btt >= te;
      float* const bcw = &sm.bc[buf][btt * bc_stride<NPL>() + 4 * (lane % 2) * (2 * NPL)];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        float v[2 * NPL];
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
          float bv = rr.bb.get(k * NPL + j), cv = rr.cc.get(k * NPL + j);
          if constexpr (NPADDED) {
            if ((4 * (lane % 2) + k) * NPL + j >= N) bv = cv = 0.0f;
          }
          if constexpr (!FULL) {
            if (tmask) bv = cv = 0.0f;
          }
          v[j] = bv;
          v[NPL + j] = cv;
        }
        float* dst = bcw + k * (2 * NPL);
        if constexpr (NPL == 1) {
          *reinterpret_cast<float2*>(dst) = make_float2(v[0], v[1]);
        } else {
#pragma unroll
          for (int j = 0; j < 2 * NPL; j += 4)
            *reinterpret_cast<float4*>(dst + j) = make_float4(v[j], v[j + 1], v[j + 2], v[j + 3]);
        }
      }
    };

    // y of tile kt: Dskip*x plus the 8 partials read into pr, times the gate,
    // stored along t (fp32, or bf16 rounded to nearest even)
    auto finish_reduce = [&](int kt, const float4 (&pr)[SS_G], const float (&yd)[4],
                             const float (&gt)[4]) {
      const int64_t t = tb + (int64_t)kt * T + tq;
      float sv[4] = {yd[0], yd[1], yd[2], yd[3]};
#pragma unroll
      for (int gg = 0; gg < SS_G; ++gg) {
        sv[0] += pr[gg].x;
        sv[1] += pr[gg].y;
        sv[2] += pr[gg].z;
        sv[3] += pr[gg].w;
      }
      if constexpr (OPT) {
        if (s_row && dok) {
          if (VEC && is_full(kt)) {
            *reinterpret_cast<float4*>(s_row + (t - tq)) = make_float4(sv[0], sv[1], sv[2], sv[3]);
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
              if (t + q < te) s_row[t - tq + q] = sv[q];
          }
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) sv[q] *= gt[q];
      if (dok) {
        if (VEC && is_full(kt)) {
          if (ybf)
            *reinterpret_cast<uint2*>(y16_row + (t - tq)) =
                make_uint2(bf16x2_rne(sv[0], sv[1]), bf16x2_rne(sv[2], sv[3]));
          else
            *reinterpret_cast<float4*>(y_row + (t - tq)) = make_float4(sv[0], sv[1], sv[2], sv[3]);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (t + q < te) {
              if (ybf)
                y16_row[t - tq + q] = (uint16_t)bf16_rne(sv[q]);
              else
                y_row[t - tq + q] = sv[q];
            }
          }
        }
      }
    };
    auto read_partials = [&](float4 (&pr)[SS_G]) {
#pragma unroll
      for (int gg = 0; gg < SS_G; ++gg) pr[gg] = *reinterpret_cast<const float4*>(p_r + gg * TS);
    };

    TileRaw<IN, NPL> raw0, raw1;  // tile j is held in raw(j % 2)
    Blk<NPL> ops[NS];             // block i of a tile uses ops[i % NS]
    float ydc[4] = {0.f, 0.f, 0.f, 0.f};  // Dskip*x of the tile in compute
    float ydp[4] = {0.f, 0.f, 0.f, 0.f};  // ... and of the tile awaiting its reduce
    float gtc[4] = {1.f, 1.f, 1.f, 1.f};  // output gate of the tile in compute
    float gtp[4] = {1.f, 1.f, 1.f, 1.f};  // ... and of the tile awaiting its reduce

    // Tile kt (buffer BUF = kt % 2): stage tile kt+1 from `rn` into the other
    // buffer and refill `rn` with tile kt+3; issue the reads of tile kt-1's
    // partials; compute the 8 blocks with reads LA blocks ahead, and finish
    // tile kt-1's reduce after the first block.
    auto tile = [&](int kt, TileRaw<IN, NPL>& rn, auto bufc) {
      constexpr int BUF = decltype(bufc)::value;
      const bool has_next = kt + 1 < ntile;
      float ydn[4] = {0.f, 0.f, 0.f, 0.f}, gtn[4] = {1.f, 1.f, 1.f, 1.f};
      wave_sync();
      if (has_next) {
        if (is_full(kt + 1))
          stage(rn, kt + 1, 1 - BUF, ydn, gtn, Flag<true>());
        else
          stage(rn, kt + 1, 1 - BUF, ydn, gtn, Flag<false>());
      }
      fetch(rn, kt + 3);
      float4 pr[SS_G];
      if (kt > 0) read_partials(pr);
      wave_sync();
#pragma unroll
      for (int bi = 0; bi < SS_NB; ++bi) {
        const int nb = bi + LA;
        if (nb < SS_NB)
          read_blk(ops[nb % NS], sm, BUF, r, g, nb);
        else if (has_next)
          read_blk(ops[nb % NS], sm, 1 - BUF, r, g, nb - SS_NB);
        // keep the read-ahead where it is: the scheduler would otherwise sink
        // the reads next to their use and expose the LDS latency
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (CK) {
          // the state before step tb + kt*T + 4*bi (states past N and rows
          // past D write to their own unused slots / row D-1's, same values)
          const int64_t t8 = (tb + (int64_t)kt * T + 4 * bi) / 8;
          if ((bi & 1) == 0 && t8 < nT8) {
#pragma unroll
            for (int j = 0; j < NPL; ++j)
              ck[((b * D + dcl) * nT8 + t8) * 16 + g * NPL + j] = hs[j];
          }
        }
        compute_blk(ops[bi % NS], Al, hs, p_w + 4 * bi);
        if (bi == 0 && kt > 0) finish_reduce(kt - 1, pr, ydp, gtp);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        ydp[q] = ydc[q];
        ydc[q] = ydn[q];
        gtp[q] = gtc[q];
        gtc[q] = gtn[q];
      }
    };

    fetch(raw0, 0);
    fetch(raw1, 1);
    if (is_full(0))
      stage(raw0, 0, 0, ydc, gtc, Flag<true>());
    else
      stage(raw0, 0, 0, ydc, gtc, Flag<false>());
    fetch(raw0, 2);
    wave_sync();
#pragma unroll
    for (int i = 0; i < LA; ++i) read_blk(ops[i], sm, 0, r, g, i);
    for (int kt = 0; kt < ntile; kt += 2) {
      tile(kt, raw1, Int<0>());
      if (kt + 1 < ntile) tile(kt + 1, raw0, Int<1>());
    }
    {
      wave_sync();
      float4 pr[SS_G];
      read_partials(pr);
      finish_reduce(ntile - 1, pr, ydp, gtp);
    }
    wave_sync();  // the next task rewrites this wavefront's LDS

    if (c + 1 < nchunks) {
      unsigned long long* out = carry + (c * nrb + rb) * (64 * NPL) + lane * NPL;
#pragma unroll
      for (int j = 0; j < NPL; ++j) carry_put(out + j, st_inc, __float_as_uint(hs[j]));
    } else if (h_last && dok) {
#pragma unroll
      for (int j = 0; j < NPL; ++j) {
        const int n = g * NPL + j;
        if (n < N) h_last[(b * D + d) * N + n] = hs[j];
      }
    }
  }
}

struct Plan {
  int64_t ndb, nrb, Lc, nchunks, grid;
  uint32_t ntasks;
};

int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  return (v && *v) ? atoi(v) : dflt;
}

// Persistent grid size and chunking for a launch.
int make_plan(int64_t B, int64_t D, int64_t L, Plan* p) {
  int cus = 0;
  int st = device_cus(&cus);
  if (st != SW_OK) return st;
  // Resident wavefronts per CU and tasks per wavefront (tuning knobs, read
  // per call).  One task per wavefront measured best at Mamba shapes: extra
  // chunks only add waits on the previous chunk's carry.
  const int waves_per_cu = env_int("SW_SS_WAVES_PER_CU", 6);
  const int tasks_per_wave = env_int("SW_SS_TASKS_PER_WAVE", 1);
  p->ndb = (D + SS_RPW - 1) / SS_RPW;
  p->nrb = B * p->ndb;
  int64_t slots = (int64_t)cus * (waves_per_cu > 0 ? waves_per_cu : 6);
  if (slots > p->nrb) slots = p->nrb;  // no more wavefronts than independent chains
  const int64_t tiles = (L + SS_T - 1) / SS_T;
  int64_t want = (slots * (tasks_per_wave > 0 ? tasks_per_wave : 1) + p->nrb - 1) / p->nrb;
  const int64_t max_chunks = (tiles + 3) / 4;  // a chunk keeps at least 4 tiles
  if (want > max_chunks) want = max_chunks;
  if (want < 1) want = 1;
  const int64_t tiles_per_chunk = (tiles + want - 1) / want;
  p->Lc = tiles_per_chunk * SS_T;
  p->nchunks = (L + p->Lc - 1) / p->Lc;
  const int64_t ntasks = p->nrb * p->nchunks;
  if (ntasks >= ((int64_t)1 << 31))
    return fail(SW_ERR_UNSUPPORTED, "%lld tasks exceed the ticket range", (long long)ntasks);
  p->ntasks = (uint32_t)ntasks;
  p->grid = ntasks < slots ? ntasks : slots;
  return SW_OK;
}

template <typename IN, int NPL, bool VEC, bool NPADDED>
int launch_cfg(const SelArgs& a, hipStream_t s) {
  const bool opt = a.z || a.delta_bias || a.softplus || a.y_bf16 || a.s_out;
  Plan p;
  int st = make_plan(a.B, a.D, a.L, &p);
  if (st != SW_OK) return st;
  ScratchSession ss;
  const size_t words = (size_t)(p.nchunks - 1) * p.nrb * 64 * NPL;
  st = ss.reserve(words, p.ntasks + (uint32_t)p.grid, s);
  if (st != SW_OK) return st;
  const uint32_t flags = (a.softplus ? SEL_SOFTPLUS : 0u) | (a.y_bf16 ? SEL_Y_BF16 : 0u) |
                         (a.z ? SEL_GATED : 0u);
  auto kern = opt ? selective_fwd_kernel<IN, NPL, VEC, NPADDED, true, false>
                  : selective_fwd_kernel<IN, NPL, VEC, NPADDED, false, false>;
  if constexpr (NPL <= 2) {
    if (a.ckpt)
      kern = opt ? selective_fwd_kernel<IN, NPL, VEC, NPADDED, true, true>
                 : selective_fwd_kernel<IN, NPL, VEC, NPADDED, false, true>;
  } else {
    if (a.ckpt) return fail(SW_ERR_UNSUPPORTED, "checkpoints need N <= 16");
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)p.grid), dim3(64), 0, s, static_cast<const IN*>(a.x),
                     static_cast<const IN*>(a.delta), a.A, static_cast<const IN*>(a.Bm),
                     static_cast<const IN*>(a.Cm), a.Dskip, static_cast<const IN*>(a.z),
                     a.delta_bias, a.h0, a.y, a.h_last, a.D, (int)a.N, a.L, p.ndb, p.nrb, p.Lc,
                     p.nchunks, p.ntasks, ss.carry, ss.ticket, ss.ticket_base, ss.epoch, flags,
                     a.ckpt, (a.L + 7) / 8, a.s_out);
  st = check_launch("selective_fwd_kernel");
  if (st != SW_OK) ss.invalidate();
  note_launch("selective_fwd_kernel: %d states per lane, %lld chunks per row", NPL,
              (long long)p.nchunks);
  return st;
}

// The vector path reads a tile's B and C as T*N consecutive elements laid out
// as T rows of 8*NPL slots, which holds only when N == 8*NPL; a padded N
// gathers them element by element.
template <typename IN, int NPL>
int launch_npl(const SelArgs& a, bool vec, hipStream_t s) {
  const bool padded = a.N != SS_G * NPL;
  if (vec && !padded) return launch_cfg<IN, NPL, true, false>(a, s);
  return launch_cfg<IN, NPL, false, true>(a, s);
}

}  // namespace

bool row16_fits(int64_t D, int64_t N, int64_t L, size_t es);
template <typename IN>
int launch_row16(const SelArgs& a, hipStream_t s);
template <typename IN>
int launch_row16_states(const SelArgs& a, hipStream_t s);
template <typename IN>
SelPlan plan_row16(const SelArgs& a, int cus);

namespace {

// The vector path loads through buffer resources with 32-bit byte offsets:
// it needs 16-byte aligned B and C (tile starts are then aligned) and every
// offset of a task, including the tiles fetched past the end, below 2^31.
template <typename IN>
bool vector_path(const SelArgs& a) {
  const int64_t es = (int64_t)sizeof(IN), pad = 4 * SS_T;
  const bool fits = SS_RPW * (a.L + pad) * es < ((int64_t)1 << 31) &&
                    (a.L + pad) * a.N * es < ((int64_t)1 << 31);
  return a.vec && fits && ((uintptr_t)a.Bm % 16 == 0) && ((uintptr_t)a.Cm % 16 == 0);
}

// N = 16 on the vector path: one state per lane, 16-lane rows
// (selective_scan16.hip); SW_SS_LAYOUT=8 keeps the 8-lane layout.
template <typename IN>
bool row16_path(const SelArgs& a) {
  return vector_path<IN>(a) && env_int("SW_SS_LAYOUT", 16) == 16 &&
         row16_fits(a.D, a.N, a.L, sizeof(IN));
}

template <typename IN>
int launch_selective(const SelArgs& a) {
  hipStream_t s = current_stream();
  const int64_t N = a.N;
  const bool v = vector_path<IN>(a);
  if (row16_path<IN>(a)) return launch_row16<IN>(a, s);
  if (N <= 8) return launch_npl<IN, 1>(a, v, s);
  if (N <= 16) return launch_npl<IN, 2>(a, v, s);
  if (N <= 32) return launch_npl<IN, 4>(a, v, s);
  return launch_npl<IN, 8>(a, v, s);
}

}  // namespace

int selective_fwd(const SelArgs& a) {
  return a.bf16_in ? launch_selective<uint16_t>(a) : launch_selective<float>(a);
}

SelPlan selective_plan(const SelArgs& a, int cus) {
  SelPlan q;
  if (a.B * a.D == 0 || a.L == 0) return q;
  if (a.bf16_in ? row16_path<uint16_t>(a) : row16_path<float>(a))
    return a.bf16_in ? plan_row16<uint16_t>(a, cus) : plan_row16<float>(a, cus);
  q.layout = 8;
  q.nseg = 1;
  q.lseg = a.L;
  return q;
}

int selective_states_fwd(const SelArgs& a, bool* taken) {
  *taken = false;
  if (a.N != 16 || !a.ckpt || a.z || a.y_bf16 || a.s_out) return SW_OK;
  if (a.bf16_in ? !row16_path<uint16_t>(a) : !row16_path<float>(a)) return SW_OK;
  *taken = true;
  hipStream_t s = current_stream();
  return a.bf16_in ? launch_row16_states<uint16_t>(a, s) : launch_row16_states<float>(a, s);
}

}  // namespace sw
