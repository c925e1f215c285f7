// selective_scan_quad.hip -- fused selective scan, forward, N = 16, for calls
// with few (b,d) rows and long sequences, on gfx950.
//
// The operation is that of selective_scan16.hip (the Mamba-style instance of
// the affine recurrence, Sec. 1 and Sec. 3.1; segments composed with Eq. (7)):
//   a_{t,n} = exp(delta_t A_n),  u_{t,n} = delta_t B_{t,n} x_t,
//   h_{t,n} = a_{t,n} h_{t-1,n} + u_{t,n},  y_t = sum_n C_{t,n} h_{t,n} + Dskip x_t.
//
// Layout: a row is a quad of lanes, lane g of the quad owning states 4g ..
// 4g+3, and a wavefront walks 16 rows on its own -- no workgroup barrier, no
// LDS shared between wavefronts.  Per step a lane does the method's work on
// its four states with plain VGPR operands (a scalar or DPP operand makes an
// fp32 operation on this part cost nearly twice as much): delta*A log2e,
// exp2, (delta x)*B and the state FMA per state, and C*h summed over its four
// states in registers.  The four partial sums of a row meet within the quad:
// a transpose-reduce over each 4-step block (two exchange levels, three DPP
// adds per lane) leaves lane g the sum of step 4j+g, which it adds to Dskip x
// and stores.  Each wavefront stages its own tile in a private slice of LDS
// (delta', delta' x, Dskip x of its 16 rows, B and C of the tile), which it
// reads back as 16-byte reads shared by the lanes of a quad (delta) or by all
// lanes of a state group (B, C).  Global memory moves in 32-step tiles, 128
// contiguous bytes of a row per 8 lanes (x, delta, z loaded a tile ahead; y
// stored from a small LDS transpose by the lanes that hold its x and z); y
// and fp32 x, delta, z, read or written once in whole lines, go non-temporal,
// B and C (read by every row block of the batch) do not.
//
// With four lanes per row the parallelism is a quarter of one lane per state,
// so rows are cut into segments and walked in the correction form of
// selective_scan16.hip (the same records in y, the same fold): (1) every
// segment walks from a zero state (the first from h0), (2) the fold composes
// the records, (3) each later segment walks again from its composed state
// until, for every state of the wavefront, the carried part has faded below
// 2^-26 of the state's own magnitude (checked every 64 steps, per wavefront).


#include "selective_common.h"

namespace sw {

// The fold of the correction form (selective_scan16.hip).
void launch_fold_corr(float* y, float* h_last, int64_t R, int64_t L, int64_t nseg, int64_t Lseg,
                      hipStream_t s);

namespace {

constexpr int Q_RPW = 16;    // rows per wavefront (a quad of lanes per row)
constexpr int Q_WAVES = 4;   // wavefronts per workgroup (independent)
constexpr int Q_S = 4;       // states per lane: lane g of a quad owns states 4g .. 4g+3
constexpr int Q_N = 16;      // states per row
constexpr int Q_T = 32;      // steps per tile
constexpr int Q_TPV = 2;     // tiles between the checks of the correction walk
constexpr int Q_SKIP = 64;   // first steps of a later segment whose y holds its records
constexpr int Q_MAX_SEG = 16;  // segments per row at most (the fold walks them in order)
constexpr float Q_LOG2E = 1.4426950408889634f;
constexpr float Q_EPS = 1.4901161193847656e-08f;  // 2^-26, as in selective_scan16.hip
static_assert(Q_SKIP == Q_T * Q_TPV, "the first check covers the records' steps");

enum : int { Q_ALL = 0, Q_CORR = 1 };

// One wavefront's tile (10 KB: four workgroups fit a CU).  delta' and
// delta' x are [row][step] with the 4-step blocks of row r rotated by r
// (block j at word 4 * ((j + r) & 7)), so the 16 quads reading block j at
// once fall on distinct banks; the y sums are [row][step] with the blocks of
// row r permuted by (r / 2) & 7 (XOR), so that both the 4-byte writes of the
// walk and the 16-byte reads of the store avoid bank conflicts.
struct QTile {
  float dl[Q_RPW * Q_T];  // delta'
  float dx[Q_RPW * Q_T];  // delta' * x
  float4 bc[Q_T][4][2];   // [step][state group]: B, then C, of states 4g .. 4g+3
  float yt[Q_RPW * Q_T];  // sum_n C h of the tile, before Dskip x and the gate
};
struct QSmem {
  QTile tile[Q_WAVES];
};

__device__ __forceinline__ int qswz(int r, int j) { return r * Q_T + 4 * ((j + r) & 7); }
__device__ __forceinline__ int yswz(int r, int j) { return r * Q_T + 4 * (j ^ ((r >> 1) & 7)); }

// Value of `v` in the lane of this quad whose index differs by M (M = 1, 2).
template <int M>
__device__ __forceinline__ float quad_xor(float v) {
  // quad_perm selectors: [1,0,3,2] for M = 1, [2,3,0,1] for M = 2
  constexpr int sel =
      M == 1 ? (1 | (0 << 2) | (3 << 4) | (2 << 6)) : (2 | (3 << 2) | (0 << 4) | (1 << 6));
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), sel, 0xf, 0xf, false));
}

// LDS writes of this wavefront are seen by its later LDS reads in every lane,
// and its earlier reads are done before its later writes.
__device__ __forceinline__ void q_wave_order() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// MODE Q_ALL: every segment (or the whole row, nseg = 1) from a zero state
// (segment 0 from h0), y stored except in the first Q_SKIP steps of later
// segments, records written.  MODE Q_CORR: segments 1 .. nseg-1 from the
// initial states the fold left in their first words, y rewritten until the
// carried part has faded.  Workgroups are (row block, segment) pairs,
// blockIdx.x = block * segments of the launch + segment; a row block is
// Q_WAVES * Q_RPW rows of one batch.  L and Lseg are multiples of the tile.
template <typename IN, bool OPT, int MODE>
__global__ __launch_bounds__(256) void selective_quad_kernel(
    const IN* __restrict__ x, const IN* __restrict__ delta, const float* __restrict__ A,
    const IN* __restrict__ Bm, const IN* __restrict__ Cm, const float* __restrict__ Dskip,
    const IN* __restrict__ z, const float* __restrict__ dbias, const float* __restrict__ h0,
    float* __restrict__ y, float* __restrict__ h_last, int D, int L, int nblk,
    uint32_t flags_in, float* __restrict__ s_out, int nseg, int Lseg) {
  constexpr bool CORR = MODE == Q_CORR;
  constexpr int ES = (int)sizeof(IN);
  constexpr int XPOL = ES == 4 ? SW_NT : 0;  // cache policy of the x, delta, z loads
  const uint32_t flags = OPT ? flags_in : 0u;
  const bool gated = OPT && (flags & SEL_GATED);
  __shared__ __align__(16) QSmem sm;

  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int nsl = CORR ? nseg - 1 : nseg;
  const int sg = (int)(blockIdx.x % (unsigned)nsl) + (CORR ? 1 : 0);
  const int blk = (int)(blockIdx.x / (unsigned)nsl);
  const int b = blk / nblk;
  const int d0 = (blk - b * nblk) * (Q_WAVES * Q_RPW) + w * Q_RPW;  // first row of the wavefront
  if (d0 >= D) return;  // wavefronts are independent: one past D has nothing to walk
  const int rows = D - d0 < Q_RPW ? D - d0 : Q_RPW;
  const int ts = sg * Lseg;                       // first step of the segment
  const int Ls = sg == nseg - 1 ? L - ts : Lseg;  // its steps (a multiple of Q_T)
  const int ntile = Ls / Q_T;
  const int64_t row0 = (int64_t)b * D + d0;
  QTile& tl = sm.tile[w];

  // ---- walk: lane = (row r, state group g)
  const int r = lane >> 2, g = lane & 3;
  const bool dok = r < rows;
  const int rcl = dok ? r : rows - 1;  // rows past D walk a copy of the last row, never stored
  const int64_t grow = row0 + rcl;
  const int n0 = Q_S * g;
  // A, h0 and h_last are only naturally aligned: element accesses
  float Al[Q_S], h[Q_S], hin[Q_S], mag[Q_S];
#pragma unroll
  for (int i = 0; i < Q_S; ++i) {
    Al[i] = A[(int64_t)(d0 + rcl) * Q_N + n0 + i] * Q_LOG2E;
    h[i] = (!CORR && sg == 0 && h0) ? h0[grow * Q_N + n0 + i] : 0.0f;
    mag[i] = 0.0f;
  }
  if constexpr (CORR) {
    const float4 v = *reinterpret_cast<const float4*>(y + grow * L + ts + n0);  // the fold's state
    h[0] = v.x;
    h[1] = v.y;
    h[2] = v.z;
    h[3] = v.w;
  }
#pragma unroll
  for (int i = 0; i < Q_S; ++i) hin[i] = h[i];

  // ---- streaming: lane l moves steps 4 (l % 8) .. +3 of rows l / 8 and
  // l / 8 + 8 (128 contiguous bytes of a row per 8 lanes), and the B and C
  // float4s of steps l / 4 and l / 4 + 16 for state group l % 4
  const int ir = lane >> 3, ij = lane & 7;
  int iro[2];
  int32_t ioff[2];
  float idsk[2], idb[2];
  bool iok[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int rr = ir + 8 * k;
    iok[k] = rr < rows;
    iro[k] = iok[k] ? rr : rows - 1;
    ioff[k] = (iro[k] * L + 4 * ij) * ES;
    idsk[k] = Dskip ? Dskip[d0 + iro[k]] : 0.0f;
    idb[k] = (OPT && dbias) ? dbias[d0 + iro[k]] : 0.0f;
  }
  const uint32_t rbytes = (uint32_t)(((int64_t)rows * L - ts) * ES);
  const __amdgpu_buffer_rsrc_t rx = buffer_rsrc(x + row0 * L + ts, rbytes);
  const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(delta + row0 * L + ts, rbytes);
  const __amdgpu_buffer_rsrc_t rz = buffer_rsrc((gated ? z : x) + row0 * L + ts, rbytes);
  const uint32_t bcbytes = (uint32_t)(((int64_t)L - ts) * Q_N * ES);
  const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(Bm + ((int64_t)b * L + ts) * Q_N, bcbytes);
  const __amdgpu_buffer_rsrc_t rc = buffer_rsrc(Cm + ((int64_t)b * L + ts) * Q_N, bcbytes);
  const int32_t boff = ((lane >> 2) * Q_N + Q_S * (lane & 3)) * ES;
  // y (and the pre-gate output) leave through resources over the
  // wavefront's rows from the segment's start; a lane with nothing to store
  // aims at the resource's end, where the store is dropped (16 rows of
  // L < 2^26 fp32 steps fit 32 bits)
  const uint32_t ybytes = (uint32_t)(((int64_t)rows * L - ts) * 4);
  const __amdgpu_buffer_rsrc_t ry = buffer_rsrc(y + row0 * L + ts, ybytes);
  const __amdgpu_buffer_rsrc_t rso = buffer_rsrc(OPT && s_out ? s_out + row0 * L + ts : y, ybytes);
  struct Raw {
    RawVec<IN, 4> d[2], x[2], z[2], b[2], c[2];
  };
  Raw nx;                      // raw inputs of the next tile
  float xc[2][4], zc[2][4];    // x and z of the tile whose y is stored next
  float xn[2][4], zn[2][4];    // the same of the tile staged last
  float dsum[2] = {0.f, 0.f};  // this lane's share of the sum of delta' of rows l/8, l/8+8
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int32_t off = ioff[k] + kt * (Q_T * ES);
      // x, delta and z are read once: non-temporal in fp32, where a tile of a
      // row is one whole 128-byte line (in bf16 it is half a line, whose other
      // half the next tile reads: the default policy measured faster there)
      nx.d[k].template load_buf<XPOL>(rd, off);
      nx.x[k].template load_buf<XPOL>(rx, off);
      if constexpr (OPT) nx.z[k].template load_buf<XPOL>(rz, off);
      const int32_t bo = boff + (kt * Q_T + 16 * k) * (Q_N * ES);
      nx.b[k].load_buf(rb, bo);
      nx.c[k].load_buf(rc, bo);
    }
  };
  // widen the next tile into LDS (delta', delta' x, B, C); keep its x and z
  auto stage_tile = [&]() {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      float dv4[4], dx4[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float dv = nx.d[k].get(q);
        const float xv = nx.x[k].get(q);
        if constexpr (OPT) {
          dv += idb[k];
          if (flags & SEL_SOFTPLUS) dv = softplus_f32(dv);
          zn[k][q] = gated ? silu_f32(nx.z[k].get(q)) : 1.0f;
        }
        dsum[k] += dv;
        dv4[q] = dv;
        dx4[q] = dv * xv;
        xn[k][q] = xv;
      }
      const int o = qswz(ir + 8 * k, ij);
      *reinterpret_cast<float4*>(&tl.dl[o]) = make_float4(dv4[0], dv4[1], dv4[2], dv4[3]);
      *reinterpret_cast<float4*>(&tl.dx[o]) = make_float4(dx4[0], dx4[1], dx4[2], dx4[3]);
      tl.bc[(lane >> 2) + 16 * k][lane & 3][0] =
          make_float4(nx.b[k].get(0), nx.b[k].get(1), nx.b[k].get(2), nx.b[k].get(3));
      tl.bc[(lane >> 2) + 16 * k][lane & 3][1] =
          make_float4(nx.c[k].get(0), nx.c[k].get(1), nx.c[k].get(2), nx.c[k].get(3));
    }
  };
  // the staged tile's x and z become those of the next y store
  auto take_next = [&]() {
#pragma unroll
    for (int k = 0; k < 2; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        xc[k][q] = xn[k][q];
        if constexpr (OPT) zc[k][q] = zn[k][q];
      }
  };
  // the sum of delta' of row r (over the staged tiles), in every lane of quad r
  auto row_dsum = [&]() {
    // rows l/8 and l/8+8 from the 8 lanes that stage each, then to the quads
    float s0 = dsum[0], s1 = dsum[1];
#pragma unroll
    for (int m = 1; m < 8; m *= 2) {
      s0 += __shfl_xor(s0, m, 8);
      s1 += __shfl_xor(s1, m, 8);
    }
    // row r's sum sits in lanes 8 (r % 8) .. of s0 (r < 8) or s1 (r >= 8)
    const float a = __shfl(s0, 8 * (r & 7)), c = __shfl(s1, 8 * (r & 7));
    return r < 8 ? a : c;
  };

  // ---- one tile: the lane's four states over 32 steps; lane g ends each
  // 4-step block j with the full sum of step 4j+g, kept in the y tile
  auto walk = [&]() {
#pragma unroll
    for (int j = 0; j < Q_T / 4; ++j) {
      const int o = qswz(r, j);
      const float4 dl4 = *reinterpret_cast<const float4*>(&tl.dl[o]);
      const float4 dx4 = *reinterpret_cast<const float4*>(&tl.dx[o]);
      const float dlq[4] = {dl4.x, dl4.y, dl4.z, dl4.w};
      const float dxq[4] = {dx4.x, dx4.y, dx4.z, dx4.w};
      float p[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float4 b4 = tl.bc[4 * j + k][g][0];
        const float4 c4 = tl.bc[4 * j + k][g][1];
        const float bq[4] = {b4.x, b4.y, b4.z, b4.w};
        const float cq[4] = {c4.x, c4.y, c4.z, c4.w};
        float acc = 0.0f;
#pragma unroll
        for (int i = 0; i < Q_S; ++i) {
          const float a = __builtin_amdgcn_exp2f(dlq[k] * Al[i]);
          const float u = dxq[k] * bq[i];
          h[i] = __builtin_fmaf(a, h[i], u);
          if constexpr (CORR) mag[i] = __builtin_fmaf(a, mag[i], __builtin_fabsf(u));
          acc = i == 0 ? cq[i] * h[i] : __builtin_fmaf(cq[i], h[i], acc);
        }
        p[k] = acc;
      }
      // transpose-reduce over the quad: after the xor-1 level lane g holds
      // the pair sums of steps g&1 and 2+(g&1), after the xor-2 level the
      // full sum of step g
      const bool o1 = (g & 1) != 0, o2 = (g & 2) != 0;
      const float q0 = (o1 ? p[1] : p[0]) + quad_xor<1>(o1 ? p[0] : p[1]);
      const float q1 = (o1 ? p[3] : p[2]) + quad_xor<1>(o1 ? p[2] : p[3]);
      tl.yt[yswz(r, j) + g] = (o2 ? q1 : q0) + quad_xor<2>(o2 ? q0 : q1);
    }
  };
  // y of the tile: Dskip x added, the gate applied, 16 bytes per lane
  auto store_y = [&](int kt) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int rr = ir + 8 * k;
      float4 s = *reinterpret_cast<const float4*>(&tl.yt[yswz(rr, ij)]);
      s.x = __builtin_fmaf(idsk[k], xc[k][0], s.x);
      s.y = __builtin_fmaf(idsk[k], xc[k][1], s.y);
      s.z = __builtin_fmaf(idsk[k], xc[k][2], s.z);
      s.w = __builtin_fmaf(idsk[k], xc[k][3], s.w);
      const int t = kt * Q_T + 4 * ij;
      const bool store = iok[k] && !(!CORR && sg > 0 && t < Q_SKIP);
      const uint32_t at = store ? (uint32_t)(iro[k] * L + t) * 4u : ybytes;
      if constexpr (OPT) {
        if (s_out)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(sw_u32x4, s), rso, (int)at, 0,
                                                 SW_NT);
        s.x *= zc[k][0];
        s.y *= zc[k][1];
        s.z *= zc[k][2];
        s.w *= zc[k][3];
      }
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(sw_u32x4, s), ry, (int)at, 0,
                                             SW_NT);
    }
  };

  // ---- prologue: tile 0 staged, tile 1 in flight
  load_tile(0);
  stage_tile();
  take_next();
  load_tile(1);
  q_wave_order();

  // One tile: walk it, store its y, stage the next and load the one after.
  // (A second tile of loads in flight measured no faster and doubles the
  // registers of the correction walk.)  In the plain walk from zero the next
  // tile is staged before the y store: that ends the loaded registers' life
  // before the y values are formed.  With the store first both were live at
  // once, the compiler moved the loaded values at the loop's join, and each
  // move waited for its load as soon as issued.  (The correction walk and the
  // calls with options keep that order: the carried x and z of the staged
  // tile would cost them a wavefront per SIMD.)
  constexpr bool STAGE_FIRST = !CORR && !OPT;
  int kt_end = ntile;  // the correction walk lowers it once the carried part has faded
#pragma unroll 1
  for (int kt = 0; kt < kt_end; ++kt) {
    walk();
    if constexpr (CORR) {
      if ((kt % Q_TPV) == Q_TPV - 1) {
        // the carried part of each state, P h_in with P = exp2(A log2e * the
        // row's sum of delta' through tile kt), against the walk's own
        // magnitude; the wavefront stops when every lane is done
        const float S = row_dsum();
        bool done = true;
#pragma unroll
        for (int i = 0; i < Q_S; ++i)
          done = done && __builtin_fabsf(__builtin_amdgcn_exp2f(Al[i] * S) * hin[i]) <=
                             Q_EPS * mag[i];
        done = done || !dok;
        if (__builtin_amdgcn_ballot_w64(!done) == 0) kt_end = kt + 1;
      }
    }
    q_wave_order();  // the tile's reads are done and its y sums written
    const bool more = kt + 1 < kt_end;
    if (STAGE_FIRST && more) stage_tile();
    store_y(kt);
    if (more) {
      if (!STAGE_FIRST) stage_tile();
      take_next();
      load_tile(kt + 2);
    }
    q_wave_order();
  }

  if constexpr (!CORR) {
    const float S = nseg > 1 ? row_dsum() : 0.0f;
    if (nseg > 1 && dok) {
      // the records: P and end state of each state of the row, in the first
      // words of the next segment (the last segment: P beside the records in
      // its own first words, the end state in h_last)
      float* wd = y + grow * L;
      float P[Q_S];
#pragma unroll
      for (int i = 0; i < Q_S; ++i) P[i] = __builtin_amdgcn_exp2f(Al[i] * S);
      if (sg < nseg - 1) {
        wd += ts + Ls;
        *reinterpret_cast<float4*>(wd + n0) = make_float4(P[0], P[1], P[2], P[3]);
        *reinterpret_cast<float4*>(wd + Q_N + n0) = make_float4(h[0], h[1], h[2], h[3]);
      } else {
        wd += ts;
        *reinterpret_cast<float4*>(wd + 2 * Q_N + n0) = make_float4(P[0], P[1], P[2], P[3]);
      }
    }
    if (h_last && dok && sg == nseg - 1) {
#pragma unroll
      for (int i = 0; i < Q_S; ++i) h_last[grow * Q_N + n0 + i] = h[i];
    }
  }
}

template <typename IN, bool OPT>
void launch_quad_t(const SelArgs& a, uint32_t flags, int64_t nseg, int64_t Lseg, hipStream_t s) {
  const int64_t nblk = (a.D + Q_WAVES * Q_RPW - 1) / (Q_WAVES * Q_RPW);
  const int64_t blocks = a.B * nblk;
  hipLaunchKernelGGL((selective_quad_kernel<IN, OPT, Q_ALL>), dim3((unsigned)(blocks * nseg)),
                     dim3(256), 0, s, static_cast<const IN*>(a.x),
                     static_cast<const IN*>(a.delta), a.A, static_cast<const IN*>(a.Bm),
                     static_cast<const IN*>(a.Cm), a.Dskip, static_cast<const IN*>(a.z),
                     a.delta_bias, a.h0, static_cast<float*>(a.y), a.h_last, (int)a.D, (int)a.L,
                     (int)nblk, flags, a.s_out, (int)nseg, (int)Lseg);
  if (nseg < 2) return;
  launch_fold_corr(static_cast<float*>(a.y), a.h_last, a.B * a.D, a.L, nseg, Lseg, s);
  hipLaunchKernelGGL((selective_quad_kernel<IN, OPT, Q_CORR>),
                     dim3((unsigned)(blocks * (nseg - 1))), dim3(256), 0, s,
                     static_cast<const IN*>(a.x), static_cast<const IN*>(a.delta), a.A,
                     static_cast<const IN*>(a.Bm), static_cast<const IN*>(a.Cm), a.Dskip,
                     static_cast<const IN*>(a.z), a.delta_bias, a.h0, static_cast<float*>(a.y),
                     nullptr, (int)a.D, (int)a.L, (int)nblk, flags, a.s_out, (int)nseg,
                     (int)Lseg);
}

}  // namespace

// True when the quad layout can take the call: fp32 y, no checkpoints,
// N = 16, whole tiles, 32-bit offsets over a wavefront's rows and a batch's
// B and C.  (Which layout and how many segments a call takes is decided with
// the 16-lane layout's choices, in selective_scan16.hip.)
template <typename IN>
bool quad_fits(const SelArgs& a) {
  if (a.N != Q_N || a.y_bf16 || a.ckpt || a.L <= 0 || a.B * a.D <= 0) return false;
  if (a.L % Q_T != 0 || a.D >= ((int64_t)1 << 30) || a.L >= ((int64_t)1 << 26)) return false;
  if ((Q_RPW * (a.L + 4 * Q_T)) * (int64_t)sizeof(IN) >= ((int64_t)1 << 31)) return false;
  if ((a.L + 4 * Q_T) * Q_N * (int64_t)sizeof(IN) >= ((int64_t)1 << 31)) return false;
  return a.B * ((a.D + Q_WAVES * Q_RPW - 1) / (Q_WAVES * Q_RPW)) * Q_MAX_SEG < ((int64_t)1 << 31);
}

// Launches the quad layout with nseg segments of Lseg steps (the last takes
// the rest, at least Q_SKIP steps: its first words hold the records of the
// segment before and its own P; Lseg a multiple of Q_SKIP, 1 <= nseg <=
// Q_MAX_SEG); the call must satisfy quad_fits.
template <typename IN>
int launch_quad(const SelArgs& a, int64_t nseg, int64_t Lseg, hipStream_t s) {
  if (nseg < 1 || nseg > Q_MAX_SEG || (nseg > 1 && (Lseg < Q_SKIP || Lseg % Q_SKIP != 0 ||
                                                    a.L - (nseg - 1) * Lseg < Q_SKIP)))
    return fail(SW_ERR_UNSUPPORTED, "quad layout: %lld segments of %lld steps for L=%lld",
                (long long)nseg, (long long)Lseg, (long long)a.L);
  if (nseg == 1) Lseg = a.L;
  const bool opt = a.z || a.delta_bias || a.softplus || a.s_out;
  const uint32_t flags = (a.softplus ? SEL_SOFTPLUS : 0u) | (a.z ? SEL_GATED : 0u);
  if (opt)
    launch_quad_t<IN, true>(a, flags, nseg, Lseg, s);
  else
    launch_quad_t<IN, false>(a, flags, nseg, Lseg, s);
  if (nseg > 1)
    note_launch("selective_quad_kernel: %lld segments of %lld steps, correction form (3 launches)",
                (long long)nseg, (long long)Lseg);
  else
    note_launch("selective_quad_kernel: whole rows");
  return check_launch("selective_quad_kernel");
}

template bool quad_fits<float>(const SelArgs&);
template bool quad_fits<uint16_t>(const SelArgs&);
template int launch_quad<float>(const SelArgs&, int64_t, int64_t, hipStream_t);
template int launch_quad<uint16_t>(const SelArgs&, int64_t, int64_t, hipStream_t);

}  // namespace sw
