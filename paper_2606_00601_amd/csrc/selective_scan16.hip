// selective_scan16.hip -- fused selective scan, forward, N = 16, on gfx950.
//
// The same operation as selective_scan.hip (the Mamba-style instance of the
// affine recurrence, Sec. 1 and Sec. 3.1; chunk composition Eq. (7)):
//   a_{t,n} = exp(delta_t A_n),  u_{t,n} = delta_t B_{t,n} x_t,
//   h_{t,n} = a_{t,n} h_{t-1,n} + u_{t,n},
//   y_t     = sum_n C_{t,n} h_{t,n} + Dskip x_t,
// for the state size of Mamba (N = 16), laid out so that the machine is full
// at Mamba shapes.  One lane owns ONE state of one (b,d) row and walks the
// whole sequence; a row is a 16-lane DPP row, a wavefront holds 4 rows and a
// workgroup 16 rows of one batch.  At B=8, D=1536 that is 3072 wavefronts,
// three per SIMD, all doing the same work, so every SIMD has other
// wavefronts to issue from while one waits, and none is left with extra work.
//
// Per step a lane issues exactly the method's work: delta*A*log2e, exp2,
// (delta*x)*B, the state FMA and C*h -- four VALU operations and one
// transcendental.  The per-row operands cost nothing per step:
//   * delta and delta*x live in registers in a transposed layout: in a
//     super-tile of 16*V steps (V = 16/sizeof(IN)), lane m of a row holds
//     steps V*m .. V*m+V-1 (one 16-byte load per lane), and each step takes
//     its value from lane m with a row_newbcast DPP operand of the multiply,
//     i.e. for free;
//   * B_{t,n} and C_{t,n} are shared by the 16 rows of the workgroup: the
//     workgroup widens each 32-step tile once into LDS (three rotating
//     buffers, one barrier per tile), transposed to [n][t] so that a lane
//     reads its state's four steps with one 16-byte LDS read;
//   * the 16 partials C_{t,n} h_{t,n} of a row meet in a per-wavefront LDS
//     transpose and are summed one tile later: lane n adds 8 states over 4
//     steps, the two halves of the row meet through a row_ror:8 DPP add, and
//     the first 8 lanes add Dskip*x and store y (16-byte stores along t).
// All global loads go through buffer resources and run ahead of use: a
// super-tile of delta/x, two tiles of B/C; lanes past the end read zeros or
// are masked.  There is no carry between workgroups: each workgroup walks
// its rows over the whole sequence.
//
// Narrow shapes (too few rows to give every SIMD a wavefront) split each row
// into segments instead, composed with Eq. (7) in three launches that need no
// memory beyond y, in one of two forms; plan_n16 below prices these choices,
// and the quad layout of selective_scan_quad.hip, per call.
// Records form: (1) each segment but the last walks from a zero state (the
// first from h0) and records its end state U and the product P of its a_t,
// formed as exp(A * the segment's sum of delta); (2) a fold turns these into
// each segment's initial state, h_in(s+1) = P_s h_in(s) + U_s; (3) every
// segment walks from its initial state and stores y.  The records of segment
// s live in y's first 32 words of segment s+1 (P in 16, U in 16; the fold
// leaves h_in in the first 16), which launch (3) reads before it overwrites
// them with y.
// Correction form (fp32 y): (1) every segment walks from a
// zero state (the first from h0), stores y except in its first super-tile,
// and records P and U as above (the last segment its P beside the records
// of its own first words, its U in h_last); (2) the fold composes them and
// corrects h_last; (3) each later segment walks again from its initial
// state, rewriting y, until the part of every state carried in from the
// segment's start has faded against the segment's own terms.  By Eq. (5)
// the state is that carried part, P_t h_in, plus the walk from zero, so y
// beyond that point already holds the result to within 2^-26 of its
// magnitude; with the decay of Mamba-like parameters the third launch walks
// a small part of each segment, and the first runs every segment at once.
#include <stdlib.h>

#include <type_traits>

#include "selective_common.h"

namespace sw {

namespace {

constexpr int R16_N = 16;                   // states per row = lanes per DPP row
constexpr int R16_WAVES = 4;                // wavefronts per workgroup
constexpr int R16_RPW = 4;                  // rows per wavefront
constexpr int R16_ROWS = R16_WAVES * R16_RPW;
constexpr int R16_T = 32;                   // steps per tile
constexpr int R16_NB = R16_T / 4;           // 4-step blocks per tile
constexpr int R16_TS = R16_T + 4;           // LDS stride of one state's B (or C) tile row
constexpr int R16_NBUF = 3;                 // B/C tile buffers
constexpr int R16_PRS = R16_N * R16_TS + 32;  // partials: row stride (rows 32 banks apart)
constexpr int R16_LA = 2;                   // read-ahead, in 4-step blocks
constexpr int R16_NS = 4;                   // rotating operand sets
constexpr float R16_LOG2E = 1.4426950408889634f;
// A byte offset past the end of every buffer resource of the kernel (their
// sizes stay below 2^31 - 16): a load there returns zeros and moves no
// memory.  The super-tile of delta and x run ahead of the walk takes it for
// steps past the segment, so that no row reads the start of the next one
// (6% of those bytes at L = 2048 in bf16).  The tiles of B, C and of x for
// the D skip run ahead too, but only a tile, and mostly hit L2.
constexpr int32_t R16_OOB = 0x7FFFFFF0;
static_assert(R16_NB == 8 && R16_NB % R16_NS == 0 && R16_LA < R16_NS,
              "operand sets must rotate over a tile");

struct R16Smem {
  float bc[R16_NBUF][2][R16_N * R16_TS];     // [buf][B, C][n * TS + t]
  float p[R16_WAVES][R16_RPW * R16_PRS];     // per wavefront: [row][n * TS + t]
  int vote[R16_WAVES];                       // correction walk: wavefronts not yet done
};

// Value of `v` in lane M of this lane's 16-lane row.
template <int M>
__device__ __forceinline__ float row_bcast(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x150 + M, 0xf, 0xf,
                                         false));
}

// Value of `v` in lane n ^ 8 of this lane's 16-lane row (rotate by 8).
__device__ __forceinline__ float row_ror8(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xf, 0xf, false));
}

__device__ __forceinline__ void wg_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ void wave_order() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// B and C of one lane's state for one 4-step block.
struct R16Ops {
  float4 b, c;
};

// Segment modes of the kernel (see the top of the file).
//   R16_SEG_ENDS, R16_SEG_FWD: launches (1) and (3) of the records form;
//   R16_SEG_ALL, R16_SEG_CORR: launches (1) and (3) of the correction form.
//   R16_STATES: a whole-row walk that writes only the states (the 8-step
//   checkpoints and h_last), for a backward call without them.
enum : int {
  R16_WHOLE = 0,
  R16_SEG_ENDS = 1,
  R16_SEG_FWD = 2,
  R16_SEG_ALL = 3,
  R16_SEG_CORR = 4,
  R16_STATES = 5
};
constexpr int R16_MAX_SEG = 16;  // segments per row at most
// The correction walk of a segment stops once, for every state of its
// workgroup, the part of the state carried in from the segment's start,
// P_t h_in (P_t the product of the a since the start), is at most this
// fraction of the magnitude m_t of the segment's own terms (the sum of their
// absolute values, tracked by the walk).  Both P_t |h_in| and every later
// carried part shrink or grow by the same factors |a| as m_t's terms, so
// from then on the part left out is at most R16_CORR_EPS times the
// magnitude of the state, and of y (an fp32 walk rounds at 2^-24 of it).
constexpr float R16_CORR_EPS = 1.4901161193847656e-08f;  // 2^-26

// The record words of the segment starting at step t of a row, in y's memory
// (fp32 or bf16 elements; t is a multiple of 64, so the words are aligned).
__device__ __forceinline__ float* seg_words(void* yv, bool ybf, int64_t row, int64_t L,
                                            int64_t t) {
  return ybf ? reinterpret_cast<float*>(static_cast<uint16_t*>(yv) + row * L + t)
             : static_cast<float*>(yv) + row * L + t;
}

// OPT: the optional Mamba-block inputs (flags, z, delta bias) are read;
// without it the kernel is the plain form (an initial state is always taken).
// CK: the state at every 8-step boundary goes to ck, laid out as
// (B*D, nT8, 16), for the backward pass.
// SEG: R16_WHOLE walks whole rows; R16_SEG_ENDS and R16_SEG_FWD are launches
// (1) and (3) of the segmented form, whose workgroups are (row block,
// segment) pairs, logical workgroup = row block * segments of the launch +
// segment (the logical order is spread over the XCDs in contiguous ranges);
// a row has nseg segments of Lseg steps, the last one taking the rest
// (shorter than Lseg, or up to a super-tile longer).
template <typename IN, bool OPT, bool CK, int SEG>
__global__ __launch_bounds__(256) void selective_row16_kernel(
    const IN* __restrict__ x, const IN* __restrict__ delta, const float* __restrict__ A,
    const IN* __restrict__ Bm, const IN* __restrict__ Cm, const float* __restrict__ Dskip,
    const IN* __restrict__ z, const float* __restrict__ dbias, const float* __restrict__ h0,
    void* __restrict__ yv, float* __restrict__ h_last, int64_t D, int64_t L, int64_t ndb,
    uint32_t flags_in, float* __restrict__ ck, int64_t nT8, float* __restrict__ s_out,
    int64_t nseg, int64_t Lseg) {
  constexpr bool WHOLE = SEG == R16_WHOLE || SEG == R16_STATES;  // one walk per row
  static_assert(!(CK && !WHOLE), "checkpoints are written by whole-row walks only");
  constexpr bool ENDS = SEG == R16_SEG_ENDS;  // no y: the segment's P and end state
  constexpr bool NOY = ENDS || SEG == R16_STATES;  // no C, no y
  constexpr bool ALL = SEG == R16_SEG_ALL;    // y from a zero state, and the segment's records
  constexpr bool CORR = SEG == R16_SEG_CORR;  // the walk from the composed initial state
  constexpr bool DSUM = ENDS || ALL || CORR;  // sum of delta over the segment
  constexpr int ES = (int)sizeof(IN);
  const uint32_t flags = OPT ? flags_in : 0u;
  constexpr int V = 16 / ES;              // steps a lane holds of a super-tile
  constexpr int ST = R16_N * V;           // steps per super-tile
  constexpr int TPS = ST / R16_T;         // tiles per super-tile
  static_assert(TPS * R16_T == ST, "a super-tile is a whole number of tiles");
  __shared__ __align__(16) R16Smem sm;

  const int tid = threadIdx.x;
  const int w = tid / 64, lane = tid % 64;
  const int r = lane / R16_N, n = lane % R16_N;
  // segment of this workgroup (launch (1) of the records form covers
  // segments 0 .. nseg-2, launch (3) of the correction form 1 .. nseg-1)
  const int64_t nsl = (ENDS || CORR) ? nseg - 1 : nseg;
  const int64_t bid = xcd_contiguous(blockIdx.x, gridDim.x);
  const int64_t sg = !WHOLE ? bid % nsl + (CORR ? 1 : 0) : 0;
  const int64_t rblk = !WHOLE ? bid / nsl : bid;
  const int64_t ts = !WHOLE ? sg * Lseg : 0;  // first step of the segment
  const int64_t Ls = !WHOLE ? (sg == nseg - 1 ? L - ts : Lseg) : L;  // its steps
  const int32_t Ls32 = (int32_t)Ls;  // below 2^31 / 16 (row16_fits)
  const int64_t b = rblk / ndb;
  const int64_t d0 = (rblk - b * ndb) * R16_ROWS;
  const int64_t d = d0 + R16_RPW * w + r;
  const bool dok = d < D;
  const int64_t dcl = dok ? d : D - 1;  // rows past D compute a copy of row D-1, never stored
  const int64_t rows = imin(R16_ROWS, D - d0);
  const int64_t row0 = b * D + d0;

  // resources start at the segment's first step (row strides stay L)
  const uint32_t rows_bytes = (uint32_t)((rows * L - ts) * ES);
  const uint32_t bc_bytes = (uint32_t)((L - ts) * R16_N * ES);
  const __amdgpu_buffer_rsrc_t rx = buffer_rsrc(x + row0 * L + ts, rows_bytes);
  const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(delta + row0 * L + ts, rows_bytes);
  const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(Bm + (b * L + ts) * R16_N, bc_bytes);
  const __amdgpu_buffer_rsrc_t rc = buffer_rsrc(Cm + (b * L + ts) * R16_N, bc_bytes);
  // the gate's input; without a gate (OPT set) the same loads read x (cached),
  // so that every path of one instantiation issues the same loads
  const __amdgpu_buffer_rsrc_t rz =
      buffer_rsrc(((flags & SEL_GATED) ? z : x) + row0 * L + ts, rows_bytes);
  const int32_t lrow = (int32_t)((dcl - d0) * L * ES);  // byte offset of this lane's row

  const float Al = A[dcl * R16_N + n] * R16_LOG2E;
  const float dsk = Dskip ? Dskip[dcl] : 0.0f;
  const float dbv = (OPT && dbias) ? dbias[dcl] : 0.0f;
  const bool ybf = (flags & SEL_Y_BF16) != 0;
  float h = (h0 && sg == 0) ? h0[(b * D + dcl) * R16_N + n] : 0.0f;
  if constexpr (SEG == R16_SEG_FWD || CORR) {
    // the initial state the fold left in this segment's first words of y
    if (sg > 0) h = seg_words(yv, ybf, b * D + dcl, L, ts)[n];
  }
  // CORR: the initial state, and the magnitude of the segment's own terms
  const float hin = h;
  float mag = 0.0f;
  // ENDS: this lane's share of the sum of delta over the segment; the product
  // of the segment's a_t is exp2(Al * that sum over the row's 16 lanes)
  float dsum = 0.0f;

  const int64_t nsup = (Ls + ST - 1) / ST;
  const int64_t ntile = nsup * TPS;  // tiles past L are identity steps, never stored

  // ---- B/C staging: thread tid widens steps tt = tid/8 of a tile, states
  // 2*(tid%8) and 2*(tid%8)+1, from one B pair and one C pair.
  const int stt = tid / 8, sn = 2 * (tid % 8);
  RawVec<IN, 2> sbr[2], scr[2];  // raw pairs of tiles kt+1 and kt+2 (by tile parity)
  auto fetch_bc = [&](RawVec<IN, 2>& rbv, RawVec<IN, 2>& rcv, int64_t kt) {
    const int32_t off = (int32_t)(((kt * R16_T + stt) * R16_N + sn) * ES);
    rbv.load_buf(rb, off);
    if constexpr (!NOY) rcv.load_buf(rc, off);  // NOY: C is not read
  };
  auto stage_bc = [&](const RawVec<IN, 2>& rbv, const RawVec<IN, 2>& rcv, int buf) {
    float* bb = &sm.bc[buf][0][sn * R16_TS + stt];
    float* cc = &sm.bc[buf][1][sn * R16_TS + stt];
    bb[0] = rbv.get(0);
    bb[R16_TS] = rbv.get(1);
    if constexpr (!NOY) {
      cc[0] = rcv.get(0);
      cc[R16_TS] = rcv.get(1);
    }
  };

  // ---- delta / x of a super-tile: this lane's V steps starting at V*n
  RawVec<IN, V> dlr, xr;  // raw bits of the next super-tile
  float dl[V], dx[V];     // delta and delta*x of the current one
  auto fetch_dx = [&](int64_t sup) {
    // Ls is a multiple of V: a lane's V steps are all in or all out
    const int32_t t = (int32_t)(sup * ST) + V * n;
    const int32_t off = t < Ls32 ? lrow + t * ES : R16_OOB;
    // delta is read once (non-temporal); x is read again for the y of its
    // tiles (fetch_yx), so this read keeps the default policy
    dlr.template load_buf<SW_NT>(rd, off);
    xr.load_buf(rx, off);
  };
  auto widen_dx = [&](int64_t sup) {
    // steps past the segment are identity steps (a = 1, u = 0): the loads
    // there returned zeros (fetch_dx), which is that already, unless the
    // options turn delta = 0 into something else; Ls is a multiple of V, so
    // a lane's V steps are all inside or all past
    const bool past = OPT && (int32_t)(sup * ST) + V * n >= Ls32;
#pragma unroll
    for (int k = 0; k < V; ++k) {
      float dv = dlr.get(k), xv = xr.get(k);
      if constexpr (OPT) {
        dv += dbv;
        if (flags & SEL_SOFTPLUS) dv = softplus_f32(dv);
        if (past) dv = xv = 0.0f;
      }
      dl[k] = dv;
      dx[k] = dv * xv;
      if constexpr (DSUM) dsum += dv;
    }
  };

  // ---- y: the 16 lanes of a row split the reduce of a tile: lane n sums
  // states 8*(n/8) .. +7 over steps 4*(n%8) .. +3 with 16-byte LDS reads,
  // the two halves meet through a row_ror:8 DPP add, and lanes n < 8 store.
  const int rq = n % 8, rh = n / 8;
  RawVec<IN, 4> yxr, yzr;  // raw x and z of those four steps, for the tile awaiting its reduce
  auto fetch_yx = [&](int64_t kt) {
    if constexpr (NOY) return;
    const int32_t off = lrow + (int32_t)((kt * R16_T + 4 * rq) * ES);
    yxr.template load_buf<SW_NT>(rx, off);  // the last read of x
    if constexpr (OPT) yzr.template load_buf<SW_NT>(rz, off);
  };
  float* const p_w = &sm.p[w][r * R16_PRS + n * R16_TS];
  const float* const p_r = &sm.p[w][r * R16_PRS + 8 * rh * R16_TS + 4 * rq];
  // y (and, OPT, y before the output gate, for the backward of a gated call)
  // leave through buffer resources over the workgroup's rows from the
  // segment's start: a 32-bit offset per lane, and lanes with nothing to
  // store aim at the resource's end, where the hardware drops the store.
  // Sizes fit 32 bits: 16 rows of L < 2^26 steps of at most 4 bytes.  Both
  // are written once, with the non-temporal policy.
  const uint32_t ys = ybf ? 2u : 4u;
  const uint32_t y_bytes = (uint32_t)((rows * L - ts) * ys);
  const __amdgpu_buffer_rsrc_t ry =
      ybf ? buffer_rsrc(static_cast<uint16_t*>(yv) + row0 * L + ts, y_bytes)
          : buffer_rsrc(static_cast<float*>(yv) + row0 * L + ts, y_bytes);
  const uint32_t y_lrow = (uint32_t)((dcl - d0) * L) * ys;
  const uint32_t s_bytes = (uint32_t)((rows * L - ts) * 4);
  const __amdgpu_buffer_rsrc_t rs =
      buffer_rsrc((OPT && s_out) ? s_out + row0 * L + ts : static_cast<float*>(yv), s_bytes);
  const uint32_t s_lrow = (uint32_t)((dcl - d0) * L) * 4u;

  auto read_partials = [&](float4 (&pr)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) pr[i] = *reinterpret_cast<const float4*>(p_r + i * R16_TS);
  };
  auto finish_reduce = [&](int64_t kt, const float4 (&pr)[8], const float (&yx)[4],
                           const float (&gt)[4]) {
    float s4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      s4[0] += pr[i].x;
      s4[1] += pr[i].y;
      s4[2] += pr[i].z;
      s4[3] += pr[i].w;
    }
    // add the other half of the row (lane n ^ 8), then Dskip*x, then the gate
#pragma unroll
    for (int q = 0; q < 4; ++q) s4[q] = __builtin_fmaf(dsk, yx[q], s4[q] + row_ror8(s4[q]));
    const int32_t t = (int32_t)(kt * R16_T) + 4 * rq;
    const bool mine = dok && rh == 0 && t < Ls32;
    // ALL: the first super-tile of every segment but the first holds the
    // records until the correction walk writes its y
    const bool skip = ALL && sg > 0 && t < ST;
    if constexpr (OPT) {
      if (s_out) {
        const uint32_t so = mine ? s_lrow + 4u * (uint32_t)t : s_bytes;
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(sw_u32x4, make_float4(s4[0], s4[1], s4[2], s4[3])), rs, (int)so,
            0, SW_NT);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) s4[q] *= gt[q];
    const uint32_t yo = (mine && !skip) ? y_lrow + ys * (uint32_t)t : y_bytes;
    if (ybf)
      __builtin_amdgcn_raw_buffer_store_b64(
          __builtin_bit_cast(sw_u32x2, make_uint2(bf16x2_rne(s4[0], s4[1]), bf16x2_rne(s4[2], s4[3]))),
          ry, (int)yo, 0, SW_NT);
    else
      __builtin_amdgcn_raw_buffer_store_b128(
          __builtin_bit_cast(sw_u32x4, make_float4(s4[0], s4[1], s4[2], s4[3])), ry, (int)yo, 0,
          SW_NT);
  };

  auto read_ops = [&](R16Ops& o, int buf, int bi) {
    o.b = *reinterpret_cast<const float4*>(&sm.bc[buf][0][n * R16_TS + 4 * bi]);
    if constexpr (!NOY) o.c = *reinterpret_cast<const float4*>(&sm.bc[buf][1][n * R16_TS + 4 * bi]);
  };

  // ---- prologue: delta/x of super-tile 0, B/C of tiles 0..2, y-x of tile 0
  fetch_dx(0);
  fetch_bc(sbr[0], scr[0], 0);
  fetch_bc(sbr[1], scr[1], 1);
  stage_bc(sbr[0], scr[0], 0);
  fetch_bc(sbr[0], scr[0], 2);
  fetch_yx(0);
  wg_barrier();
  R16Ops ops[R16_NS];
#pragma unroll
  for (int i = 0; i < R16_LA; ++i) read_ops(ops[i], 0, i);

  float yx_prev[4] = {0.f, 0.f, 0.f, 0.f};  // x of the tile awaiting its reduce
  float gt_prev[4] = {1.f, 1.f, 1.f, 1.f};  // ... and its output gate
  int buf = 0;                             // B/C buffer of the tile being computed

  // One tile: stage B/C of tile kt+1, issue the reads of tile kt-1's
  // partials, wait for the workgroup, then compute the 8 blocks with the
  // operands of block i+LA read ahead (into tile kt+1's buffer at the end).
  auto tile = [&](int64_t kt, auto ttc) {
    constexpr int TT = decltype(ttc)::value;  // tile within the super-tile
    const int nbuf = buf == R16_NBUF - 1 ? 0 : buf + 1;
    const bool has_next = kt + 1 < ntile;
    stage_bc(sbr[(TT + 1) & 1], scr[(TT + 1) & 1], nbuf);
    fetch_bc(sbr[(TT + 1) & 1], scr[(TT + 1) & 1], kt + 3);
    float yx[4], gt[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      yx[q] = yxr.get(q);
      gt[q] = (OPT && (flags & SEL_GATED)) ? silu_f32(yzr.get(q)) : 1.0f;
    }
    fetch_yx(kt + 1);
    wg_barrier();
    // this wavefront's own partials: after the barrier, so that the barrier
    // only drains the staging writes
    float4 pr[8];
    if (!NOY && kt > 0) read_partials(pr);
#pragma unroll
    for (int bi = 0; bi < R16_NB; ++bi) {
      const int nb = bi + R16_LA;
      if (nb < R16_NB)
        read_ops(ops[nb % R16_NS], buf, nb);
      else if (has_next)
        read_ops(ops[nb % R16_NS], nbuf, nb - R16_NB);
      if constexpr (CK) {
        // the state before step kt*T + 4*bi; rows past D write the same
        // values as row D-1 to row D-1's slots
        const int64_t t8 = (kt * R16_T + 4 * bi) / 8;
        if ((bi & 1) == 0 && t8 < nT8) ck[((b * D + dcl) * nT8 + t8) * R16_N + n] = h;
      }
      const R16Ops& o = ops[bi % R16_NS];
      const float bq[4] = {o.b.x, o.b.y, o.b.z, o.b.w};
      const float cq[4] = {o.c.x, o.c.y, o.c.z, o.c.w};
      float p4[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        constexpr int S0 = TT * R16_T;  // step of the super-tile at block 0
        const int s = S0 + 4 * bi + q;
        float dlv, dxv;
        // the source lane and register are compile-time constants
        switch (s / V) {
#define SW_R16_CASE(M)             \
  case M:                          \
    dlv = row_bcast<M>(dl[s % V]); \
    dxv = row_bcast<M>(dx[s % V]); \
    break;
          SW_R16_CASE(0) SW_R16_CASE(1) SW_R16_CASE(2) SW_R16_CASE(3)
          SW_R16_CASE(4) SW_R16_CASE(5) SW_R16_CASE(6) SW_R16_CASE(7)
          SW_R16_CASE(8) SW_R16_CASE(9) SW_R16_CASE(10) SW_R16_CASE(11)
          SW_R16_CASE(12) SW_R16_CASE(13) SW_R16_CASE(14) SW_R16_CASE(15)
#undef SW_R16_CASE
          default:
            dlv = dxv = 0.0f;
        }
        const float a = __builtin_amdgcn_exp2f(dlv * Al);
        const float u = dxv * bq[q];
        h = __builtin_fmaf(a, h, u);
        if constexpr (CORR) mag = __builtin_fmaf(a, mag, __builtin_fabsf(u));
        if constexpr (NOY) {
          p4[q] = 0.0f;
        } else {
          p4[q] = cq[q] * h;
        }
      }
      if constexpr (!NOY) {
        *reinterpret_cast<float4*>(p_w + 4 * bi) = make_float4(p4[0], p4[1], p4[2], p4[3]);
        if (bi == 0 && kt > 0) finish_reduce(kt - 1, pr, yx_prev, gt_prev);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      yx_prev[q] = yx[q];
      gt_prev[q] = gt[q];
    }
    buf = nbuf;
    wave_order();  // this wavefront's partials are written before its next reads
  };

  int64_t kt_end = ntile;  // tiles walked
  for (int64_t sup = 0; sup < nsup; ++sup) {
#pragma unroll
    for (int tt = 0; tt < TPS; ++tt) {
      // the delta/x registers switch to this super-tile at its first tile,
      // and the next super-tile is loaded (every super-tile, so that each
      // path has the same loads in flight)
      if (tt == 0) {
        widen_dx(sup);
        fetch_dx(sup + 1);
      }
      switch (tt) {
        case 0: tile(sup * TPS + 0, std::integral_constant<int, 0>()); break;
        case 1: tile(sup * TPS + 1, std::integral_constant<int, 1>()); break;
        case 2: if constexpr (TPS > 2) tile(sup * TPS + 2, std::integral_constant<int, 2>()); break;
        case 3: if constexpr (TPS > 3) tile(sup * TPS + 3, std::integral_constant<int, 3>()); break;
        default: break;
      }
    }
    if constexpr (CORR) {
      // the carried part of each state, P h_in with P = exp2(A log2e * the
      // row's sum of delta so far), against the walk's own magnitude; the
      // workgroup stops together (its wavefronts share the B/C staging)
      float srow = dsum;
#pragma unroll
      for (int mm = 8; mm >= 1; mm /= 2) srow += __shfl_xor(srow, mm, R16_N);
      const float carried = __builtin_amdgcn_exp2f(Al * srow) * hin;
      const bool done = !dok || __builtin_fabsf(carried) <= R16_CORR_EPS * mag;
      const uint64_t open = __builtin_amdgcn_ballot_w64(!done);
      if (lane == 0) sm.vote[w] = open != 0;
      wg_barrier();
      const bool stop = (sm.vote[0] | sm.vote[1] | sm.vote[2] | sm.vote[3]) == 0;
      if (stop) {
        kt_end = (sup + 1) * TPS;
        break;
      }
    }
  }
  if constexpr (ENDS) {
    // the records of this segment, in the first words of the next one
#pragma unroll
    for (int m = 8; m >= 1; m /= 2) dsum += __shfl_xor(dsum, m, R16_N);
    if (dok) {
      float* wd = seg_words(yv, ybf, b * D + d, L, ts + Ls);
      wd[n] = __builtin_amdgcn_exp2f(Al * dsum);
      wd[R16_N + n] = h;
    }
  } else if constexpr (SEG == R16_STATES) {
    if (h_last && dok) h_last[(b * D + d) * R16_N + n] = h;
  } else {
    float4 pr[8];
    read_partials(pr);
    finish_reduce(kt_end - 1, pr, yx_prev, gt_prev);
    if constexpr (ALL) {
      // the records of this segment: its P and end state in the first words
      // of the next segment; the last segment's P beside the records there,
      // its end state in h_last (the fold composes both)
#pragma unroll
      for (int mm = 8; mm >= 1; mm /= 2) dsum += __shfl_xor(dsum, mm, R16_N);
      if (dok) {
        const float P = __builtin_amdgcn_exp2f(Al * dsum);
        if (sg < nseg - 1) {
          float* wd = seg_words(yv, false, b * D + d, L, ts + Ls);
          wd[n] = P;
          wd[R16_N + n] = h;
        } else {
          seg_words(yv, false, b * D + d, L, ts)[2 * R16_N + n] = P;
        }
      }
    }
    if constexpr (!CORR) {
      if (h_last && dok && (WHOLE || sg == nseg - 1))
        h_last[(b * D + d) * R16_N + n] = h;
    }
  }
}

// Launch (2) of the segmented form: one lane per (row, state) walks the
// segments' records in order and leaves each segment's initial state in its
// first words: h_in(1) = U_0 (segment 0 started from h0), then
// h_in(s+1) = P_s h_in(s) + U_s.
__global__ __launch_bounds__(256) void row16_fold_kernel(void* __restrict__ yv, bool ybf,
                                                         int64_t R, int64_t L, int64_t nseg,
                                                         int64_t Lseg) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= R * R16_N) return;
  const int64_t row = i / R16_N;
  const int n = (int)(i % R16_N);
  // all records first (independent loads in flight together), then the fold
  float P[R16_MAX_SEG], U[R16_MAX_SEG];
#pragma unroll
  for (int sgi = 1; sgi < R16_MAX_SEG; ++sgi) {
    if (sgi < nseg) {
      const float* wd = seg_words(yv, ybf, row, L, sgi * Lseg);
      P[sgi] = wd[n];
      U[sgi] = wd[R16_N + n];
    }
  }
  float h = 0.0f;
#pragma unroll
  for (int sgi = 1; sgi < R16_MAX_SEG; ++sgi) {
    if (sgi < nseg) {
      h = sgi == 1 ? U[sgi] : __builtin_fmaf(P[sgi], h, U[sgi]);
      seg_words(yv, ybf, row, L, sgi * Lseg)[n] = h;
    }
  }
}

// Launch (2) of the correction form: one lane per (row, state) composes the
// segments' records in order, h_in(1) = U_0 (segment 0 started from h0),
// h_in(s+1) = P_s h_in(s) + U_s, leaves h_in(s) in the first words of segment
// s, and corrects the final state: h_last = P_last h_in(last) + U_last.
__global__ __launch_bounds__(256) void row16_fold_corr_kernel(float* __restrict__ y,
                                                              float* __restrict__ h_last,
                                                              int64_t R, int64_t L, int64_t nseg,
                                                              int64_t Lseg) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= R * R16_N) return;
  const int64_t row = i / R16_N;
  const int n = (int)(i % R16_N);
  float P[R16_MAX_SEG], U[R16_MAX_SEG];
#pragma unroll
  for (int sgi = 1; sgi < R16_MAX_SEG; ++sgi) {
    if (sgi < nseg) {
      const float* wd = seg_words(y, false, row, L, sgi * Lseg);
      P[sgi] = wd[n];  // of segment sgi - 1
      U[sgi] = wd[R16_N + n];
    }
  }
  float h = 0.0f;
#pragma unroll
  for (int sgi = 1; sgi < R16_MAX_SEG; ++sgi) {
    if (sgi < nseg) {
      h = sgi == 1 ? U[sgi] : __builtin_fmaf(P[sgi], h, U[sgi]);
      seg_words(y, false, row, L, sgi * Lseg)[n] = h;
    }
  }
  if (h_last) {
    const float Pl = seg_words(y, false, row, L, (nseg - 1) * Lseg)[2 * R16_N + n];
    h_last[row * R16_N + n] = __builtin_fmaf(Pl, h, h_last[row * R16_N + n]);
  }
}

}  // namespace

// The fold of the correction form, shared with the quad layout
// (selective_scan_quad.hip), which keeps its records in the same places.
void launch_fold_corr(float* y, float* h_last, int64_t R, int64_t L, int64_t nseg, int64_t Lseg,
                      hipStream_t s) {
  const int64_t lanes = R * R16_N;
  hipLaunchKernelGGL(row16_fold_corr_kernel, dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0,
                     s, y, h_last, R, L, nseg, Lseg);
}

template <typename IN>
bool quad_fits(const SelArgs& a);
template <typename IN>
int launch_quad(const SelArgs& a, int64_t nseg, int64_t Lseg, hipStream_t s);

// True when the N = 16 layout can take the call: vector-aligned rows, and
// every byte offset of a workgroup (including loads run ahead past the end)
// below 2^31.
bool row16_fits(int64_t D, int64_t N, int64_t L, size_t es) {
  if (N != R16_N) return false;
  const int64_t vstep = 16 / (int64_t)es;
  if (L % vstep != 0) return false;
  const int64_t pad = 4 * R16_N * vstep;
  return R16_ROWS * (L + pad) * (int64_t)es < ((int64_t)1 << 31) &&
         (L + pad) * R16_N * (int64_t)es < ((int64_t)1 << 31) && D > 0;
}

// ---- which layout, how many segments and which form an N = 16 call takes
//
// The candidates: the 16-lane layout walking whole rows; the 16-lane layout
// with 2..16 segments per row, in the records or the correction form; the
// quad layout (four lanes per row, selective_scan_quad.hip) with 2..16
// segments, correction form.  Each is priced with a model of its launches
// and the cheapest is taken.  A launch of G workgroups on `cus` CUs runs in
// rounds: its busiest CU holds ceil(G / cus) workgroups, at most `cap` at a
// time (three of the 16-lane layout, four of the quad layout, by LDS), and a
// round with o workgroups resident per CU takes `ns[o]` per step of its walk
// -- the per-step times of each layout measured on MI355X with one to four
// workgroups per CU, fp32 inputs (the quad layout is 8% faster with bf16
// inputs; its four-per-CU time, 226 ns with every CU at four, is set at 220
// ns, what B=1, D=5120, L=65536 measures with three quarters of the CUs at
// four).  Every segment of a launch walks at once, so a launch is priced at
// its longest segment.  A correction walk is priced at the fading length of Mamba-like
// decay, 1024 steps plus one check (slower decay walks further, up to the
// whole segment: slower, never wrong); a segmented call adds 8 us for its
// fold and two more launches; the first walk of the records form (no C, no
// y) is priced at 0.85 of a walk.  Over 42 shapes (B = 1..4, D = 1280..8192,
// L = 4096..65536, fp32 and bf16 inputs) the model's choice came within 1.2%
// of the fastest measured candidate on average and 10% at worst, where
// fixed occupancy bands had been 29% and 150% off.
// SW_SS_QUAD=0 leaves the quad layout out, =1 takes it whenever the call
// allows; SW_SS_SEGMENTS=k keeps only the candidates with k segments (1:
// whole rows; the 16-lane layout unless SW_SS_QUAD=1); SW_SS_SEGFORM=1 or 2
// keeps only the records or the correction form of the 16-lane layout.
struct StepCost {
  int cap;
  float ns[5];
};
constexpr StepCost R16_COST = {3, {0.0f, 28.8f, 42.3f, 57.1f, 0.0f}};
constexpr StepCost QUAD_COST = {4, {0.0f, 98.6f, 135.8f, 171.6f, 220.0f}};
constexpr int64_t PLAN_CORR_STEPS = 1024;
constexpr double PLAN_SEG_US = 8.0;
constexpr double PLAN_ENDS_SHARE = 0.85;
constexpr int64_t QUAD_SKIP = 64;  // the quad layout's segment granularity and check interval

double launch_us(int64_t G, int64_t steps, int cus, const StepCost& c, double scale) {
  const int64_t per = (G + cus - 1) / cus;  // workgroups on the busiest CU
  const int64_t full = per / c.cap, rest = per % c.cap;
  const double ns = (double)full * c.ns[c.cap] + (rest > 0 ? c.ns[rest] : 0.0);
  return (double)steps * ns * scale * 1e-3;
}

int64_t env_i64(const char* name) {
  const char* v = getenv(name);
  return (v && *v) ? atoll(v) : -1;
}

struct N16Plan {
  bool quad = false;
  int64_t nseg = 1;  // 1: whole rows
  int64_t Lseg = 0;
  bool corr = false;
};

// Segments of the 16-lane layout for a count k: L / k rounded up to whole
// super-tiles of st steps, as many segments as that takes, the last one the
// rest; a rest shorter than a super-tile (too short for the records the
// segment before leaves in its first words) joins the segment before.  n = 0
// when k gives fewer than two.
void r16_geometry(int64_t L, int64_t st, int64_t k, int64_t* n, int64_t* Lseg) {
  *n = 0;
  if (k < 2 || k > R16_MAX_SEG || L / st < 2) return;
  const int64_t per = (L + k - 1) / k;
  *Lseg = (per + st - 1) / st * st;
  int64_t m = (L + *Lseg - 1) / *Lseg;
  if (L - (m - 1) * *Lseg < st) --m;
  if (m >= 2 && m <= R16_MAX_SEG) *n = m;
}

// Segments of the quad layout for a count k: k - 1 segments of Lseg steps (a
// multiple of QUAD_SKIP) and the last taking the rest.  Lseg is L / k rounded
// up, which leaves the last segment the shortest, unless that leaves it fewer
// than QUAD_SKIP steps (its first words hold 48 words of records); then
// rounded down (the last the longest).  Lseg < QUAD_SKIP: no such geometry.
void quad_geometry(int64_t L, int64_t k, int64_t* Lseg, int64_t* last) {
  const int64_t per = (L + k - 1) / k;
  *Lseg = (per + QUAD_SKIP - 1) / QUAD_SKIP * QUAD_SKIP;
  if (L - (k - 1) * *Lseg < QUAD_SKIP) *Lseg = (L / k) / QUAD_SKIP * QUAD_SKIP;
  *last = L - (k - 1) * *Lseg;
}

// `cus`: the compute units the launches are priced for.
template <typename IN>
N16Plan plan_n16(const SelArgs& a, int64_t ndb, int cus) {
  N16Plan best;
  if (a.ckpt) return best;  // checkpoints are written by whole-row walks
  const int64_t L = a.L, st = R16_N * (16 / (int64_t)sizeof(IN));
  const int64_t quad_env = env_i64("SW_SS_QUAD"), seg_env = env_i64("SW_SS_SEGMENTS");
  const int64_t form_env = env_i64("SW_SS_SEGFORM");
  const bool qfits = quad_fits<IN>(a);
  const bool quad_only = quad_env == 1 && qfits;
  const bool with_quad = qfits && quad_env != 0 && (seg_env < 0 || quad_only);
  const bool corr_ok = !a.y_bf16;
  const double qscale = sizeof(IN) == 2 ? 0.92 : 1.0;
  const int64_t G16 = a.B * ndb, Gq = a.B * ((a.D + 63) / 64);
  double best_us = 1e300;
  auto consider = [&](double us, bool quad, int64_t nseg, int64_t Lseg, bool corr) {
    if (us < best_us) {
      best_us = us;
      best.quad = quad;
      best.nseg = nseg;
      best.Lseg = Lseg;
      best.corr = corr;
    }
  };
  const int64_t kmin = seg_env > 0 ? (seg_env < 16 ? seg_env : 16) : 1;
  const int64_t kmax = seg_env > 0 ? kmin : 16;
  if (!quad_only) {
    if (kmin == 1) consider(launch_us(G16, L, cus, R16_COST, 1.0), false, 1, L, false);
    for (int64_t k = (kmin > 2 ? kmin : 2); k <= kmax; ++k) {
      int64_t n, Lseg;
      r16_geometry(L, st, k, &n, &Lseg);
      if (n < 2 || G16 * n >= ((int64_t)1 << 31)) continue;
      // every segment walks at once: the longest sets the launch's time
      const int64_t last = L - (n - 1) * Lseg;
      const int64_t longest = last > Lseg ? last : Lseg;
      const double first = launch_us(G16 * n, longest, cus, R16_COST, 1.0);
      if (corr_ok && form_env != 1) {
        const int64_t walk = longest < PLAN_CORR_STEPS + st ? longest : PLAN_CORR_STEPS + st;
        consider(first + launch_us(G16 * (n - 1), walk, cus, R16_COST, 1.0) + PLAN_SEG_US, false,
                 n, Lseg, true);
      }
      if (form_env != 2)
        consider(PLAN_ENDS_SHARE * launch_us(G16 * (n - 1), Lseg, cus, R16_COST, 1.0) + first +
                     PLAN_SEG_US,
                 false, n, Lseg, false);
    }
    // a forced count that gives fewer than two segments walks whole rows
    if (best_us == 1e300) consider(0.0, false, 1, L, false);
  }
  if (with_quad) {
    // a forced count is capped at one segment per QUAD_SKIP steps
    const int64_t kcap = L / QUAD_SKIP;
    if (quad_only && (kmin == 1 || (seg_env > 0 && kcap < 2)))
      consider(launch_us(Gq, L, cus, QUAD_COST, qscale), true, 1, L, false);
    const int64_t qmin = seg_env > 0 && kmin > kcap ? kcap : kmin;
    const int64_t qmax = seg_env > 0 && kmax > kcap ? kcap : kmax;
    for (int64_t k = (qmin > 2 ? qmin : 2); k <= qmax; ++k) {
      int64_t Lseg, last;
      quad_geometry(L, k, &Lseg, &last);
      if (Lseg < QUAD_SKIP) continue;
      // every segment walks at once: the longest sets the launch's time
      const int64_t longest = last > Lseg ? last : Lseg;
      const int64_t walk =
          longest < PLAN_CORR_STEPS + QUAD_SKIP ? longest : PLAN_CORR_STEPS + QUAD_SKIP;
      consider(launch_us(Gq * k, longest, cus, QUAD_COST, qscale) +
                   launch_us(Gq * (k - 1), walk, cus, QUAD_COST, qscale) + PLAN_SEG_US,
               true, k, Lseg, true);
    }
    if (quad_only && best_us == 1e300) consider(0.0, true, 1, L, false);
  }
  return best;
}

template <typename IN, bool OPT>
void launch_row16_segments(const SelArgs& a, int64_t ndb, uint32_t flags, int64_t nseg,
                           int64_t Lseg, hipStream_t s) {
  const int64_t R = a.B * a.D;
  const int64_t rblocks = a.B * ndb;
  hipLaunchKernelGGL((selective_row16_kernel<IN, OPT, false, R16_SEG_ENDS>),
                     dim3((unsigned)(rblocks * (nseg - 1))), dim3(256), 0, s,
                     static_cast<const IN*>(a.x), static_cast<const IN*>(a.delta), a.A,
                     static_cast<const IN*>(a.Bm), static_cast<const IN*>(a.Cm), a.Dskip,
                     static_cast<const IN*>(a.z), a.delta_bias, a.h0, a.y, nullptr, a.D, a.L,
                     ndb, flags, nullptr, (int64_t)0, nullptr, nseg, Lseg);
  const int64_t lanes = R * R16_N;
  hipLaunchKernelGGL(row16_fold_kernel, dim3((unsigned)((lanes + 255) / 256)), dim3(256), 0, s,
                     a.y, a.y_bf16, R, a.L, nseg, Lseg);
  hipLaunchKernelGGL((selective_row16_kernel<IN, OPT, false, R16_SEG_FWD>),
                     dim3((unsigned)(rblocks * nseg)), dim3(256), 0, s,
                     static_cast<const IN*>(a.x), static_cast<const IN*>(a.delta), a.A,
                     static_cast<const IN*>(a.Bm), static_cast<const IN*>(a.Cm), a.Dskip,
                     static_cast<const IN*>(a.z), a.delta_bias, a.h0, a.y, a.h_last, a.D, a.L,
                     ndb, flags, nullptr, (int64_t)0, a.s_out, nseg, Lseg);
}

// The correction form: (1) every segment walks from a zero state (the first
// from h0), stores y (all but its first super-tile) and records its P and
// end state; (2) the fold composes the records into each segment's initial
// state and corrects h_last; (3) every segment but the first walks again from
// its initial state, rewriting y, until the part carried in from the start
// is negligible against the segment's own terms (R16_CORR_EPS).
template <typename IN, bool OPT>
void launch_row16_corr(const SelArgs& a, int64_t ndb, uint32_t flags, int64_t nseg,
                       int64_t Lseg, hipStream_t s) {
  const int64_t R = a.B * a.D;
  const int64_t rblocks = a.B * ndb;
  hipLaunchKernelGGL((selective_row16_kernel<IN, OPT, false, R16_SEG_ALL>),
                     dim3((unsigned)(rblocks * nseg)), dim3(256), 0, s,
                     static_cast<const IN*>(a.x), static_cast<const IN*>(a.delta), a.A,
                     static_cast<const IN*>(a.Bm), static_cast<const IN*>(a.Cm), a.Dskip,
                     static_cast<const IN*>(a.z), a.delta_bias, a.h0, a.y, a.h_last, a.D, a.L,
                     ndb, flags, nullptr, (int64_t)0, a.s_out, nseg, Lseg);
  launch_fold_corr(static_cast<float*>(a.y), a.h_last, R, a.L, nseg, Lseg, s);
  hipLaunchKernelGGL((selective_row16_kernel<IN, OPT, false, R16_SEG_CORR>),
                     dim3((unsigned)(rblocks * (nseg - 1))), dim3(256), 0, s,
                     static_cast<const IN*>(a.x), static_cast<const IN*>(a.delta), a.A,
                     static_cast<const IN*>(a.Bm), static_cast<const IN*>(a.Cm), a.Dskip,
                     static_cast<const IN*>(a.z), a.delta_bias, a.h0, a.y, nullptr, a.D, a.L,
                     ndb, flags, nullptr, (int64_t)0, a.s_out, nseg, Lseg);
}

template <typename IN>
int launch_row16(const SelArgs& a, hipStream_t s) {
  const bool opt = a.z || a.delta_bias || a.softplus || a.y_bf16 || a.s_out;
  const int64_t ndb = (a.D + R16_ROWS - 1) / R16_ROWS;
  const int64_t grid = a.B * ndb;
  if (grid >= ((int64_t)1 << 31))
    return fail(SW_ERR_UNSUPPORTED, "%lld workgroups exceed the grid range", (long long)grid);
  int cus = 0;
  if (device_cus(&cus) != SW_OK) cus = 256;  // a forced choice needs no device facts
  const N16Plan p = plan_n16<IN>(a, ndb, cus);
  if (p.quad) return launch_quad<IN>(a, p.nseg, p.Lseg, s);
  const uint32_t flags = (a.softplus ? SEL_SOFTPLUS : 0u) | (a.y_bf16 ? SEL_Y_BF16 : 0u) |
                         (a.z ? SEL_GATED : 0u);
  const int64_t nseg = p.nseg, Lseg = p.Lseg;
  if (nseg > 1 && p.corr) {
    if (opt)
      launch_row16_corr<IN, true>(a, ndb, flags, nseg, Lseg, s);
    else
      launch_row16_corr<IN, false>(a, ndb, flags, nseg, Lseg, s);
    note_launch("selective_row16_kernel: %lld segments of %lld steps, correction form (3 launches)",
                (long long)nseg, (long long)Lseg);
    return check_launch("selective_row16_kernel (segments, correction form)");
  }
  if (nseg > 1) {
    if (opt)
      launch_row16_segments<IN, true>(a, ndb, flags, nseg, Lseg, s);
    else
      launch_row16_segments<IN, false>(a, ndb, flags, nseg, Lseg, s);
    note_launch("selective_row16_kernel: %lld segments of %lld steps, records form (3 launches)",
                (long long)nseg, (long long)Lseg);
    return check_launch("selective_row16_kernel (segments)");
  }
  auto kern = opt ? (a.ckpt ? selective_row16_kernel<IN, true, true, R16_WHOLE>
                            : selective_row16_kernel<IN, true, false, R16_WHOLE>)
                  : (a.ckpt ? selective_row16_kernel<IN, false, true, R16_WHOLE>
                            : selective_row16_kernel<IN, false, false, R16_WHOLE>);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), 0, s, static_cast<const IN*>(a.x),
                     static_cast<const IN*>(a.delta), a.A, static_cast<const IN*>(a.Bm),
                     static_cast<const IN*>(a.Cm), a.Dskip, static_cast<const IN*>(a.z),
                     a.delta_bias, a.h0, a.y, a.h_last, a.D, a.L, ndb, flags, a.ckpt,
                     (a.L + 7) / 8, a.s_out, (int64_t)1, a.L);
  note_launch("selective_row16_kernel: whole rows");
  return check_launch("selective_row16_kernel");
}

// The states of a whole-row walk without y (R16_STATES): the 8-step
// checkpoints into a.ckpt and, if given, h_last; x, delta, B, A, h0 and the
// delta options are read, C, Dskip, z and y are not.  The call must satisfy
// row16_fits and the forward's vector-path conditions.
template <typename IN>
int launch_row16_states(const SelArgs& a, hipStream_t s) {
  const int64_t ndb = (a.D + R16_ROWS - 1) / R16_ROWS;
  const int64_t grid = a.B * ndb;
  if (grid >= ((int64_t)1 << 31))
    return fail(SW_ERR_UNSUPPORTED, "%lld workgroups exceed the grid range", (long long)grid);
  const bool opt = a.delta_bias || a.softplus;
  const uint32_t flags = a.softplus ? SEL_SOFTPLUS : 0u;
  auto kern = opt ? selective_row16_kernel<IN, true, true, R16_STATES>
                  : selective_row16_kernel<IN, false, true, R16_STATES>;
  // y is never written in this mode: x stands in for its pointer
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), 0, s, static_cast<const IN*>(a.x),
                     static_cast<const IN*>(a.delta), a.A, static_cast<const IN*>(a.Bm),
                     static_cast<const IN*>(a.Cm), a.Dskip, static_cast<const IN*>(nullptr),
                     a.delta_bias, a.h0, const_cast<void*>(a.x), a.h_last, a.D, a.L, ndb, flags,
                     a.ckpt, (a.L + 7) / 8, static_cast<float*>(nullptr), (int64_t)1, a.L);
  return check_launch("selective_row16_kernel (states)");
}

// What launch_row16 would enqueue for `a` on a part with `cus` compute units.
template <typename IN>
SelPlan plan_row16(const SelArgs& a, int cus) {
  const N16Plan p = plan_n16<IN>(a, (a.D + R16_ROWS - 1) / R16_ROWS, cus);
  SelPlan q;
  q.layout = p.quad ? 4 : 16;
  q.nseg = p.nseg;
  q.lseg = p.nseg > 1 ? p.Lseg : a.L;
  q.form = p.nseg > 1 ? (p.corr ? 2 : 1) : 0;
  return q;
}

template int launch_row16<float>(const SelArgs&, hipStream_t);
template int launch_row16<uint16_t>(const SelArgs&, hipStream_t);
template SelPlan plan_row16<float>(const SelArgs&, int);
template SelPlan plan_row16<uint16_t>(const SelArgs&, int);
template int launch_row16_states<float>(const SelArgs&, hipStream_t);
template int launch_row16_states<uint16_t>(const SelArgs&, hipStream_t);

}  // namespace sw
