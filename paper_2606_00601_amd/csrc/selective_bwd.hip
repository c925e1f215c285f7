// selective_bwd.hip -- backward of the fused selective scan on gfx950.
//
// The gradient of sum_t dy_t y_t (+ sum_n dh_last_n h_last_n) by the chain
// rule through the forward recurrence h_t = a_t h_{t-1} + u_t (Eq. (3)),
// a_{t,n} = exp(delta_t A_n), u_{t,n} = delta_t B_{t,n} x_t,
// y_t = (sum_n C_{t,n} h_{t,n} + Dskip x_t) g_t, g_t = silu(z_t) or 1.
// The adjoint lam_t = dL/dh_t obeys the same kind of recurrence run
// backwards in time, lam_t = ds_t C_t + a_{t+1} lam_{t+1} (ds_t = dy_t g_t),
// the affine pair of Eq. (6) with the order of Eq. (7) reversed.  With
// q_t = a_t h_{t-1}:
//   ddelta_t = sum_n lam (q A_n + B x_t)        dx_t = delta_t sum_n lam B + ds_t Dskip
//   dA_n    += lam q delta_t                    dB_{t,n} += lam delta_t x_t   (over d)
//   dC_{t,n} += ds_t h_t                        (over d)
//   dh0 = a_0 lam_0,  dDskip += ds x,  dz = dy s silu'(z) with s the pre-gate y.
//
// One workgroup (4 wavefronts) owns 16 (b,d) rows of one batch; lane n of a
// 16-lane row owns state n (N <= 16; states past N are identity steps).
//   1. A forward sweep over the sequence stores the state at the start of
//      every 8-step tile (a checkpoint per lane per tile, in a workspace).
//   2. A reverse sweep over the tiles: the tile's delta, delta*x, ds and
//      B, C are staged in LDS; every lane reloads its checkpoint, recomputes
//      the tile's a_t and q_t forward into registers, then walks the tile
//      backwards carrying lam.  Per step it forms four partial products:
//      lam q A and lam B (summed over n, per row and step, into ddelta and
//      dx) go to LDS; lam delta x and ds h (summed over the 16 rows, per step
//      and state, into this workgroup's share of dB and dC) are first summed
//      over the wavefront's four rows by lane-half exchanges, and only those
//      sums go to LDS.
//   3. Half of the workgroup sums the first pair per (row, step), the other
//      half adds the four wavefronts' row sums per (step, state); the shares
//      of dB / dC, dA, dDskip and ddelta_bias go to a workspace, and a second
//      kernel adds the shares in a fixed order (no atomics: the result is
//      reproducible).
// The pre-gate output s needed by dz comes from the forward kernel run
// without the gate.
#include "selective_common.h"

namespace sw {
namespace {

constexpr int BW_N = 16;                 // state lanes per row
constexpr int BW_T = 8;                  // steps per tile
constexpr int BW_TS = 8;                 // LDS stride of one [t] run (16-byte aligned)
constexpr int BW_ROWS = 16;              // (b,d) rows per workgroup
// stride of one row's [n][t] block: 8 mod 64 banks, so that the 64 lanes of a
// role-a reduce (8 rows x 8 steps) read 64 different banks
constexpr int BW_RS = BW_N * BW_TS + 8;
constexpr int BW_RING = 4;               // raw tile registers: loads run 3 tiles ahead
constexpr float BW_LOG2E = 1.4426950408889634f;

// Position of step t of state n inside its 8-step run: the two 4-step halves
// trade places for n >= 8, so that the 16 states of a row (float4 accesses)
// and the 16 x 4 (state, step) lanes of the reduces fall on 64 different banks.
__device__ __forceinline__ int swz(int n, int t) { return t ^ ((n >> 1) & 4); }

struct BwSmem {
  float rv[2][3][BW_ROWS][BW_TS];  // two tile buffers; per row and step: delta, delta*x, ds
  float bc[2][2][BW_N][BW_TS];     // two tile buffers; B, C of the tile as [n][t]
  // partials, two buffers (tile k uses k & 1): the sums of tile k+1 are read
  // while tile k's are written, so one barrier per tile orders both
  float sp[2][2][BW_ROWS * BW_RS];  // per row [n][t]: lam q A, lam B      (sum over n)
  float pw[2][4][64 * 4];           // per wavefront and lane: four row sums (rows4_sum)
};

// Sums over the four 16-lane rows of a wavefront, by the two lane-half
// exchanges of gfx950: v_permlane32_swap trades lanes 32-63 of its first
// operand with lanes 0-31 of its second, v_permlane16_swap the odd 16-lane
// rows of the first with the even rows of the second.  In: a lane's
// lam delta x (dx) and ds h (dh) at the tile's 8 steps.  Out: lane l holds,
// for state l % 16, the sums over the four rows of dx (l < 32) or dh
// (l >= 32) at steps 4 ((l / 16) & 1) + 0..3.
__device__ __forceinline__ void rows4_sum(const float (&dx)[8], const float (&dh)[8],
                                          float (&out)[4]) {
  float r[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    // lanes 0-31 get dx of lanes l and l+32, lanes 32-63 dh of l-32 and l
    const auto v = __builtin_amdgcn_permlane32_swap(__float_as_uint(dx[t]),
                                                    __float_as_uint(dh[t]), false, false);
    r[t] = __uint_as_float(v[0]) + __uint_as_float(v[1]);
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    // row 0 of the wavefront gets rows 0 + 1 of r[t], row 1 rows 0 + 1 of
    // r[t+4], rows 2 and 3 likewise from rows 2 + 3
    const auto v = __builtin_amdgcn_permlane16_swap(__float_as_uint(r[t]),
                                                    __float_as_uint(r[t + 4]), false, false);
    out[t] = __uint_as_float(v[0]) + __uint_as_float(v[1]);
  }
}

__device__ __forceinline__ float sigmoid_f32(float v) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-v * BW_LOG2E));
}

__device__ __forceinline__ void bw_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

struct BwWork {
  float* ck;       // (B*D, ntile, 16) states at tile starts
  const float* s;  // (B*D, L) pre-gate output (gated calls)
  float* dA_p;     // (B*D, 16)
  float* dD_p;     // (B*D)
  float* db_p;     // (B*D)
  float* dB_p;     // (B, G, L, 16)
  float* dC_p;     // (B, G, L, 16)
  float* trash;    // 256 floats: the target of stores a lane does not need
};

// Raw bits of one element as loaded; widened to fp32 only when used, so that
// the load is not waited for until then.
template <typename T>
__device__ __forceinline__ float widen(T r) {
  if constexpr (sizeof(T) == 4)
    return r;
  else
    return __uint_as_float((uint32_t)r << 16);
}

// One staging thread's raw inputs of one tile.  Waves 0-1 read x, delta, dy
// (and z, s) of (row, step); waves 2-3 read B, C of (step, state) through the
// same two slots r0, r1, so that every thread runs the same straight-line
// loads (their dy, z, s slots read a valid, unused element).
template <typename IN, typename DYT>
struct TileRaw {
  IN r0, r1, z;
  DYT dy;
  float s;
  bool ok;  // role a: a step of a real row inside the sequence; role b: t < L, n < N
};

// One element of type T at byte offset voff + soff of a raw buffer resource
// (zero past the resource's end).
template <typename T>
__device__ __forceinline__ T buf_ld(__amdgpu_buffer_rsrc_t r, int32_t voff, int32_t soff) {
  if constexpr (sizeof(T) == 4)
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
  else
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0));
}

// All global loads below are unconditional, from valid addresses, with the
// unwanted values replaced afterwards: the loads of the next tile then stay in
// flight across the current one instead of being waited for inside a branch.
// BUF: the loads go through raw buffer resources over the workgroup's rows
// (and its batch's B, C), so that a tile's address is a per-lane offset fixed
// for the whole kernel plus a scalar one (every offset below 2^31, checked by
// the host); without it, 64-bit addresses clamped into range.
template <typename IN, typename DYT, bool GATED, bool BUF>
__global__ __launch_bounds__(256) void selective_bwd_kernel(const BwdArgs a, const BwWork w,
                                                            int64_t G, int64_t ntile, int n0) {
  __shared__ __align__(16) BwSmem sm;
  const IN* __restrict__ X = static_cast<const IN*>(a.x);
  const IN* __restrict__ DL = static_cast<const IN*>(a.delta);
  const IN* __restrict__ BM = static_cast<const IN*>(a.Bm);
  const IN* __restrict__ CM = static_cast<const IN*>(a.Cm);
  const IN* __restrict__ Z = static_cast<const IN*>(a.z);
  const DYT* __restrict__ DY = static_cast<const DYT*>(a.dy);
  const int64_t D = a.D, L = a.L, N = a.N;

  const int tid = threadIdx.x;
  const int wv = __builtin_amdgcn_readfirstlane(tid / 64);  // wave-uniform
  const int lane = tid % 64;
  const int rr = 4 * wv + lane / 16;  // compute role: row within the workgroup
  const int n = lane % 16;            // ... and state
  const int64_t b = blockIdx.x / G;
  const int64_t g = blockIdx.x - b * G;
  const int64_t d0 = g * BW_ROWS;
  const int64_t d = d0 + rr;
  const bool dok = d < D;
  // this launch's states are n0 .. n0+15 (groups of 16 for N > 16); the
  // first group also adds the terms that do not depend on the state
  const int ns = n0 + n;  // the lane's state
  const bool nok = ns < N;
  const bool first = n0 == 0;
  const int64_t row = b * D + (dok ? d : D - 1);

  // staging / reduce roles (by wavefront): waves 0-1 own (row sr, step st),
  // waves 2-3 own (step bt, state bn)
  const bool role_a = wv < 2;
  const int sr = (tid % 128) / BW_T, st = tid % BW_T;
  const int bt = (tid % 128) / BW_N, bn = tid % BW_N;
  const int64_t sd = d0 + sr;
  const bool sdok = sd < D;
  const int64_t srow = b * D + (sdok ? sd : D - 1);

  const float Ar = a.A[(dok ? d : D - 1) * N + (nok ? ns : 0)] * (nok ? 1.0f : 0.0f);
  const float Al = Ar * BW_LOG2E;
  const float dbias = a.delta_bias ? a.delta_bias[sdok ? sd : D - 1] : 0.0f;
  const float Dsk = a.Dskip ? a.Dskip[sdok ? sd : D - 1] : 0.0f;

  // --- staging helpers -----------------------------------------------------
  const IN* __restrict__ P0 = role_a ? X : BM;
  const IN* __restrict__ P1 = role_a ? DL : CM;
  using Raw = TileRaw<IN, DYT>;
  // BUF: resources and per-lane element offsets.  Role a (and the dy, z, s
  // loads of every lane) index (row - d0) * L + t of the workgroup's rows,
  // role b (t * N + n) of the batch's B, C.
  const int64_t row0 = b * D + d0;
  const int64_t nrows = imin(BW_ROWS, D - d0);
  const int32_t ea = (int32_t)(((sdok ? sd : D - 1) - d0) * L) + st;
  const int32_t eb = bt * (int32_t)N + (n0 + bn < N ? n0 + bn : (int32_t)N - 1);
  const int32_t e01 = role_a ? ea : eb;
  const int32_t ts01 = role_a ? BW_T : BW_T * (int32_t)N;  // elements per tile
  // (built in both variants; only BUF uses them)
  const uint32_t rows_b = (uint32_t)(nrows * L * (int64_t)sizeof(IN));
  const uint32_t bc_b = (uint32_t)(L * N * (int64_t)sizeof(IN));
  const __amdgpu_buffer_rsrc_t r0s =
      buffer_rsrc(role_a ? (const void*)(X + row0 * L) : (const void*)(BM + b * L * N),
                  role_a ? rows_b : bc_b);
  const __amdgpu_buffer_rsrc_t r1s =
      buffer_rsrc(role_a ? (const void*)(DL + row0 * L) : (const void*)(CM + b * L * N),
                  role_a ? rows_b : bc_b);
  const __amdgpu_buffer_rsrc_t rdy =
      buffer_rsrc(DY + row0 * L, (uint32_t)(nrows * L * (int64_t)sizeof(DYT)));
  const __amdgpu_buffer_rsrc_t rz = buffer_rsrc(GATED ? Z + row0 * L : X, GATED ? rows_b : 0u);
  const __amdgpu_buffer_rsrc_t rs =
      buffer_rsrc(GATED ? w.s + row0 * L : w.trash, GATED ? (uint32_t)(nrows * L * 4) : 0u);
  const __amdgpu_buffer_rsrc_t rck =
      buffer_rsrc(w.ck + row0 * ntile * BW_N, (uint32_t)(nrows * ntile * BW_N * 4));
  const int32_t eck = (int32_t)(((dok ? d : D - 1) - d0) * ntile * BW_N) + n;
  const uint32_t ck_b = (uint32_t)(nrows * ntile * BW_N * 4);
  // BUF: the reduce's outputs through resources too, picked by the
  // wavefront's role: role a the workgroup's rows of ddelta, dx (and dz),
  // role b this workgroup's share of dB, dC; a lane with nothing to store
  // aims at the resource's end, where the store is dropped (and a load
  // returns zero)
  const uint32_t out_b = role_a ? (uint32_t)(nrows * L * 4) : (uint32_t)(L * BW_N * 4);
  const __amdgpu_buffer_rsrc_t ro0 =
      buffer_rsrc(role_a ? a.ddelta + row0 * L : w.dB_p + (b * G + g) * L * BW_N, out_b);
  const __amdgpu_buffer_rsrc_t ro1 =
      buffer_rsrc(role_a ? a.dx + row0 * L : w.dC_p + (b * G + g) * L * BW_N, out_b);
  const __amdgpu_buffer_rsrc_t roz =
      buffer_rsrc(GATED ? a.dz + row0 * L : a.dx, GATED && role_a ? out_b : 0u);
  auto load_tile = [&](int64_t k, Raw& v) {
    if constexpr (BUF) {
      // a tile before the start reads tile 0 (unused); past the end, the
      // offsets run out of the resources or into other rows (unused)
      const int64_t kc = k < 0 ? 0 : k;
      const int64_t rem = L - k * BW_T;
      const int32_t lim = k < 0 ? 0 : (int32_t)(rem < 0 ? 0 : (rem < BW_T ? rem : BW_T));
      v.ok = role_a ? (sdok && st < lim) : (bt < lim && n0 + bn < N);
      const int32_t tk = (int32_t)kc * BW_T;  // first step of the tile
      v.r0 = buf_ld<IN>(r0s, e01 * (int32_t)sizeof(IN), tk * (ts01 / BW_T) * (int32_t)sizeof(IN));
      v.r1 = buf_ld<IN>(r1s, e01 * (int32_t)sizeof(IN), tk * (ts01 / BW_T) * (int32_t)sizeof(IN));
      v.dy = buf_ld<DYT>(rdy, ea * (int32_t)sizeof(DYT), tk * (int32_t)sizeof(DYT));
      if constexpr (GATED) {
        v.z = buf_ld<IN>(rz, ea * (int32_t)sizeof(IN), tk * (int32_t)sizeof(IN));
        v.s = buf_ld<float>(rs, ea * 4, tk * 4);
      }
      return;
    }
    // every address is clamped into range, so tiles past either end (the
    // read-ahead) load valid, unused elements
    const int64_t ta = k * BW_T + st;
    const int64_t tca = ta < 0 ? 0 : (ta < L ? ta : L - 1);
    const int64_t ia = srow * L + tca;
    const int64_t tb = k * BW_T + bt;
    const int64_t tcb = tb < 0 ? 0 : (tb < L ? tb : L - 1);
    const int64_t ib = (b * L + tcb) * N + (n0 + bn < N ? n0 + bn : N - 1);
    v.ok = role_a ? (sdok && ta >= 0 && ta < L) : (tb >= 0 && tb < L && n0 + bn < N);
    const int64_t i01 = role_a ? ia : ib;
    v.r0 = P0[i01];
    v.r1 = P1[i01];
    v.dy = DY[ia];
    if constexpr (GATED) {
      v.z = Z[ia];
      v.s = w.s[ia];
    }
  };
  // delta after bias and softplus, and d delta / d raw (1 without softplus)
  auto widen_delta = [&](float raw, bool live, float& dlv, float& sg) {
    float v = raw + dbias;
    sg = 1.0f;
    if (a.softplus) {
      sg = sigmoid_f32(v);
      v = softplus_f32(v);
    }
    dlv = live ? v : 0.0f;
  };
  auto bc_val = [&](IN r, bool ok) { return ok ? widen<IN>(r) : 0.0f; };
  const int64_t ck_row = row * ntile;
  auto ck_at = [&](int64_t k) {
    const int64_t kc = k < 0 ? 0 : (k < ntile ? k : ntile - 1);
    return w.ck + (ck_row + kc) * BW_N + n;
  };
  // the checkpoint of tile k (clamped into range; the ones outside are unused)
  auto ck_load = [&](int64_t k) {
    if constexpr (BUF) {
      const int64_t kc = k < 0 ? 0 : (k < ntile ? k : ntile - 1);
      return buf_ld<float>(rck, eck * 4, (int32_t)kc * (BW_N * 4));
    } else {
      return *ck_at(k);
    }
  };

  // Raw inputs of tile j live in ring[j % BW_RING]: loads run BW_RING - 1
  // tiles ahead of their use.
  Raw ring[BW_RING];

  // --- 1. forward sweep: checkpoints (unless the forward pass supplied them)
  float h = (a.h0 && dok && nok) ? a.h0[row * N + ns] : 0.0f;
  const int64_t ntile1 = a.ckpt ? 0 : ntile;
#pragma unroll
  for (int u = 0; u < BW_RING - 1; ++u) load_tile(u, ring[u]);
  for (int64_t k0 = 0; k0 < ntile1; k0 += BW_RING) {
#pragma unroll
    for (int u = 0; u < BW_RING; ++u) {
      const int64_t k = k0 + u;
      if (k >= ntile1) break;
      const int buf = u & 1;  // BW_RING is even, so this is k & 1
      Raw& cur = ring[u];
      if (role_a) {
        float dlv, sg;
        widen_delta(widen<IN>(cur.r1), cur.ok, dlv, sg);
        sm.rv[buf][0][sr][st] = dlv;
        sm.rv[buf][1][sr][st] = cur.ok ? dlv * widen<IN>(cur.r0) : 0.0f;
      } else {
        sm.bc[buf][0][bn][swz(bn, bt)] = bc_val(cur.r0, cur.ok);
      }
      load_tile(k + BW_RING - 1, ring[(u + BW_RING - 1) % BW_RING]);
      bw_barrier();  // one per tile: the other buffer is the one staged next
      if constexpr (BUF)
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(h), rck, dok ? eck * 4 : (int32_t)ck_b,
                                              (int32_t)k * (BW_N * 4), 0);
      else
        *(dok ? w.ck + (ck_row + k) * BW_N + n : w.trash + tid) = h;
#pragma unroll
      for (int q = 0; q < BW_T; q += 4) {
        const float4 dl4 = *reinterpret_cast<const float4*>(&sm.rv[buf][0][rr][q]);
        const float4 dx4 = *reinterpret_cast<const float4*>(&sm.rv[buf][1][rr][q]);
        const float4 b4 = *reinterpret_cast<const float4*>(&sm.bc[buf][0][n][swz(n, q)]);
        const float dlq[4] = {dl4.x, dl4.y, dl4.z, dl4.w};
        const float dxq[4] = {dx4.x, dx4.y, dx4.z, dx4.w};
        const float bq[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
        for (int j = 0; j < 4; ++j)
          h = __builtin_fmaf(__builtin_amdgcn_exp2f(dlq[j] * Al), h, dxq[j] * bq[j]);
      }
    }
  }
  bw_barrier();  // the reverse sweep restages the buffers of the last tiles

  // --- 2./3. reverse sweep ---------------------------------------------------
  float lam = (a.dh_last && dok && nok) ? a.dh_last[row * N + ns] : 0.0f;
  float dA_acc = 0.0f;
  float dD_acc = 0.0f, db_acc = 0.0f;  // role a: this thread's (row, step slot)
  float hring[BW_RING];
#pragma unroll
  for (int u = 0; u < BW_RING - 1; ++u) {
    load_tile(ntile - 1 - u, ring[u]);
    hring[u] = ck_load(ntile - 1 - u);
  }
  // Sums of tile k from partial buffer pb (role a: over the states, ddelta
  // and dx of row sr, step st; role b: over the four wavefronts' row sums,
  // this workgroup's share of dB, dC at step bt, state bn), with the
  // role-a values saved from that tile's staging.  The stores are the same
  // instructions for every lane, aimed at the trash slots where a lane has
  // nothing to store.
  float p_dlv = 0.f, p_sg = 1.f, p_ds = 0.f, p_gp = 0.f, p_xv = 0.f, p_dyv = 0.f, p_sv = 0.f;
  bool p_live = false;
  auto reduce_tile = [&](int64_t k, int pb) {
    float v0, v1, v2 = 0.f;
    float *p0, *p1, *p2 = w.trash + tid;
    uint32_t o = out_b;  // BUF: the byte offset of both outputs
    if (role_a) {
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int m = 0; m < BW_N; ++m) {
        s1 += sm.sp[pb][0][sr * BW_RS + m * BW_TS + swz(m, st)];
        s2 += sm.sp[pb][1][sr * BW_RS + m * BW_TS + swz(m, st)];
      }
      const float ddl = p_live ? (s1 + p_xv * s2) * p_sg : 0.0f;
      v0 = ddl;
      v1 = __builtin_fmaf(p_dlv, s2, first ? p_ds * Dsk : 0.0f);
      if constexpr (BUF) {
        if (p_live) o = (uint32_t)(ea + (int32_t)k * BW_T) * 4u;
      } else {
        const int64_t i = srow * L + (p_live ? k * BW_T + st : 0);
        p0 = p_live ? a.ddelta + i : w.trash + tid;
        p1 = p_live ? a.dx + i : w.trash + tid;
        if constexpr (GATED) p2 = p_live ? a.dz + i : w.trash + tid;
      }
      if constexpr (GATED) v2 = p_dyv * p_sv * p_gp;
      if (first) dD_acc = __builtin_fmaf(p_ds, p_xv, dD_acc);
      db_acc += ddl;
    } else {
      // lane (bt / 4) * 16 + bn of each wavefront holds the dB sums of
      // steps 4 (bt / 4) .. +3 at state bn, lane 32 more the dC sums
      const int lb = (bt >> 2) * 16 + bn, tb = bt & 3;
      float sb = 0.f, sc = 0.f;
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        sb += sm.pw[pb][m][lb * 4 + tb];
        sc += sm.pw[pb][m][(32 + lb) * 4 + tb];
      }
      const int64_t t = k * BW_T + bt;
      v0 = sb;
      v1 = sc;
      if constexpr (BUF) {
        if (t < L) o = (uint32_t)((int32_t)t * BW_N + bn) * 4u;
      } else {
        const int64_t i = ((b * G + g) * L + (t < L ? t : 0)) * BW_N + bn;
        p0 = t < L ? w.dB_p + i : w.trash + tid;
        p1 = t < L ? w.dC_p + i : w.trash + tid;
      }
    }
    if constexpr (BUF) {
      if (role_a && !first) {  // later state groups add to the sums over the states
        v0 += buf_ld<float>(ro0, (int32_t)o, 0);
        v1 += buf_ld<float>(ro1, (int32_t)o, 0);
      }
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v0), ro0, (int32_t)o, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v1), ro1, (int32_t)o, 0, 0);
      if constexpr (GATED) {
        if (first) __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v2), roz, (int32_t)o, 0, 0);
      }
    } else {
      if (role_a && !first) {  // later state groups add to the sums over the states
        v0 += *p0;
        v1 += *p1;
      }
      *p0 = v0;
      *p1 = v1;
      if constexpr (GATED) {
        if (first) *p2 = v2;
      }
    }
  };

  for (int64_t k0 = ntile - 1; k0 >= 0; k0 -= BW_RING) {
#pragma unroll
    for (int u = 0; u < BW_RING; ++u) {
      const int64_t k = k0 - u;
      if (k < 0) break;
      // tile k is in ring[u] (its index counted down from the last tile)
      const int buf = (int)(k & 1);
      Raw& cur = ring[u];
      float dlv = 0.f, sg = 1.f, ds = 0.f, gp = 0.f, xv = 0.f, dyv = 0.f, sv = 0.f;
      const bool live = role_a && cur.ok;
      if (role_a) {
        widen_delta(widen<IN>(cur.r1), live, dlv, sg);
        xv = widen<IN>(cur.r0);
        dyv = widen<DYT>(cur.dy);
        float gt = 1.0f;
        if constexpr (GATED) {
          const float zv = widen<IN>(cur.z);
          const float sz = sigmoid_f32(zv);
          gt = zv * sz;
          gp = sz * (1.0f + zv * (1.0f - sz));
          sv = cur.s;
        }
        ds = live ? dyv * gt : 0.0f;
        sm.rv[buf][0][sr][st] = dlv;
        sm.rv[buf][1][sr][st] = live ? dlv * xv : 0.0f;
        sm.rv[buf][2][sr][st] = ds;
      } else {
        sm.bc[buf][0][bn][swz(bn, bt)] = bc_val(cur.r0, cur.ok);
        sm.bc[buf][1][bn][swz(bn, bt)] = bc_val(cur.r1, cur.ok);
      }
      const float hstart = dok ? hring[u] : 0.0f;
      load_tile(k - (BW_RING - 1), ring[(u + BW_RING - 1) % BW_RING]);
      hring[(u + BW_RING - 1) % BW_RING] = ck_load(k - (BW_RING - 1));
      bw_barrier();  // tile k is staged, tile k+1's partials are complete

      if (k + 1 < ntile) reduce_tile(k + 1, (int)((k + 1) & 1));
      p_dlv = dlv;
      p_sg = sg;
      p_ds = ds;
      p_gp = gp;
      p_xv = xv;
      p_dyv = dyv;
      p_sv = sv;
      p_live = live;

      // recompute a_t, q_t = a_t h_{t-1} and h_t of the tile; delta, delta*x
      // and B stay in registers for the backward walk
      float av[BW_T], qv[BW_T], hv[BW_T], dlr[BW_T], dxr[BW_T], br[BW_T];
      {
        float hh = hstart;
#pragma unroll
        for (int q = 0; q < BW_T; q += 4) {
          const float4 dl4 = *reinterpret_cast<const float4*>(&sm.rv[buf][0][rr][q]);
          const float4 dx4 = *reinterpret_cast<const float4*>(&sm.rv[buf][1][rr][q]);
          const float4 b4 = *reinterpret_cast<const float4*>(&sm.bc[buf][0][n][swz(n, q)]);
          const float dlq[4] = {dl4.x, dl4.y, dl4.z, dl4.w};
          const float dxq[4] = {dx4.x, dx4.y, dx4.z, dx4.w};
          const float bq[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            dlr[q + j] = dlq[j];
            dxr[q + j] = dxq[j];
            br[q + j] = bq[j];
            av[q + j] = __builtin_amdgcn_exp2f(dlq[j] * Al);
            qv[q + j] = av[q + j] * hh;
            hh = __builtin_fmaf(dxq[j], bq[j], qv[q + j]);
            hv[q + j] = hh;
          }
        }
      }
      // walk the tile backwards
      float* const sp0 = &sm.sp[buf][0][rr * BW_RS + n * BW_TS];
      float* const sp1 = &sm.sp[buf][1][rr * BW_RS + n * BW_TS];
      float pdx[BW_T], pdh[BW_T];  // lam delta x and ds h, summed over rows below
#pragma unroll
      for (int q = BW_T - 4; q >= 0; q -= 4) {
        const float4 ds4 = *reinterpret_cast<const float4*>(&sm.rv[buf][2][rr][q]);
        const float4 c4 = *reinterpret_cast<const float4*>(&sm.bc[buf][1][n][swz(n, q)]);
        const float dsq[4] = {ds4.x, ds4.y, ds4.z, ds4.w};
        const float cq[4] = {c4.x, c4.y, c4.z, c4.w};
        float o0[4], o1[4];
#pragma unroll
        for (int j = 3; j >= 0; --j) {
          const int t = q + j;
          const float l = __builtin_fmaf(dsq[j], cq[j], lam);
          const float p = l * qv[t];
          dA_acc = __builtin_fmaf(p, dlr[t], dA_acc);
          o0[j] = p * Ar;
          o1[j] = l * br[t];
          pdx[t] = l * dxr[t];
          pdh[t] = dsq[j] * hv[t];
          lam = av[t] * l;
        }
        const int qs = swz(n, q);
        *reinterpret_cast<float4*>(sp0 + qs) = make_float4(o0[0], o0[1], o0[2], o0[3]);
        *reinterpret_cast<float4*>(sp1 + qs) = make_float4(o1[0], o1[1], o1[2], o1[3]);
      }
      {
        float o[4];
        rows4_sum(pdx, pdh, o);
        *reinterpret_cast<float4*>(&sm.pw[buf][wv][lane * 4]) =
            make_float4(o[0], o[1], o[2], o[3]);
      }
    }
  }
  bw_barrier();  // tile 0's partials are complete
  reduce_tile(0, 0);

  if (dok && nok) {
    if (a.dh0) a.dh0[row * N + ns] = lam;
    w.dA_p[row * BW_N + n] = dA_acc;
  }
  // per-row sums of the step slots (8 consecutive lanes of role a)
  if (role_a) {
#pragma unroll
    for (int off = 1; off < BW_T; off *= 2) {
      dD_acc += __shfl_xor(dD_acc, off);
      db_acc += __shfl_xor(db_acc, off);
    }
    if (st == 0 && sdok) {
      if (first) {
        w.dD_p[srow] = dD_acc;
        w.db_p[srow] = db_acc;
      } else {
        w.db_p[srow] += db_acc;
      }
    }
  }
}

// Adds the shares in a fixed order: dB, dC over the workgroups of a batch
// (one thread per 4 states of one (b, t) and one of dB / dC, float4 loads,
// eight in flight, summed in workgroup order); dA, dDskip, ddelta_bias over
// the batch.
// With state groups (N > 16) it runs after each group's main kernel and
// writes that group's states n0 .. n0+15; dDskip and ddelta_bias after the
// last group (last = true).
__global__ __launch_bounds__(256) void selective_bwd_reduce_kernel(const BwdArgs a,
                                                                   const BwWork w, int64_t G,
                                                                   int n0, bool last) {
  const int64_t B = a.B, D = a.D, N = a.N, L = a.L;
  const int64_t ng = N - n0 < BW_N ? N - n0 : BW_N;  // states of this group
  const int64_t nq = B * L * (BW_N / 4);  // float4 chunks of one of dB / dC
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t gstep = L * (BW_N / 4);   // float4 stride between workgroup shares
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < 2 * nq; i += stride) {
    const bool isC = i >= nq;
    const int64_t r = isC ? i - nq : i;  // r = (b*L + t)*4 + c
    const int64_t c = r % (BW_N / 4), bt = r / (BW_N / 4);
    const int64_t b = bt / L;
    const float4* __restrict__ src =
        reinterpret_cast<const float4*>(isC ? w.dC_p : w.dB_p) + b * G * gstep + (bt - b * L) * 4 + c;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    int64_t g = 0;
    for (; g + 8 <= G; g += 8) {
      float4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = src[(g + u) * gstep];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        acc.x += v[u].x;
        acc.y += v[u].y;
        acc.z += v[u].z;
        acc.w += v[u].w;
      }
    }
    for (; g < G; ++g) {
      const float4 v = src[g * gstep];
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
    float* const dst = (isC ? a.dC : a.dB) + bt * N + n0;
    const float av[4] = {acc.x, acc.y, acc.z, acc.w};
    if (N == BW_N && (((uintptr_t)a.dB | (uintptr_t)a.dC) & 15) == 0) {
      *reinterpret_cast<float4*>(dst + 4 * c) = acc;
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (4 * c + u < ng) dst[4 * c + u] = av[u];
    }
  }
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < D * ng; i += stride) {
    const int64_t d = i / ng, nn = i - d * ng;
    float s = 0.f;
    for (int64_t b = 0; b < B; ++b) s += w.dA_p[(b * D + d) * BW_N + nn];
    a.dA[d * N + n0 + nn] = s;
  }
  if (!last) return;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < D; i += stride) {
    float sd = 0.f, sbias = 0.f;
    for (int64_t b = 0; b < B; ++b) {
      sd += w.dD_p[b * D + i];
      sbias += w.db_p[b * D + i];
    }
    if (a.dDskip) a.dDskip[i] = sd;
    if (a.ddelta_bias) a.ddelta_bias[i] = sbias;
  }
}

// True when every byte offset of the buffer-resource path stays below 2^31:
// a workgroup's rows of x, delta, dy, z and s, a batch's B and C, and a
// workgroup's checkpoints, with the read-ahead tiles past the end.
bool bwd_buf_fits(const BwdArgs& a, int64_t ntile) {
  const int64_t lim = (int64_t)1 << 31;
  const int64_t Lp = a.L + 4 * BW_RING * BW_T;
  return BW_ROWS * Lp * 4 < lim && Lp * a.N * 4 < lim && Lp * BW_N * 4 < lim &&
         BW_ROWS * (ntile + 2 * BW_RING) * BW_N * 4 < lim;
}

template <typename IN, typename DYT>
void launch_bwd_dy(const BwdArgs& a, const BwWork& w, int64_t G, int64_t ntile, int64_t grid,
                   int n0, hipStream_t s) {
  const bool buf = bwd_buf_fits(a, ntile);
  auto kern = a.z ? (buf ? selective_bwd_kernel<IN, DYT, true, true>
                         : selective_bwd_kernel<IN, DYT, true, false>)
                  : (buf ? selective_bwd_kernel<IN, DYT, false, true>
                         : selective_bwd_kernel<IN, DYT, false, false>);
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), 0, s, a, w, G, ntile, n0);
}

void launch_bwd(const BwdArgs& a, const BwWork& w, int64_t G, int64_t ntile, int64_t grid,
                int n0, hipStream_t s) {
  if (a.bf16_in) {
    if (a.dy_bf16)
      launch_bwd_dy<uint16_t, uint16_t>(a, w, G, ntile, grid, n0, s);
    else
      launch_bwd_dy<uint16_t, float>(a, w, G, ntile, grid, n0, s);
  } else {
    if (a.dy_bf16)
      launch_bwd_dy<float, uint16_t>(a, w, G, ntile, grid, n0, s);
    else
      launch_bwd_dy<float, float>(a, w, G, ntile, grid, n0, s);
  }
}

}  // namespace

int selective_bwd(const BwdArgs& a) {
  if (a.ckpt && a.N > BW_N)
    return fail(SW_ERR_UNSUPPORTED, "checkpoints hold 16 states (N=%lld)", (long long)a.N);
  hipStream_t s = current_stream();
  const int64_t B = a.B, D = a.D, L = a.L;
  const int64_t G = (D + BW_ROWS - 1) / BW_ROWS;
  const int64_t ntile = (L + BW_T - 1) / BW_T;
  const int64_t grid = B * G;
  if (grid >= ((int64_t)1 << 31))
    return fail(SW_ERR_UNSUPPORTED, "%lld workgroups exceed the grid range", (long long)grid);
  const size_t R = (size_t)(B * D);
  // without the forward's checkpoints the kernel rebuilds them in a workspace
  const size_t n_ck = a.ckpt ? 0 : R * (size_t)ntile * BW_N;
  const size_t n_s = (a.z && !a.s_pre) ? R * (size_t)L : 0;
  const size_t n_dA = R * BW_N, n_bc = (size_t)(B * G) * (size_t)L * BW_N;
  const size_t total = n_ck + n_s + n_dA + 2 * R + 2 * n_bc + 256;
  void* base = nullptr;
  int st = workspace_alloc(&base, total * sizeof(float), s);
  if (st != SW_OK) return st;
  float* f = static_cast<float*>(base);
  BwWork w;
  w.ck = a.ckpt ? const_cast<float*>(a.ckpt) : f;  // read-only when given
  f += n_ck;
  float* s_pre = (a.z && !a.s_pre) ? f : nullptr;
  w.s = a.s_pre ? a.s_pre : s_pre;
  f += n_s;
  w.dA_p = f;
  f += n_dA;
  w.dD_p = f;
  f += R;
  w.db_p = f;
  f += R;
  w.dB_p = f;
  f += n_bc;
  w.dC_p = f;
  f += n_bc;
  w.trash = f;
  // with a gate, the forward without the gate runs anyway (for the pre-gate
  // output); for N <= 16 it also writes the tile checkpoints, so the backward
  // kernel skips its own forward sweep (the checkpoints are bit-identical)
  BwdArgs ab = a;
  if (a.z && !a.s_pre) {
    // the pre-gate output: the forward pass without the gate
    SelArgs fa{};
    fa.x = a.x;
    fa.delta = a.delta;
    fa.Bm = a.Bm;
    fa.Cm = a.Cm;
    fa.A = a.A;
    fa.Dskip = a.Dskip;
    fa.delta_bias = a.delta_bias;
    fa.h0 = a.h0;
    fa.y = s_pre;
    fa.B = B;
    fa.D = D;
    fa.N = a.N;
    fa.L = L;
    fa.bf16_in = a.bf16_in;
    fa.softplus = a.softplus;
    fa.vec = a.vec;
    if (!a.ckpt && a.N <= BW_N) {
      fa.ckpt = w.ck;
      ab.ckpt = w.ck;
    }
    st = selective_fwd(fa);
    if (st != SW_OK) {
      workspace_free(base, s);
      return st;
    }
  }
  // still without checkpoints: where the forward takes its 16-lane layout,
  // its walk without y writes them (the states do not depend on the gate),
  // cheaper than the backward kernel's own sweep and bit-identical to it
  const char* ck_from = a.ckpt ? "given" : ab.ckpt ? "from the ungated forward" : nullptr;
  if (!ab.ckpt && a.N == BW_N) {
    SelArgs fa{};
    fa.x = a.x;
    fa.delta = a.delta;
    fa.Bm = a.Bm;
    fa.Cm = a.Cm;
    fa.A = a.A;
    fa.delta_bias = a.delta_bias;
    fa.h0 = a.h0;
    fa.B = B;
    fa.D = D;
    fa.N = a.N;
    fa.L = L;
    fa.bf16_in = a.bf16_in;
    fa.softplus = a.softplus;
    fa.vec = a.vec;
    fa.ckpt = w.ck;
    bool taken = false;
    st = selective_states_fwd(fa, &taken);
    if (st != SW_OK) {
      workspace_free(base, s);
      return st;
    }
    if (taken) {
      ab.ckpt = w.ck;
      ck_from = "from the forward's walk without y";
    }
  }
  if (!ck_from) ck_from = "rebuilt by the backward kernel";
  // the states in groups of 16: each group's main kernel, then its reduction
  // (dA, dB, dC of its states; the sums over the states accumulate)
  for (int n0 = 0; n0 < a.N && st == SW_OK; n0 += BW_N) {
    launch_bwd(ab, w, G, ntile, grid, n0, s);
    st = check_launch("selective_bwd_kernel");
    if (st != SW_OK) break;
    int64_t work = 2 * B * L * (BW_N / 4);
    if (work < D * BW_N) work = D * BW_N;
    int64_t blocks = (work + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(selective_bwd_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, w,
                       G, n0, n0 + BW_N >= a.N);
    st = check_launch("selective_bwd_reduce_kernel");
  }
  workspace_free(base, s);
  if (st == SW_OK)
    note_launch("selective_bwd_kernel + selective_bwd_reduce_kernel (%lld state group%s), "
                "checkpoints %s",
                (long long)((a.N + BW_N - 1) / BW_N), a.N > BW_N ? "s" : "", ck_from);
  return st;
}

}  // namespace sw
