/*
 * scanweaver.h -- C ABI of libscanweaver.so, the MI355X (gfx950) library for
 * the forward affine recurrence and the Mamba-style fused selective scan.
 *
 * The operation (ScanWeaver, Sec. 3.1-3.2): for every independent channel,
 *
 *     h_t = a_t * h_{t-1} + bx_t                                   Eq. (3)
 *
 * evaluated as a prefix scan over the affine pairs (A_t, U_t) = (a_t, bx_t)
 * of Eq. (6) under the composition of Eq. (7),
 *
 *     (A2, U2) (+) (A1, U1) = (A2*A1, A2*U1 + U2)   (left = later segment),
 *
 * so that h_t = A_{1:t} h_0 + U_{1:t}.  The library returns the inclusive
 * states h_1..h_L, i.e. exactly what a sequential traversal produces
 * (Sec. 3.2), for every (b, d) row.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Arrays are caller-owned DEVICE pointers (hipMalloc / torch CUDA tensors)
 *    on the current HIP device, dense and row-major; the library never frees
 *    or keeps them.  Host pointers are rejected with SW_ERR_INVALID_ARG.
 *  - Alignment: natural alignment of the element type is required (4 bytes for
 *    fp32/int32, 2 bytes for bf16).  Wider vector loads are used when every
 *    pointer is 16-byte aligned and L allows it; results do not depend on it.
 *  - Calls are asynchronous: SW_OK means the work was enqueued on the stream
 *    set with sw_set_stream() for the calling thread (default: the null
 *    stream).  Faults surface at the caller's next synchronisation.
 *  - Validation happens before anything is enqueued: on any non-OK return no
 *    output has been written and nothing is launched.  sw_last_error() gives
 *    a message for the last non-OK return on the calling thread.
 *  - Negative sizes are SW_ERR_INVALID_ARG.  A call whose output is empty
 *    (B*D == 0, or L == 0 for the bare scan) returns SW_OK and touches
 *    nothing; pointers are not inspected in that case.
 *  - Outputs must not overlap inputs or each other (SW_ERR_INVALID_ARG).
 *  - Scratch memory: calls whose sequences are split across workgroups use
 *    a small scratch per (device, stream) -- carry words and a ticket
 *    counter -- allocated from the device's default stream-ordered pool on
 *    the first such call on that stream, kept for later calls (grown when a
 *    call needs more) and never freed by the library.  The backward pass
 *    takes a per-call workspace from the same pool on the same stream and
 *    releases it, stream-ordered, before returning.  The library raises that
 *    pool's release threshold so freed blocks stay cached for the next call
 *    (a process-wide setting of the device's default pool).  SW_ERR_ALLOC if
 *    an allocation fails.
 *  - Threads using distinct streams may call concurrently.
 *  - HIP graph capture: a call that uses neither the scratch nor a workspace
 *    can be captured and replayed: it launches kernels only.  Such calls are
 *    the fused forward at N = 16 with L a multiple of 8 for bf16 or of 4 for
 *    fp32, 16-byte aligned arrays and a workgroup's byte offsets below 2^31;
 *    the bare scan and its projection form when a row fits one chunk
 *    (L <= 2048) or the rows alone fill the GPU (B*D >= 8 per compute unit);
 *    sw_affine_scan_noalloc on every path (its look-back words live in a
 *    static array that each call clears with a fill kernel and starts from
 *    the same epoch and ticket, so a replay repeats the call exactly); and
 *    the Blelloch schedule entry points.  A call that uses the scratch
 *    is not replay-safe (a replay would repeat the ticket range and epoch the
 *    host gave the captured launch), and the backward allocates a workspace
 *    per call: while the stream is capturing, those calls return
 *    SW_ERR_UNSUPPORTED before enqueuing anything.
 */
#ifndef SCANWEAVER_H
#define SCANWEAVER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sw_status {
  SW_OK = 0,              /* enqueued */
  SW_ERR_INVALID_ARG = 1, /* NULL / host / misaligned / overlapping pointer, negative size */
  SW_ERR_UNSUPPORTED = 2, /* a size outside what the kernels handle (e.g. N > 64) */
  SW_ERR_HIP = 3,         /* a HIP runtime call or launch failed */
  SW_ERR_ALLOC = 4        /* scratch allocation failed */
} sw_status;

/* Version of this ABI, major*10000 + minor*100 + patch (200: the training
 * forward and the backward exchange the pre-gate output, s_pre). */
int sw_version(void);

/*
 * Bare affine scan, fp32 (Eq. (3); pairs Eq. (6); composition Eq. (7)).
 *   a, bx, h_out : (B, D, L) fp32, L fastest.  h_out[b,d,t] is the state
 *                  after step t, i.e. a[b,d,t]*h_out[b,d,t-1] + bx[b,d,t].
 *   h0           : (B, D) fp32 initial state h[b,d,-1], or NULL for zero.
 * Arithmetic is fp32 (the composition is evaluated in an order that differs
 * from the sequential loop, so results are not bitwise equal to it; they
 * agree to within the rounding of fp32 affine compositions).
 */
int sw_affine_scan(const float* a, const float* bx, const float* h0, float* h_out, int64_t B,
                   int64_t D, int64_t L);

/*
 * Bare affine scan in the int32 wraparound ring Z/2^32: the same recurrence
 * on two's-complement bit patterns with arithmetic modulo 2^32.  The ring is
 * exact under any association order, so the result is bit-identical to the
 * sequential loop for every schedule.
 *   a, bx, h_out : (B, D, L) int32;  h0 : (B, D) int32 or NULL for zero.
 */
int sw_affine_scan_i32(const int32_t* a, const int32_t* bx, const int32_t* h0, int32_t* h_out,
                       int64_t B, int64_t D, int64_t L);

/*
 * sw_affine_scan for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, layout, results (within fp32 rounding of the same
 * schedule) and errors as sw_affine_scan, but no hipMalloc, hipFree or
 * allocating library routine is called: the look-back tickets and chunk
 * carries live in a static array in the library's device code (256 bytes +
 * 24 bytes per chunk, 1.5 MiB for SW_NOALLOC_MAX_CHUNKS chunks), one copy per
 * GPU, held until the process ends; its address is looked up on the first
 * call on each device (make that call before capturing one into a HIP
 * graph).  Each call clears the part it uses with a fill kernel on the
 * call's stream before the scan.
 *   - Calls whose chunk-parallel look-back kernel would need more than
 *     SW_NOALLOC_MAX_CHUNKS chunks return SW_ERR_UNSUPPORTED before enqueuing
 *     anything.  That kernel runs when L > 2048 and B*D < 8 * (compute
 *     units); its chunk count is B * D * ceil(L / 2048).  Other calls (one
 *     chunk per row, or enough rows to give each its own workgroup) use no
 *     scratch and have no limit beyond sw_affine_scan's.
 *   - Every call on one GPU shares that GPU's array: two calls that may run
 *     at the same time on one GPU (on different streams, or from different
 *     host threads without ordering) race and give wrong results.  Order
 *     them on one stream.
 */
#define SW_NOALLOC_MAX_CHUNKS 65536
int sw_affine_scan_noalloc(const float* a, const float* bx, const float* h0, float* h_out,
                           int64_t B, int64_t D, int64_t L);

/* Scan schedules of sw_affine_scan_schedule. */
enum {
  SW_SCHED_DEFAULT = 0,  /* the library's: lane-sequential composition, DPP wavefront scan,
                            LDS combine, decoupled look-back (what sw_affine_scan runs) */
  SW_SCHED_BLELLOCH = 1  /* the paper's (Sec. 3.3): a Blelloch upsweep / root / downsweep tree
                            over 2048-pair chunks in LDS, then affine-prefix reconstruction;
                            one workgroup per row, chunk carries in registers */
};

/*
 * sw_affine_scan (fp32) and sw_affine_scan_i32 with an explicit scan
 * schedule, for comparing schedules on the same recurrence.  Same arguments,
 * layout, results (bit-identical in int32; within fp32 rounding in fp32) and
 * errors, plus SW_ERR_INVALID_ARG for an unknown schedule.  The Blelloch
 * schedule gives each (b,d) row one workgroup, so it fills the GPU only when
 * there are many rows.
 */
int sw_affine_scan_schedule(const float* a, const float* bx, const float* h0, float* h_out,
                            int64_t B, int64_t D, int64_t L, int schedule);
int sw_affine_scan_schedule_i32(const int32_t* a, const int32_t* bx, const int32_t* h0,
                                int32_t* h_out, int64_t B, int64_t D, int64_t L, int schedule);

/*
 * The fused selective scan (plain form: fp32 y, zero initial state, no
 * options) with an explicit schedule.  SW_SCHED_DEFAULT is
 * sw_selective_scan_fwd / _bf16 (in_dtype F32 / BF16).  SW_SCHED_BLELLOCH
 * scans every (b,d,n) recurrence over t with the paper's Blelloch tree in LDS
 * (2048-step chunks, one workgroup per row looping over the states,
 * y accumulated in registers), for comparing schedules on the method's own
 * workload.  Arguments, layouts, results (within fp32 rounding) and errors
 * as for sw_selective_scan_fwd, plus SW_ERR_INVALID_ARG for an unknown dtype
 * or schedule.
 */
int sw_selective_scan_fwd_schedule(const void* x, const void* delta, const float* A,
                                   const void* Bm, const void* Cm, const float* Dskip, float* y,
                                   float* h_last, int64_t B, int64_t D, int64_t N, int64_t L,
                                   int in_dtype, int schedule);

/*
 * Recurrence with input and output projections, elementwise (Eq. (3)-(4)):
 *   h[b,d,t] = a[b,d,t] * h[b,d,t-1] + b[b,d,t] * x[b,d,t]      (h[b,d,-1] = h0)
 *   y[b,d,t] = c[b,d,t] * h[b,d,t]
 * The weighted prefix of Eq. (10) is the case x = 1, c = 1 (alpha -> a,
 * beta -> b).
 *   a, b, y      : (B, D, L) fp32, L fastest, required.
 *   x, c         : (B, D, L) fp32, or NULL for all ones.
 *   h0           : (B, D) fp32 initial state, or NULL for zero.
 *   h_last       : (B, D) fp32, receives h[b,d,L-1] (h0, or zero, when
 *                  L == 0), or NULL.
 * b*x and c*h are each rounded to fp32 once; the scan itself is that of
 * sw_affine_scan on the pairs (a, b*x), so with x and c NULL, y equals the
 * h_out of sw_affine_scan bit for bit.  Same conventions as sw_affine_scan
 * otherwise: caller-owned device pointers, outputs may not overlap inputs,
 * SW_ERR_INVALID_ARG for a NULL required pointer, misalignment, foreign or
 * host memory, negative sizes or overlap; SW_ERR_UNSUPPORTED when B*D*L
 * overflows.
 */
int sw_affine_scan_proj(const float* a, const float* b, const float* x, const float* c,
                        const float* h0, float* y, float* h_last, int64_t B, int64_t D,
                        int64_t L);

/*
 * The same in the int32 wraparound ring: b*x, the recurrence and c*h modulo
 * 2^32 on two's-complement bit patterns; bit-identical to the sequential loop.
 */
int sw_affine_scan_proj_i32(const int32_t* a, const int32_t* b, const int32_t* x,
                            const int32_t* c, const int32_t* h0, int32_t* y, int32_t* h_last,
                            int64_t B, int64_t D, int64_t L);

/*
 * Fused selective scan, forward, fp32 inputs (the Mamba-style instance of
 * Eq. (3) that motivates the method, Sec. 1 and Sec. 3.1), zero initial state:
 *
 *   a[b,d,t,n]  = exp(delta[b,d,t] * A[d,n])
 *   u[b,d,t,n]  = delta[b,d,t] * Bm[b,t,n] * x[b,d,t]
 *   h[b,d,t,n]  = a * h[b,d,t-1,n] + u                 (h[.,-1,.] = 0)
 *   y[b,d,t]    = sum_n Cm[b,t,n] * h[b,d,t,n] + Dskip[d] * x[b,d,t]
 *   h_last      = h[b,d,L-1,:]
 *
 *   x, delta : (B, D, L) fp32          A      : (D, N) fp32
 *   Bm, Cm   : (B, L, N) fp32          Dskip  : (D) fp32, or NULL for no skip
 *   y        : (B, D, L) fp32 output   h_last : (B, D, N) fp32 output or NULL
 * 1 <= N <= 64, else SW_ERR_UNSUPPORTED.  State and accumulation are fp32.
 * With L == 0 and B*D > 0, h_last (if given) is set to zero.
 * With N = 16, a call whose rows leave SIMDs idle or unevenly loaded may
 * split each row into up to 16 segments composed with Eq. (7), and may walk
 * each row with four lanes (four states each) instead of sixteen (fp32 y,
 * L a multiple of 32).  The library prices each choice with a model of its
 * launches on the device (per-step times measured per layout and occupancy)
 * and takes the cheapest; calls that write checkpoints walk whole rows.
 * Segments take one of two forms.  Correction form (fp32 y): every segment
 * walks from a zero state, a fold composes the carries, and each later
 * segment is walked again from its composed state only until the part
 * carried in has faded below 2^-26 of the magnitude of the state's own
 * terms (the whole segment when it does not fade).  Records form: each
 * segment's carry is formed first, then every segment walks once from its
 * initial state.  Results of both agree with a whole-row walk within fp32
 * rounding, not bit for bit.  The environment variables SW_SS_QUAD (0: never
 * four lanes per row, 1: whenever the call allows), SW_SS_SEGMENTS (the
 * count, 1: whole rows) and SW_SS_SEGFORM (1: records, 2: correction), read
 * per call, force the choice; sw_last_launch() names what a call enqueued.
 * A count k gives segments of L / k steps rounded up to the layout's
 * granularity (a 64- or 128-step super-tile with sixteen lanes per row, 64
 * steps with four), the last one the rest (a rest shorter than that
 * granularity joins the segment before, or, with four lanes per row, the
 * length is rounded down instead).
 * y's memory holds the segments' carries between the call's kernels, so y
 * must not be read until the call completes on its stream (as for any
 * output).
 */
int sw_selective_scan_fwd(const float* x, const float* delta, const float* A, const float* Bm,
                          const float* Cm, const float* Dskip, float* y, float* h_last,
                          int64_t B, int64_t D, int64_t N, int64_t L);

/*
 * As sw_selective_scan_fwd, with x, delta, Bm and Cm given as bf16 (raw
 * uint16 bit patterns, widened exactly to fp32 inside the kernel).  A, Dskip,
 * the state, y and h_last are fp32.
 */
int sw_selective_scan_fwd_bf16(const uint16_t* x, const uint16_t* delta, const float* A,
                               const uint16_t* Bm, const uint16_t* Cm, const float* Dskip,
                               float* y, float* h_last, int64_t B, int64_t D, int64_t N,
                               int64_t L);

/* Element types of sw_selective_scan_fwd_ex's arrays. */
typedef enum sw_dtype {
  SW_DTYPE_F32 = 0,  /* fp32 */
  SW_DTYPE_BF16 = 1  /* bf16, as raw uint16 bit patterns */
} sw_dtype;

/* Flags of sw_selective_scan_fwd_ex. */
enum { SW_DELTA_SOFTPLUS = 1 /* delta' = softplus(delta + delta_bias) */ };

/*
 * Fused selective scan, forward, with the optional inputs of a Mamba block
 * (the production kernel the method is measured against fuses the same
 * pieces; Sec. 1, Sec. 6.3).  With z, delta_bias, h0 NULL and flags 0 it is
 * sw_selective_scan_fwd (in_dtype F32) or sw_selective_scan_fwd_bf16 (BF16):
 *
 *   delta'[b,d,t] = delta[b,d,t] + delta_bias[d]        (bias: 0 if NULL)
 *                   then softplus(v) = log(1 + e^v)      if flags & SW_DELTA_SOFTPLUS
 *   a = exp(delta' * A[d,n]),  u = delta' * Bm[b,t,n] * x[b,d,t]
 *   h[b,d,-1,n] = h0[b,d,n]                              (0 if h0 is NULL)
 *   h[b,d,t,n] = a * h[b,d,t-1,n] + u                    (Eq. (3))
 *   y[b,d,t] = sum_n Cm[b,t,n] h[b,d,t,n] + Dskip[d] x[b,d,t]
 *   y[b,d,t] *= silu(z[b,d,t]) = z / (1 + e^-z)           if z is not NULL
 *   h_last[b,d,n] = h[b,d,L-1,n]
 *
 *   x, delta, z : (B, D, L) of in_dtype        Bm, Cm : (B, L, N) of in_dtype
 *   A : (D, N) fp32      Dskip, delta_bias : (D) fp32 or NULL
 *   h0, h_last : (B, D, N) fp32 or NULL        y : (B, D, L) of out_dtype
 * bf16 y is the fp32 result rounded to nearest even.  Softplus and silu are
 * evaluated in fp32 (a few ulps).  h0 may be the h_last of the previous
 * chunk of the same sequences, which continues the scan across calls; with
 * L == 0, h_last receives h0 (or zeros).  Unknown dtypes or flags:
 * SW_ERR_INVALID_ARG.  Other conventions as for sw_selective_scan_fwd.
 */
int sw_selective_scan_fwd_ex(const void* x, const void* delta, const float* A, const void* Bm,
                             const void* Cm, const float* Dskip, const void* z,
                             const float* delta_bias, const float* h0, void* y, float* h_last,
                             int64_t B, int64_t D, int64_t N, int64_t L, int in_dtype,
                             int out_dtype, int flags);

/*
 * sw_selective_scan_fwd_ex that also keeps what the backward pass needs
 * (training; always walks whole rows, so y is bit-identical to that of
 * sw_selective_scan_fwd_ex run with SW_SS_SEGMENTS=1): ckpt (B, D,
 * ceil(L/8), 16) fp32, required, receives the state
 * h[b,d,8k-1,n] before step 8k (h0, or zero, for k = 0) in slot
 * [b, d, k, n]; slots n >= N hold no state.  N <= 16 (SW_ERR_UNSUPPORTED
 * above).  s_pre (B, D, L) fp32, or NULL, receives y before the output gate
 * (y = s_pre * silu(z); without z, s_pre = y in fp32).  Handing ckpt (and,
 * with z, s_pre) to sw_selective_scan_bwd with the same inputs spares the
 * backward its own forward sweep (and its forward without the gate).
 * Otherwise as sw_selective_scan_fwd_ex.
 */
int sw_selective_scan_fwd_train(const void* x, const void* delta, const float* A, const void* Bm,
                                const void* Cm, const float* Dskip, const void* z,
                                const float* delta_bias, const float* h0, void* y, float* h_last,
                                float* ckpt, float* s_pre, int64_t B, int64_t D, int64_t N,
                                int64_t L, int in_dtype, int out_dtype, int flags);

/*
 * Backward of sw_selective_scan_fwd_ex: the gradients of
 *   sum_{b,d,t} dy[b,d,t] y[b,d,t] + sum_{b,d,n} dh_last[b,d,n] h_last[b,d,n]
 * with respect to every input, by the chain rule through Eq. (3).  The
 * paper gives the forward only; the adjoint lam = dL/dh is the same affine
 * recurrence run backwards in time (Eq. (6)-(7) with the order reversed):
 *   ds_t = dy_t silu(z_t) (dy_t without z),  lam_t = ds_t Cm_t + a_{t+1} lam_{t+1}
 * and every gradient follows from lam, h and the inputs (see the oracle's
 * documentation for the full list of formulas).
 *
 * Inputs: as for sw_selective_scan_fwd_ex (same dtypes, same flags), plus
 *   dy      : (B, D, L) of dy_dtype (fp32 or bf16), required
 *   dh_last : (B, D, N) fp32 or NULL (zero)
 *   ckpt    : the ckpt of sw_selective_scan_fwd_train on the same inputs,
 *             or NULL (the backward then rebuilds it in its workspace: for
 *             N = 16 where the forward takes its 16-lane layout, with the
 *             forward's walk without y; else in its own kernel; the results
 *             are the same bits either way)
 *   s_pre   : with z, the s_pre of sw_selective_scan_fwd_train on the same
 *             inputs, or NULL (the backward then reruns the forward without
 *             the gate, which also writes the checkpoints when N <= 16);
 *             SW_ERR_INVALID_ARG without z
 * Outputs (fp32, overwritten, never accumulated into):
 *   dx, ddelta : (B, D, L), required; ddelta is with respect to the delta
 *                passed in (before bias and softplus)
 *   dA : (D, N), dB, dC : (B, L, N), required (sums over b, resp. over d)
 *   dDskip, ddelta_bias : (D) or NULL (not written); each is the gradient at
 *                the given value (at zero when the input is NULL)
 *   dz : (B, D, L), or NULL; requires z
 *   dh0 : (B, D, N) or NULL; the gradient with respect to the initial state
 *                (h0, or the zero state when h0 is NULL)
 * With L == 0 (or B*D == 0) the sums are zero and dh0 = dh_last.
 * Results are deterministic: cross-row sums are added in a fixed order.
 * N in [1, 64] (states above 16 run as further passes over the sequence,
 * 16 states each); with ckpt, N <= 16.  A workspace of about
 * (B*D*L*8 without ckpt + B*ceil(D/16)*L*128 + B*D*L*4 if z) bytes is taken from the
 * device's stream-ordered pool for the call.  Other conventions (and
 * errors) as for sw_selective_scan_fwd_ex.
 */
int sw_selective_scan_bwd(const void* x, const void* delta, const float* A, const void* Bm,
                          const void* Cm, const float* Dskip, const void* z,
                          const float* delta_bias, const float* h0, const void* dy,
                          const float* dh_last, const float* ckpt, const float* s_pre,
                          float* dx, float* ddelta,
                          float* dA, float* dB,
                          float* dC, float* dDskip, float* dz, float* ddelta_bias, float* dh0,
                          int64_t B, int64_t D, int64_t N, int64_t L, int in_dtype, int dy_dtype,
                          int flags);

/* Stream used by the calling thread's subsequent calls (a hipStream_t;
 * NULL = the null stream).  Always SW_OK. */
int sw_set_stream(void* hip_stream);
void* sw_get_stream(void);

/* Static text for a status code; never NULL. */
const char* sw_status_string(int status);

/* Message for the calling thread's last non-OK return ("" if none). */
const char* sw_last_error(void);

/*
 * The kernels sw_selective_scan_fwd_ex (train = 0) or
 * sw_selective_scan_fwd_train (train = 1) would enqueue for these sizes and
 * dtypes, with 16-byte aligned arrays, on a part with `cus` compute units
 * (cus <= 0: the current device's), under the same SW_SS_* environment;
 * nothing is launched and no device memory is touched, so with cus > 0 it
 * needs no GPU.  Outputs (all required):
 *   layout : 16 (one lane per state), 4 (four lanes per row, four states
 *            each), 8 (the kernel for any N, which chains its own sequence
 *            chunks), or 0 when there is nothing to launch (B*D or L zero)
 *   nseg, lseg : the row is walked as nseg segments of lseg steps, the last
 *            taking the rest (1 and L: whole rows; 0 and 0 with layout 0)
 *   form   : 0 whole rows, 1 records form, 2 correction form (see
 *            sw_selective_scan_fwd)
 * Errors as the forward call's for the same sizes: SW_ERR_INVALID_ARG
 * (unknown dtype, negative size, NULL output), SW_ERR_UNSUPPORTED (N outside
 * [1, 64], train with N > 16, sizes past the launch limits); SW_ERR_HIP when
 * cus <= 0 and the device cannot be queried.
 */
int sw_selective_scan_plan(int64_t B, int64_t D, int64_t N, int64_t L, int in_dtype,
                           int out_dtype, int train, int cus, int* layout, int64_t* nseg,
                           int64_t* lseg, int* form);

/* Which kernels the calling thread's last successful fused forward or
 * backward call (sw_selective_scan_fwd*, sw_selective_scan_bwd; "" before
 * any) enqueued: for the forward the layout, and for a call split into
 * segments their count, length and form -- e.g. "selective_quad_kernel: 9
 * segments of 7296 steps, correction form (3 launches)"; for the backward
 * where its checkpoints came from.  For tuning and benchmarks; the text is
 * not a stable format. */
const char* sw_last_launch(void);

#ifdef __cplusplus
}
#endif

#endif /* SCANWEAVER_H */
