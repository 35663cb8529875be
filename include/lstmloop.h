/*
 * lstmloop: a device-side, data-dependent LSTM while-loop and its gradient
 * loop for AMD Instinct MI355X (gfx950).
 *
 * What the library computes (Dynamic Control Flow in Large-Scale Machine
 * Learning, Sections 2.1, 4.2, 5.1-5.3, 6.2):
 *
 *   while_loop(pred, body, inits) with pred = (t < T_eff), where
 *   T_eff = max_b seq_len[b] is decided on the GPU (no host round trip per
 *   step); a loop whose predicate is false at entry returns its inits
 *   (Section 4.2).  The body is one LSTM step (textbook cell with forget
 *   gate, gate column blocks i, f, g, o):
 *       z = [x_t, h_{t-1}] W + b;  i,f,o = sigmoid;  g = tanh
 *       c_t = f*c_{t-1} + i*g;     h_t = o*tanh(c_t)
 *   Rows with t >= seq_len[b] keep their state and output y = 0.  The
 *   body can instead be the Elman recurrence h_t = tanh([x_t, h_{t-1}] W + b)
 *   or a GRU step (desc.cell = LL_CELL_RNN / LL_CELL_GRU, below).
 *   Each iteration pushes what the gradient needs onto a stack (Section 5.1);
 *   the gradient loop runs the same number of iterations in reverse, pops
 *   the stack, carries dh/dc as loop variables and sums the gradients of the
 *   loop constants (W, bias) over iterations (Section 5.1).  The gradient of
 *   reading x_t is a write of dx_t (Section 5.2).  The stack can be swapped
 *   out to pinned host memory on copy streams that run beside the compute
 *   stream and prefetched back before the gradient loop needs it
 *   (Section 5.3).
 *
 * Conventions for every entry point
 *   - Array arguments are DEVICE pointers owned by the caller, contiguous,
 *     row-major.  Sequences are time-major: x [T_max,B,I], y/dy [T_max,B,H],
 *     dx [T_max,B,I].  Per-layer arrays are passed as HOST arrays of device
 *     pointers (length = layers).
 *   - W of layer l is [I_l + H, 4H]: rows 0..I_l-1 multiply x_t, rows
 *     I_l..I_l+H-1 multiply h_{t-1}; column blocks are gates i, f, g, o.
 *     I_0 = I, I_1 = H.  Its element type is desc.dtype (float or bfloat16
 *     bits); bias is always float [4H].  (LL_CELL_RNN: 4H reads H here and
 *     below: W [I_l + H, H], bias, dW and dbias [.., H].  LL_CELL_GRU: W and
 *     dW [I_l + H, 3H], bias and dbias [4H].)
 *   - State, stack and accumulation are float32.  In LL_BF16 mode the
 *     matrix-core operands are bfloat16 (round to nearest even): x, W,
 *     h_{t-1} in the forward; dz, [x_t, h_{t-1}] and W in the backward.
 *     Layer 2 reads bf16(y of layer 1).  db sums unrounded dz.
 *   - `stream` is a hipStream_t passed as void*.  Compute calls are
 *     asynchronous on it; they return after enqueueing.
 *   - A plan serves one stream at a time.  Calls on one plan must not
 *     overlap.  The recurrent loops are persistent kernels that need every
 *     compute unit of the device at once: the library chains the loop
 *     launches of all plans on one device (each waits for the previous one to
 *     complete, whichever stream enqueued it), so plans on different streams
 *     are safe.  While all loop launches on a device come from one stream,
 *     stream order does this at no cost; the first loop launch from a
 *     second stream synchronises the device once (host-side), and later
 *     launches order themselves with events.  Other work that holds compute
 *     units for long (another
 *     process's kernels) delays a loop's start (waits are bounded: 5 s, then
 *     LL_DEVERR_BARRIER).  Under graph capture the chain is not used: the
 *     caller orders captured loops itself.
 *   - Every array pointer is 16-byte aligned (the kernels move 16-byte
 *     chunks); lstm_loop_fwd and lstm_loop_bwd return LL_EINVAL otherwise.
 *   - Errors: checkable arguments give an error code synchronously and the
 *     thread-local message of ll_last_error(); nothing is enqueued then.
 *     Data-dependent errors (seq_len outside [0, T_max]) are detected on the
 *     device: the loops then run zero iterations and ll_status_sync()
 *     reports a nonzero device error word.  No exception or abort crosses
 *     this interface.
 */
#ifndef LSTMLOOP_H
#define LSTMLOOP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LL_OK = 0,
  LL_EINVAL = 1,        /* bad argument (null pointer, shape, state)        */
  LL_ENOMEM = 2,        /* device or pinned host allocation failed          */
  LL_EHIP = 3,          /* a HIP runtime call failed                        */
  LL_ESTATE = 4,        /* backward without a matching saved forward        */
  LL_EUNSUPPORTED = 5   /* shape the kernels do not handle (see below)      */
} ll_status;

typedef enum { LL_F32 = 0, LL_BF16 = 1 } ll_dtype;

/* Loop body (cell).  LL_CELL_LSTM: gates i, f, g, o (W [I_l + H, 4H], bias
 * [4H]), state (h, c).  LL_CELL_RNN: the Elman recurrence h_t = tanh(x_t W_x
 * + h_{t-1} W_h + b) (W [I_l + H, H], bias [H]), state h.  LL_CELL_GRU: the
 * gated recurrent unit with the reset gate applied after the recurrent
 * product, column blocks r, u, n (W [I_l + H, 3H]; bias [4H] = b_x [3H],
 * then b_hn [H]):
 *     zx = x_t W_x + b_x,  zh = h_{t-1} W_h
 *     r = sigmoid(zx_r + zh_r),  u = sigmoid(zx_u + zh_u)
 *     n = tanh(zx_n + r * (zh_n + b_hn)),  h_t = (1 - u) n + u h_{t-1}
 * state h; dbias [4H] = [db_x, db_hn].  For both one-state cells c0, cT,
 * dcT and dc0 are ignored (cT and dc0, if given, are written as zeros).
 * LL_CELL_LSTM_SKIP: the LSTM body holding a data-dependent conditional
 * (Section 2.1, cond(pred, true_fn, false_fn)), decided per row and step:
 *     s = (x_t . w_px + h_{t-1} . w_ph) + b_p     (float32 sums of operands)
 *     (h_t, c_t) = s > 0 ? LSTM step : (h_{t-1}, c_{t-1})
 * and y_t = h_t at every valid step.  W is the LSTM's [I_l + H, 4H]; bias
 * [4H + I_l + H + 1] = [b (4H), w_px (I_l), w_ph (H), b_p] (w_p rounded to
 * the operand type like W).  The forward pushes every guard value onto the
 * stack and the gradient loop pops it to run the gradient of the branch
 * taken (Section 5.1, conditionals nested in a loop): the LSTM step's, or
 * the identity.  dbias has the bias's length, zero in the predicate part
 * (a step function has no gradient).  The loop construct, masking, stack and
 * gradient loop are the same for every body: the paper's while-loop and its
 * gradient (Sections 3 and 5) do not depend on it. */
typedef enum {
  LL_CELL_LSTM = 0,
  LL_CELL_RNN = 1,
  LL_CELL_GRU = 2,
  LL_CELL_LSTM_SKIP = 3,
  LL_CELL_LSTM_ACT = 4
} ll_cell;

/* LL_CELL_LSTM_ACT: the LSTM body holding a nested while-loop whose trip
 * count is decided on the device from the state (Section 2.2 motivates it
 * with Adaptive Computation Time; Section 5.1 gives the gradient of nested
 * loops).  For each row still running at step t:
 *     (h, c) = (h_{t-1}, c_{t-1}); P = 0; n = 0
 *     repeat: (h, c) = LSTM step(x_t, h, c); n += 1;
 *             if n == ponder_max: stop
 *             P += sigmoid(h . w_p + b_p)   (float32 sums of operands)
 *             if P >= 1 - eps: stop          (eps = LL_ACT_EPS)
 *     (h_t, c_t) = (h, c); y_t = h_t
 * with the same x_t at every ponder step.  The forward pushes every ponder
 * step's values and the inner trip count of each (step, row tile); the
 * gradient loop runs the nested gradient loop in reverse, popping them.  W
 * is the LSTM's [I + H, 4H]; bias [5H + 1] = [b (4H), w_p (H), b_p]; dbias
 * has the bias's length, zero in the halting part (the halting decision is a
 * step function).  dx_t sums the ponder steps' dz W_x^T.  Single layer,
 * XCD-local loops, no spill or recompute (else LL_EUNSUPPORTED); ACT's
 * mean-field output and ponder cost are not part of this body. */
#define LL_ACT_EPS 0.01f
#define LL_ACT_PONDER_MAX 8

/* Device error word bits (ll_status_sync). */
#define LL_DEVERR_SEQ_LEN 1      /* some seq_len[b] < 0 or > T_max          */
/* a loop wait (grid barrier or exchange flag) exceeded its bound */
#define LL_DEVERR_BARRIER 2

/*
 * Problem description.
 *   T_max, B, I, H >= 1; layers in {1, 2}; dtype an ll_dtype.
 *   Supported tiling: H % 32 == 0, I % 8 == 0 (bf16) or I % 4 == 0 (f32),
 *   B <= 4096; otherwise ll_plan_create returns LL_EUNSUPPORTED.
 *   spill = 0: the stack lives in device memory (T_max*B rows capacity).
 *   spill = 1: the stack is swapped to pinned host memory (Section 5.3):
 *     the loops run one launch per chunk of spill_chunk_steps time steps
 *     (0 = 32; the loop state passes exactly from one launch to the next),
 *     the stack is a device ring of R chunk slots.  Swapping starts only
 *     when the ring is full and nothing is swapped twice: a chunk that a
 *     later chunk evicts from its slot is copied to host memory on the
 *     plan's copy stream after the forward launch that filled it, and
 *     copied back once, ahead of the gradient launches that read it; the
 *     last R chunks never leave the device, so a budget that holds every
 *     chunk moves nothing.  R = device_stack_budget_bytes /
 *     (chunk_steps * B * 5H * 4), at least 3 (0 = 4); the results are
 *     bitwise those of spill = 0.
 *     Needs the XCD-local loops (see ll_plan_geometry); otherwise
 *     ll_plan_create returns LL_EUNSUPPORTED.  The h history, the input
 *     projections and dz stay in device memory.
 *   recompute = 1 (the alternative to spilling; recomputation is the line
 *     of work the paper's related-work section places swapping in): the
 *     forward pushes only
 *     c_t (4 bytes per unit instead of 20); the gradient pass runs one
 *     launch per chunk of spill_chunk_steps steps (0 = 32) and, just before
 *     each, recomputes that chunk's gates i, f, g, o into a device buffer
 *     of one chunk: z = x_t W_x + b + h_{t-1} W_h as two matrix products
 *     over the chunk's rows (h_{t-1} from the h history the dW products use
 *     anyway), then the activations.  The values popped equal the saved ones
 *     up to the summation order of z, so results stay within the parity
 *     tolerance but are not bitwise those of recompute = 0.  Needs the
 *     XCD-local loops and spill = 0 (else LL_EUNSUPPORTED); the two layers
 *     then run one after the other.  The bias passed to lstm_loop_fwd is
 *     copied into the plan for the gradient pass.
 *   reserved: must be 0 (LL_EINVAL otherwise), so that a later field can
 *     take its place without changing what a zero-filled descriptor means.
 *   cell: an ll_cell.  LL_CELL_RNN, LL_CELL_GRU and LL_CELL_LSTM_SKIP need
 *     the XCD-local loops, spill = 0 and recompute = 0 (else
 *     LL_EUNSUPPORTED); the RNN's stack holds h_t only, the GRU's r, u, n,
 *     zh_n + b_hn and h_{t-1}, the cond body's the LSTM's values and one
 *     guard per (step, row).
 */
typedef struct {
  int32_t T_max;
  int32_t B;
  int32_t I;
  int32_t H;
  int32_t layers;
  int32_t dtype;
  int32_t spill;
  int32_t spill_chunk_steps;
  int64_t device_stack_budget_bytes;
  int32_t recompute;
  int32_t cell;
  int32_t ponder_max; /* LL_CELL_LSTM_ACT: at most this many ponder steps per
                         step, 1 .. LL_ACT_PONDER_MAX; 0 for every other cell */
  int32_t reserved;   /* must be 0 (LL_EINVAL otherwise): room for later fields */
} ll_desc;

typedef struct ll_plan ll_plan;   /* opaque: owns the stack, scratch arrays,
                                     pinned host memory, copy streams, events
                                     and the device error word */

/* Validate `desc`, allocate the plan's device stack and scratch memory on
 * `device` (and pinned host memory when spill = 1).  On success *out is a
 * new plan; on failure *out is NULL and nothing stays allocated. */
ll_status ll_plan_create(const ll_desc* desc, int device, ll_plan** out);

/* Free everything the plan owns.  Waits for the plan's outstanding work (the
 * last call's work on its stream, and the plan's own side and copy streams;
 * no device-wide synchronisation).  Call it before the process exits: the HIP
 * runtime may already be torn down inside exit handlers.  NULL is accepted. */
ll_status ll_plan_destroy(ll_plan* plan);

/* Bytes of stack storage the plan holds in device memory and in pinned host
 * memory.  Either output pointer may be NULL. */
ll_status ll_plan_stack_bytes(const ll_plan* plan, int64_t* device_bytes,
                              int64_t* host_bytes);

/* Forms of the recurrent loops (ll_plan_geometry). */
#define LL_LOOPS_GRID 0   /* one grid-wide barrier per step                   */
#define LL_LOOPS_XCD 1    /* each XCD runs its own rows through its own L2    */
#define LL_LOOPS_CHIP 2   /* weights split over all XCDs, per-tile flags      */

/* Launch geometry the plan chose for the recurrent loops (for reports):
 * work-groups per loop launch, hidden units per work-group (the cell units
 * of a work-group in the chip-wide form), row groups (independent
 * recurrences), the loop form (LL_LOOPS_*: XCD-local where one XCD holds the
 * recurrent weights, chip-wide where it cannot (bf16 H = 2048, f32
 * H = 1024, B <= 256), grid-barrier otherwise), and whether a two-layer plan runs its layers
 * as a wavefront (1: one launch per direction runs both layers, the upper
 * layer's step t beside the lower layer's step t+1 (forward) or t-1
 * (gradient); 0: one launch per layer).  Any output may be NULL.
 * Environment variables read at plan creation: LSTMLOOP_LOOPS=grid forces
 * the grid-barrier form; LSTMLOOP_WAVEFRONT=off runs the layers one after
 * the other.  The wavefront needs the XCD-local loops, no spill and
 * 2H / units_per_workgroup <= 32; its results equal the layer-by-layer
 * ones up to the order of floating-point sums.  dw_in_place: bit l set when
 * layer l's dW products read x (or the layer below's h history), the h history
 * and dz in place, row by row (bfloat16 layers whose reduction is short enough
 * for that to be faster and whose operands stay below 2^31 bytes); clear when
 * they read transposed copies. */
ll_status ll_plan_geometry(const ll_plan* plan, int32_t* loop_workgroups,
                           int32_t* units_per_workgroup,
                           int32_t* row_groups, int32_t* loop_form,
                           int32_t* wavefront, int32_t* dw_in_place);

/*
 * Forward while-loop (Sections 2.1, 4.2, 5.1).
 *   x        [T_max,B,I] dtype; entries at t >= seq_len[b] are never read
 *            into a kept result (they may hold NaN).
 *   seq_len  [B] int32, each in [0, T_max].
 *   W, bias  host arrays of `layers` device pointers (see conventions).
 *   h0, c0   [layers,B,H] float, or NULL for zeros.
 *   y        [T_max,B,H] float output of the top layer (0 where t >=
 *            seq_len[b]), or NULL.
 *   hT, cT   [layers,B,H] float: state after seq_len[b] steps (h0/c0 for
 *            zero-length rows).  Required (cT: LSTM only; NULL allowed for
 *            the one-state cells).
 *   trip_count  device int32 scalar receiving T_eff, or NULL.
 *   save_for_backward  nonzero: push the stack for lstm_loop_bwd; the plan
 *            keeps x, seq_len, W, h0, c0 pointers, which must stay valid and
 *            unchanged until the backward has been enqueued (lstm_loop_bwd
 *            takes x, seq_len and W again and checks that they are the same
 *            pointers).
 *            Zero: inference, nothing is saved.
 */
ll_status lstm_loop_fwd(ll_plan* plan, void* stream,
                        const void* x, const int32_t* seq_len,
                        const void* const* W, const float* const* bias,
                        const float* h0, const float* c0,
                        float* y, float* hT, float* cT,
                        int32_t* trip_count, int32_t save_for_backward);

/*
 * Gradient while-loop (Sections 5.1, 5.2): runs T_eff iterations in reverse,
 * popping the stack of the last lstm_loop_fwd(save_for_backward=1) on this
 * plan.  Returns LL_ESTATE if there is none.  Consumes the saved stack.
 *   x, seq_len, W  the same device pointers (W: host array of `layers`
 *            device pointers) as the matching lstm_loop_fwd; the gradient
 *            pass reads x and W again (dW products, dx = dz W_x^T) and the
 *            lengths through the forward's length order.  A pointer that
 *            differs from the saved forward's gives LL_EINVAL; nothing is
 *            enqueued and the saved stack is kept.
 *   dy       [T_max,B,H] float gradient of y, or NULL (zero).
 *   dhT, dcT [layers,B,H] float gradients of hT/cT, or NULL (zero).
 *   dx       [T_max,B,I] float output (0 where t >= seq_len[b]) or NULL.
 *   dW       host array of `layers` device pointers to float [I_l+H,4H];
 *            OVERWRITTEN with the gradient (not accumulated into).
 *   dbias    host array of `layers` device pointers to float [4H];
 *            overwritten.
 *   dh0, dc0 [layers,B,H] float outputs, or NULL.
 */
ll_status lstm_loop_bwd(ll_plan* plan, void* stream,
                        const void* x, const int32_t* seq_len, const void* const* W,
                        const float* dy, const float* dhT, const float* dcT,
                        float* dx, float* const* dW, float* const* dbias,
                        float* dh0, float* dc0);

/*
 * Inference forward without allocation, for callers that cannot allocate
 * device memory or create streams (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): computes exactly what
 * lstm_loop_fwd(plan for *desc, ..., save_for_backward = 0) computes, with the
 * same kernels, but without a plan.  Every buffer the forward needs (length
 * order, transposed weights, input projections, h history, exchange rings and
 * flags) is carved from a scratch array of LL_NOALLOC_SCRATCH_BYTES bytes that
 * the library holds in each device's memory from the moment it is loaded
 * until the process ends.  The call makes no hipMalloc or hipFree, creates no
 * stream or event, and sets up no memory with hipMemset: what must start at
 * zero is cleared by kernels on `stream`.
 *   desc     as for ll_plan_create; spill and recompute must be 0
 *            (LL_EUNSUPPORTED otherwise: nothing is saved).  A problem whose
 *            buffers exceed the scratch array gives LL_EUNSUPPORTED with the
 *            bytes it would need (roughly T_max * B * (4 H * 4 + H * operand
 *            bytes) plus the weights; use a plan for it).
 *   stream   the call's stream; the call runs on the current device.
 *   x .. trip_count  as for lstm_loop_fwd.
 *   device_error  device int32 that receives the device error word
 *            (LL_DEVERR_* bits) at the end of the call, or NULL.
 * Every call on one device shares that device's scratch array and leaves its
 * contents behind: two calls whose work overlaps on one device (different
 * streams, or different threads) race and give wrong results, so callers
 * serialise them (one stream, or their own ordering).  The loops also need
 * the whole device (as for plans): no plan's loop may run beside it.
 */
#define LL_NOALLOC_SCRATCH_BYTES (128ull << 20)
ll_status lstm_loop_fwd_noalloc(const ll_desc* desc, void* stream,
                                const void* x, const int32_t* seq_len,
                                const void* const* W, const float* const* bias,
                                const float* h0, const float* c0,
                                float* y, float* hT, float* cT,
                                int32_t* trip_count, int32_t* device_error);

/* Wait for the plan's work on the stream of its last call, then read and
 * clear the device error word (LL_DEVERR_* bits) into *device_error
 * (may be NULL). */
ll_status ll_status_sync(ll_plan* plan, int32_t* device_error);

/* Message describing the last failure on the calling thread ("" if none). */
const char* ll_last_error(void);

/*
 * Stage timing, for benchmarks.  While enabled, the plan records a pair of
 * HIP events around every stage it enqueues, on the call's stream, so each
 * pair brackets that stage's kernels exactly as the stream runs them.
 * ll_plan_set_timing(plan, 1) clears the accumulators and starts recording
 * every stage; 0 stops.  ll_plan_set_timing_stages records only the stages
 * whose bit (1 << stage) is set in stage_mask (each event pair costs a few
 * microseconds of stream time, so a benchmark times few stages in its timed
 * region); a mask naming no ll_stage is LL_EINVAL.  ll_plan_read_timing waits
 * for the recorded events, then returns the accumulated milliseconds and the
 * number of recorded instances of `stage` (an ll_stage).  Outputs may be
 * NULL.
 */
typedef enum {
  LL_STAGE_PREP = 0,          /* trip count, length order, compact offsets,  */
                              /* and the W transposes in the same launch     */
  LL_STAGE_INPUT_PROJ = 1,    /* x_t W_x + b of all rows                     */
  LL_STAGE_FWD_LOOP = 2,      /* forward recurrence (one launch per layer)   */
  LL_STAGE_BWD_LOOP = 3,      /* gradient recurrence (one launch per layer)  */
  LL_STAGE_BWD_OPERANDS = 4,  /* transposed operands of the dW products      */
  LL_STAGE_DW = 5,            /* dW = sum_t [x_t, h_{t-1}]^T dz_t, db        */
  LL_STAGE_DX = 6,            /* dx_t = dz_t W_x^T (and finished-row zeros)  */
  LL_STAGE_LOOP_SETUP = 7,    /* exchange arrays filled, h0 rows reordered   */
  LL_STAGE_RECOMPUTE = 8,     /* recompute = 1: gates of a chunk recomputed  */
  LL_STAGE_COUNT = 9
} ll_stage;

ll_status ll_plan_set_timing(ll_plan* plan, int32_t enable);
ll_status ll_plan_set_timing_stages(ll_plan* plan, uint32_t stage_mask);
ll_status ll_plan_read_timing(ll_plan* plan, int32_t stage, double* total_ms,
                              int64_t* instances);

/* Diagnostic for reports: the sustained dense matrix-core rate of `device`
 * for `dtype` in TFLOP/s, measured with a kernel in which every wave runs
 * independent MFMA chains on every CU (about 10 ms; synchronous).
 *   shape = 16: the 16x16 k-step the loops use (16x16x32 bfloat16, or four
 *               16x16x4 float instructions);
 *   shape = 32: the 32x32 shape (32x32x16 bfloat16, 32x32x2 float), which on
 *               gfx950 runs at the datasheet rate.
 * Other shape values give LL_EINVAL. */
ll_status ll_measure_mfma_peak(int32_t device, int32_t dtype, int32_t shape, double* tflops);

/* Diagnostic: the cell's activation functions exactly as the loop kernels
 * compute them, applied to n floats on `device` (in, out: device pointers;
 * synchronous).  fn = 0: the logistic sigmoid 1 / (1 + e^-u) of the i, f, o
 * gates; fn = 1: tanh (the g gate, tanh(c_t), the Elman and GRU bodies).  The
 * paper gives no cell equations; these are the textbook LSTM's.  Other fn
 * values or n < 0 give LL_EINVAL. */
ll_status ll_eval_activations(int32_t device, const float* in, float* out, int64_t n, int32_t fn);

/* Library version string. */
const char* ll_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LSTMLOOP_H */
