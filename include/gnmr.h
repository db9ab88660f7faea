/*
 * gnmr.h -- C ABI of libgnmr, the per-step GNMR controller pass on one
 * AMD Instinct MI355X (gfx950).
 *
 * One controller step does, for every monitored unit b (paper notation):
 *   n_{b,t}   = ||g_{b,t}||_2 over all of b's gradient tensors
 *               (Sec. 2, local-gradient equation; Sec. 3.4: a whole block may
 *               be one unit, so a unit may own several tensors),
 *   GNMR, Delta-GNMR, A_{b,t}, Q_b   (Alg. 1; definitions of Sec. 3.1, 3.2),
 *   R_{b,t} = max(GNMR/alpha_t, Delta-GNMR/beta_t)  (Alg. 2; Sec. 3.3),
 *   C_t = {R > 1} U {Lock > 0}, A_t = Top_maxO(C_t; R), lock update
 *               (Alg. 2; Sec. 3.3; Sec. 3.4: maxO is a hard cap on |A_t|).
 *
 * Conventions the paper leaves open, fixed here:
 *   - Top_maxO breaks ties in R by the smaller unit index.
 *   - t is the global step, starting at 1; every step is an observation.
 *   - eps = 0 and a zero Delta-GNMR denominator give Delta-GNMR = 1.
 *   - A non-finite n_{b,t} (outside the paper): GNMR = Delta-GNMR = R = +inf,
 *     A_b is kept, 1.0 enters Q_b, and the unit is counted in n_nonfinite.
 *     The gradient pass sums squares in fp32, whose range ends at 2^128: a
 *     unit whose sum of squares reaches 2^128 (norm >= 2^64) gets n = +inf.
 *     Inf or NaN gradient elements give n = +inf or NaN.
 *   - Units that are monitored but not recoverable get n, GNMR, Delta-GNMR
 *     and R, never enter C_t, and keep Lock = 0.
 *
 * Every call returns a gnmr_status; on an error nothing about the controller
 * state has changed and gnmr_last_error() describes the problem.  Calls on
 * one context must not overlap; different contexts are independent.
 * `stream` arguments are hipStream_t values (NULL = the null stream).
 * "device" pointers are HIP device (or managed) memory of the current device;
 * "host" pointers are ordinary host memory.
 */
#ifndef GNMR_H
#define GNMR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gnmr_ctx gnmr_ctx;

typedef enum {
  GNMR_OK = 0,
  GNMR_E_INVALID = -1, /* bad argument; nothing changed                        */
  GNMR_E_NOMEM = -2,   /* device or host allocation failed                      */
  GNMR_E_HIP = -3,     /* a HIP runtime call failed                             */
  GNMR_E_STATE = -4    /* call not valid in the context's current state          */
} gnmr_status;

/* element types of gradient segments */
enum { GNMR_F32 = 0, GNMR_BF16 = 1 };

/* Budget conventions.  ACTIVE (canonical, Sec. 3.4): maxO caps the active
 * set, |A_t| <= maxO.  ADMITTED (the budget-convention remark of App. C): maxO
 * caps only the newly admitted units; candidates already in A_{t-1} stay
 * active and Top_maxO ranks the remaining candidates, so
 * A_t = (C_t & A_{t-1}) U Top_maxO(C_t minus A_{t-1}; R). */
enum { GNMR_BUDGET_ACTIVE = 0, GNMR_BUDGET_ADMITTED = 1, GNMR_BUDGET_STATIC = 2 };
/* STATIC is the ADAPT-style static baseline of App. E.4: during the first
 * warmup_steps = W >= 1 steps every recoverable unit takes the recovery path
 * and GNMR is recorded; at t = W + 1 the max_o recoverable units with the
 * largest mean GNMR over steps 1..W (ties: smaller index) become the recovery
 * set, fixed from then on.  Locks are not used (Lock stays 0). */

/* Controller settings (Alg. 1 and Alg. 2 inputs that do not change per step). */
typedef struct {
  int32_t num_units;          /* |B| >= 1, monitored units                       */
  int32_t window;             /* delta >= 1, Delta-GNMR window                    */
  int32_t max_o;              /* maxO >= 0, cap on the active recovery set        */
  int32_t lock_len;           /* T_lock >= 0                                      */
  double eps;                 /* epsilon >= 0, finite                              */
  const uint8_t* recoverable; /* host [num_units], nonzero = in B_rec; NULL = all */
  int32_t budget_mode;        /* GNMR_BUDGET_ACTIVE, _ADMITTED or _STATIC           */
  int32_t warmup_steps;       /* W >= 0: for t <= W every recoverable unit takes the
                                 recovery path (high-fidelity warm-up, App. E.6):
                                 C_t = A_t = B_rec, the lock rule of Alg. 2 applies,
                                 GNMR state updates as usual; 0 = none           */
} gnmr_config;

/* Gradient layout: unit b owns segments [unit_seg_off[b], unit_seg_off[b+1]).
 * A segment is a contiguous run of seg_numel[s] elements of type seg_dtype[s]
 * starting at device address seg_ptr[s], which must be aligned to the element
 * size (any other alignment is accepted).  All arrays are host memory and are
 * copied by gnmr_init; the caller may free them afterwards.  Segments may be
 * empty (numel 0) and units may own no segment (their norm is 0). */
typedef struct {
  int64_t num_segments;          /* S >= 0                                       */
  const int64_t* unit_seg_off;   /* host [num_units + 1], [0] = 0, non-decreasing,
                                    [num_units] = S                              */
  const int64_t* seg_numel;      /* host [S], >= 0                                */
  const int32_t* seg_dtype;      /* host [S], GNMR_F32 or GNMR_BF16               */
  const void* const* seg_ptr;    /* host [S] of device pointers, or NULL: then
                                    every gnmr_step / gnmr_sumsq must pass them  */
} gnmr_segments;

/* Per-step counters (trigger sparsity, promotion and hit-maxO rates of the
 * paper's trigger-overhead measurements).  Counts are over recoverable units,
 * except n_nonfinite, which is over all units. */
typedef struct {
  int64_t t;             /* step just completed (1-based)                          */
  int32_t n_trig_gnmr;   /* #{GNMR/alpha_t > 1}                                    */
  int32_t n_trig_dgnmr;  /* #{Delta-GNMR/beta_t > 1}                               */
  int32_t n_trig;        /* #{R > 1}                                               */
  int32_t n_cand;        /* |C_t|                                                  */
  int32_t n_active;      /* |A_t| (<= maxO under GNMR_BUDGET_ACTIVE)               */
  int32_t hit_maxo;      /* 1 if the ranked pool (C_t, or C_t minus A_{t-1} under
                            GNMR_BUDGET_ADMITTED) is non-empty and >= maxO; 0 in
                            the warm-up                                           */
  int32_t n_nonfinite;   /* units with a non-finite norm                           */
  int32_t reserved;
} gnmr_stats;

/* Create a controller for the inputs of Alg. 1 (delta, eps) and Alg. 2
 * (B_rec, maxO, T_lock) and the units of Sec. 3.4: t = 0, A = 0, Q empty,
 * Lock = 0 (the state before the first step of Alg. 1 / Alg. 2).  Allocates
 * all device state (O(U * delta) doubles plus one float per 64 KiB work
 * item) and builds the work list over
 * the segments: each segment takes one item per started 64 KiB, at most
 * 16,777,215 items in all (the most one launch's grid can hold), and
 * seg_numel <= 2^50; GNMR_E_INVALID beyond.  `stream` orders the initial
 * clears.  *out receives the context, or NULL on error. */
gnmr_status gnmr_init(gnmr_ctx** out, const gnmr_config* cfg,
                      const gnmr_segments* segs, void* stream);

/* Release every resource of the context (waits for its pending work).
 * NULL is accepted and ignored. */
gnmr_status gnmr_destroy(gnmr_ctx* ctx);

/* One full controller step t -> t + 1: the gradient norm of every unit
 * (Sec. 2), Alg. 1 for every unit, then Alg. 2: reads every gradient byte
 * once, then updates A, Q, Lock and the outputs.
 * alpha_t, beta_t > 0 and finite (values below 1 are legal).  seg_ptr: host
 * [S] of device pointers for this step, or NULL to reuse the last bound ones.
 * Asynchronous: only enqueues work on `stream`.  The gradient buffers must
 * stay valid and unmodified until that work is done.
 * HIP graphs: with seg_ptr == NULL (pointers bound before) and profiling off,
 * a step enqueues kernels only (no allocation, copy or memset) and can be
 * captured; the step counter lives on the device, so every replay performs
 * the next step.  alpha_t and beta_t are fixed at capture time. */
gnmr_status gnmr_step(gnmr_ctx* ctx, double alpha_t, double beta_t,
                      const void* const* seg_ptr, void* stream);

/* Alg. 1 and Alg. 2 with the norms n_{b,t} given (the gradient norm of
 * Sec. 2 computed by the caller): d_norm is device [num_units] float64
 * n_{b,t}; the gradient pass is skipped.  For callers that already hold the
 * norms (and for testing the state update and selection alone).  Capturable
 * in a HIP graph like gnmr_step. */
gnmr_status gnmr_step_from_norms(gnmr_ctx* ctx, const double* d_norm,
                                 double alpha_t, double beta_t, void* stream);

/* The gradient pass alone (Sec. 2, local-gradient equation, squared: the
 * sum of squares over all of a unit's tensors), without touching controller
 * state: writes sum_i g_i^2 per unit (float64, device [num_units]) to
 * d_sumsq, the float64 sum of the fp32 item partials (no range limit
 * applied).  seg_ptr as in gnmr_step.  Asynchronous. */
gnmr_status gnmr_sumsq(gnmr_ctx* ctx, const void* const* seg_ptr,
                       double* d_sumsq, void* stream);

/* The gradient pass of gnmr_sumsq for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): no context, and no allocation, free or allocating
 * library call.  The work list and the item partials live in a fixed device
 * array of the library, GNMR_NOALLOC_SCRATCH_BYTES (32 MiB) per device, held
 * from the first call on a device until the process ends.  segs describes the
 * gradients as for gnmr_init, with seg_ptr required (host [S] of device
 * pointers); the same checks apply.  Writes the same float64 sums of squares
 * as gnmr_sumsq over the same layout, bit for bit, to d_sumsq (device
 * [num_units]).  A layout whose work list and partials do not fit the array
 * (about 1.6 million 64 KiB items, some 100 GB of gradients) is refused with
 * GNMR_E_INVALID.  Enqueues an upload of the work list and two kernels on
 * `stream`, then waits for `stream` (the host copy of the work list must
 * outlive the upload).  All calls on one device share its array: calls that
 * overlap (on different streams or threads) race; calls on one stream are
 * ordered. */
#define GNMR_NOALLOC_SCRATCH_BYTES (32u << 20)
gnmr_status gnmr_sumsq_noalloc(int32_t num_units, const gnmr_segments* segs, double* d_sumsq,
                               void* stream);

/* ---- producer-fused gradient pass (the norm from the weight-gradient GEMM) --
 *
 * The controller takes one number per unit from the gradient: its norm
 * (Alg. 1; Sec. 3.3).  The producer of a linear layer's weight gradient
 * holds every value of it in registers before writing it, so it can emit the
 * sum of squares itself and the gradient pass (K1) never re-reads the
 * gradient from HBM.
 *
 * gnmr_wgrad_sumsq: the weight-gradient GEMM of a linear layer y = x W^T,
 *   dw[o][i] = bf16_rne( sum_t dy[t][o] * x[t][i] )     (fp32 accumulation)
 * dy: device [tokens][out_features] bf16, x: device [tokens][in_features]
 * bf16, dw: device [out_features][in_features] bf16, all row-major and
 * 16-byte aligned; out_features and in_features multiples of 8 below 2^24;
 * tokens >= 0 (0 gives dw = 0).  tile_sumsq: device float [gnmr_wgrad_num_tiles(out,
 * in)], written with the fp32 sum of float(dw)^2 over each 256x256 output
 * tile (row-major tile order, ragged edge tiles included), each in a fixed
 * order: deterministic.  The caller owns every buffer; dw and tile_sumsq
 * must overlap neither each other nor dy or x (checked).  Asynchronous on
 * `stream`.  GNMR_E_INVALID on a bad shape, pointer, alignment or overlap,
 * GNMR_E_HIP on a launch failure. */
int64_t gnmr_wgrad_num_tiles(int32_t out_features, int32_t in_features);
gnmr_status gnmr_wgrad_sumsq(const void* dy, const void* x, void* dw, int64_t tokens,
                             int32_t out_features, int32_t in_features,
                             float* tile_sumsq, void* stream);

/* Several weight-gradient GEMMs (e.g. the seven projections of a decoder
 * layer) in one launch, so that their tiles share the machine: each problem
 * as in gnmr_wgrad_sumsq; problem i's tile sums start at tile_sumsq + the
 * tile counts of problems 0..i-1 (the layout gnmr_bind_partials expects with
 * one unit per problem).  A problem with accumulate = 1 adds its product to
 * the gradient already stored in dw (gradient accumulation over
 * micro-batches): dw = bf16_rne(fp32(dw + product)), one fp32 addition and
 * one rounding to bf16, and its tile sums are those of the accumulated dw.
 * `problems` is a host array, read before return; every check of
 * gnmr_wgrad_sumsq applies to each problem (and accumulate is 0 or 1,
 * reserved 0); across the batch no dw may overlap another problem's dw, dy
 * or x, or tile_sumsq (operands may be shared between problems: the seven
 * projections read three inputs).  Nothing is launched if a check fails.
 * The overwriting and the accumulating problems of a batch run as separate
 * launches (one kernel instance per kind), in that order. */
typedef struct {
  const void* dy;        /* device [tokens][out_features] bf16 */
  const void* x;         /* device [tokens][in_features] bf16  */
  void* dw;              /* device [out_features][in_features] bf16 */
  int64_t tokens;
  int32_t out_features;
  int32_t in_features;
  int32_t accumulate;    /* 0: dw = product; 1: dw += product */
  int32_t reserved;      /* 0 */
} gnmr_wgrad_problem;
gnmr_status gnmr_wgrad_sumsq_batched(const gnmr_wgrad_problem* problems,
                                     int32_t num_problems, float* tile_sumsq,
                                     void* stream);

/* Declare where a producer writes the units' partial sums of squares: unit b
 * owns partials [unit_part_off[b], unit_part_off[b+1]) of a float array of
 * num_partials (host array of num_units + 1, non-decreasing, [0] = 0, last =
 * num_partials; copied).  Waits for the device; may be called again to
 * re-bind.  GNMR_E_INVALID on a bad layout. */
gnmr_status gnmr_bind_partials(gnmr_ctx* ctx, int64_t num_partials,
                               const int64_t* unit_part_off);

/* One controller step (K2 + K3) from the bound partials: n_b = sqrt of the
 * float64 sum, in a fixed order, of unit b's partials in d_partial (device
 * float [num_partials], e.g. the tile_sumsq of gnmr_wgrad_sumsq calls laid
 * end to end), then Alg. 1 and Alg. 2 exactly as gnmr_step.  Asynchronous;
 * capturable in a HIP graph.  GNMR_E_STATE if no layout is bound. */
gnmr_status gnmr_step_from_partials(gnmr_ctx* ctx, const float* d_partial,
                                    double alpha_t, double beta_t, void* stream);

/* The outputs of Alg. 1 and Alg. 2 for the last step: A_t as a mask, the lock
 * counters, n_{b,t}, GNMR, Delta-GNMR (Alg. 1) and R (Alg. 2), and the step's
 * counters.  Copies them to host memory; every destination may be NULL.
 * Waits for `stream`.  Arrays are [num_units]: mask (1 = in A_t, recovery
 * path), lock (Lock_b after the step), norm (n_{b,t}), gnmr, dgnmr, risk (R).
 * GNMR_E_STATE before the first step. */
gnmr_status gnmr_query(gnmr_ctx* ctx, uint8_t* mask, int32_t* lock, double* norm,
                       double* gnmr, double* dgnmr, double* risk,
                       gnmr_stats* stats, void* stream);

/* The same outputs of Alg. 1 and Alg. 2, zero-copy: their device addresses
 * (owned by the context, valid until gnmr_destroy, overwritten by the next
 * step; the mask can drive the actuator directly).  Any pointer may be NULL. */
gnmr_status gnmr_device_outputs(gnmr_ctx* ctx, const uint8_t** mask,
                                const int32_t** lock, const double** norm,
                                const double** gnmr, const double** dgnmr,
                                const double** risk, const gnmr_stats** stats);

/* The state of Alg. 1 and Alg. 2 (t, A, Q, Lock; A_{t-1}; the static
 * baseline's GNMR sums) as a flat, versioned byte blob, for checkpoint and
 * resume (outside the paper: resume).  gnmr_state_size gives the blob size;
 * get copies it to host `buf` of `bytes` >= that size (waits for `stream`);
 * set restores a blob taken from a context with the same num_units, window,
 * max_o, lock_len, eps, budget_mode and warmup_steps (GNMR_E_INVALID
 * otherwise, nothing changed).  Restoring and then stepping reproduces the
 * original run bit for bit.  The per-step outputs are not part of the state:
 * after a restore gnmr_query returns GNMR_E_STATE until the next step. */
gnmr_status gnmr_state_size(const gnmr_ctx* ctx, size_t* bytes);
gnmr_status gnmr_get_state(gnmr_ctx* ctx, void* buf, size_t bytes, void* stream);
gnmr_status gnmr_set_state(gnmr_ctx* ctx, const void* buf, size_t bytes, void* stream);

/* Kernel timing.  While enabled, every step records HIP events around each of
 * its kernels on its stream.  gnmr_profile_read waits for them and returns the
 * summed milliseconds of the gradient pass, the state update and the
 * selection kernels over the steps recorded since enabling, and that number of
 * steps; any output may be NULL.  Enabling resets the sums. */
gnmr_status gnmr_set_profiling(gnmr_ctx* ctx, int enable);
gnmr_status gnmr_profile_read(gnmr_ctx* ctx, double* ms_sumsq, double* ms_update,
                              double* ms_select, int64_t* steps);

/* Work-list facts: K1 work items, bytes per item, gradient bytes per step and
 * kernel launches per gnmr_step.  Any output may be NULL. */
gnmr_status gnmr_info(const gnmr_ctx* ctx, int64_t* num_items, int64_t* item_bytes,
                      int64_t* bytes_per_step, int32_t* launches_per_step);

/* ---------------------------------------------------------------------------
 * Recovery actuator: routes each unit's saved activations to the low-cost or
 * the recovery path chosen by the controller (Alg. 2: "use the recovery path
 * for b" / "use the low-cost path").  Both paths are per-token fake
 * quantisation (App. E.2 quantisation-simulated operators; Sec. 5.1 and App.
 * E.4: token-wise low-bit saved activations; Sec. 5.3 and App. E.3: INT8): every token (row) is scaled into
 * the format's representable range by its largest magnitude, rounded to the
 * nearest representable value (ties to the even significand or integer,
 * saturating) and rescaled, in fp32: inv = fmax / amax, s = amax / fmax, y = x * inv,
 * out = bf16_rne(round(y) * s), signs kept; an all-zero token becomes +0.
 * GNMR_FMT_BF16 leaves the row unchanged.
 * ------------------------------------------------------------------------- */
enum {
  GNMR_FMT_BF16 = 0,  /* identity (the BF16 path)                      */
  GNMR_FMT_E2M1 = 1,  /* 4-bit, max 6                                  */
  GNMR_FMT_E3M2 = 2,  /* 6-bit, max 28                                 */
  GNMR_FMT_E4M3 = 3,  /* 8-bit, max 448                                */
  GNMR_FMT_E5M2 = 4,  /* 8-bit, max 57344                              */
  GNMR_FMT_INT8 = 5   /* symmetric integer grid -127 .. 127 (Sec. 5.3, App.
                         E.3: the INT8 low-cost path); rint, ties to even  */
};

/* One unit's saved activations: a row-major bf16 [rows][cols] matrix, one
 * row per token. */
typedef struct {
  const void* in;   /* device, 16-byte aligned                                  */
  void* out;        /* device, 16-byte aligned; equal to `in` (in place) or not
                       overlapping any segment's input; no two segments' outputs
                       overlap, and no segment's input is another's output (all
                       checked by gnmr_actuator_create)                          */
  int64_t rows;     /* tokens, >= 0                                             */
  int32_t cols;     /* features: a multiple of 8, 8 .. 16384                     */
  int32_t unit;     /* controller unit whose mask entry picks the format, 0 .. U-1 */
} gnmr_act_segment;

typedef struct gnmr_actuator gnmr_actuator;

/* Build the row work list over the segments (host array, copied; the caller
 * may free it).  num_units bounds the unit indices.  Allocates device memory
 * for the tables (8 B per row, 24 B per segment).  At most 67,108,860 rows of
 * up to 4096 features and 16,777,215 longer rows in all (the most one
 * launch's grid can hold); GNMR_E_INVALID beyond. */
gnmr_status gnmr_actuator_create(gnmr_actuator** out, const gnmr_act_segment* segs,
                                 int64_t num_segments, int32_t num_units, void* stream);

/* Apply the formats: rows of unit b use fmt_recovery when d_mask[b] != 0 (b in
 * A_t), else fmt_low.  d_mask: device [num_units] (for example the mask from
 * gnmr_device_outputs).  Asynchronous on `stream`.  A BF16 row in place is not
 * touched (no memory traffic). */
gnmr_status gnmr_actuate(gnmr_actuator* act, const uint8_t* d_mask, int32_t fmt_low,
                         int32_t fmt_recovery, void* stream);

/* One activation matrix without a row table (the rows of one segment
 * passed by value): the same per-token quantisation, for callers whose
 * buffers change every call, such as the input of one linear layer inside a
 * forward pass.  in: device bf16 [rows][cols], row-major, 16-byte aligned;
 * out: equal to `in` (in place) or not overlapping it, 16-byte aligned; cols
 * a multiple of 8 in [8, 16384]; 0 <= rows <= 67,108,860 (cols <= 4096) or
 * 16,777,215 (longer rows), the most one launch's grid can hold; the matrix takes
 * fmt_recovery when d_mask[unit] != 0, else fmt_low (d_mask: device bytes,
 * e.g. the controller's mask from gnmr_device_outputs, read when the kernel
 * runs).  Allocates nothing and launches one kernel (none when rows = 0);
 * asynchronous on `stream`.  GNMR_E_INVALID on a bad argument, GNMR_E_HIP on
 * a launch failure. */
gnmr_status gnmr_actuate_matrix(const void* in, void* out, int64_t rows, int32_t cols,
                                const uint8_t* d_mask, int32_t unit, int32_t fmt_low,
                                int32_t fmt_recovery, void* stream);

/* Rows in the work list and bf16 bytes of all segments' inputs. */
gnmr_status gnmr_actuator_info(const gnmr_actuator* act, int64_t* rows, int64_t* bytes);

gnmr_status gnmr_actuator_destroy(gnmr_actuator* act);

/* Message of the last failed call on this thread ("" if none). */
const char* gnmr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GNMR_H */
