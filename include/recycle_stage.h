/*
 * recycle_stage.h — C ABI of one pipeline stage's training step with the
 * backward pass decoupled into an input-gradient pass and a deferred
 * weight-gradient pass, after ReCycle (Gandhi et al., SOSP'24).
 *
 * The stage is L pre-LN GPT transformer layers (the paper's evaluation trains
 * Megatron GPT-3 with tensor parallelism 1, Evaluation section, Workloads).
 * The four compute calls follow the paper's statement of the problem:
 *
 *   rc_stage_forward          F of micro-batch (j, k)
 *   rc_stage_backward_input   B_input: gradient w.r.t. the stage input only,
 *                             ready to send upstream at once (Decoupled
 *                             BackProp, section 3.2)
 *   rc_stage_backward_weight  B_weight: gradients w.r.t. the parameters,
 *                             deferred, any order, accumulated over own and
 *                             re-routed micro-batches (sections 3.1, 3.2; the
 *                             WeightGradStore / WeightBackwardPass of section 5)
 *   rc_stage_optimizer_step   this stage's AdamW step, issued on its own with
 *                             no cross-stage synchronisation (Staggered
 *                             Optimizer, section 3.3; AdamW, section 5)
 *
 * Micro-batches are identified as in the op 5-tuple (i, j, k, c, k_s) of the
 * schedule MILP notation (section 4.2.2): the handle is stage i on pipeline
 * k_s; each call names (j, k); c is the call itself.
 *
 * Conventions for every function:
 *  - Returns rc_status; RC_OK == 0.  On failure a message is available from
 *    rc_last_error() (thread-local, valid until the next failing call on
 *    that thread).
 *  - Compute calls are asynchronous with respect to the device: they enqueue
 *    kernels on the handle's HIP stream and return.  Device faults surface as
 *    RC_ERR_HIP at a later call or at rc_stage_synchronize.
 *  - A call that returns an error other than RC_ERR_HIP has enqueued no
 *    device work and left the handle's state unchanged.
 *  - All device memory is supplied by the caller (three arenas sized by
 *    rc_stage_memory_requirements); the library allocates none.
 *  - Several handles per process are allowed (data-parallel peers or
 *    neighbouring stages emulated on one GPU).  A handle must not be used
 *    from two threads at once.
 */
#ifndef RECYCLE_STAGE_H
#define RECYCLE_STAGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rc_status {
  RC_OK = 0,
  RC_ERR_INVALID_ARG = -1,   /* null pointer, bad size, unknown id, misaligned buffer */
  RC_ERR_BAD_STATE = -2,     /* call out of order for this micro-batch / iteration */
  RC_ERR_OUT_OF_STASH = -3,  /* no free stash slot for another forward */
  RC_ERR_HIP = -4,           /* a HIP runtime call or kernel launch failed */
  RC_ERR_UNSUPPORTED = -5    /* shape or option the library does not implement */
} rc_status;

typedef enum rc_dtype {
  RC_FP32 = 0,  /* fp32 storage and arithmetic throughout */
  RC_BF16 = 1   /* bf16 activations / weight copies, fp32 accumulation, fp32 grads, master weights and Adam moments */
} rc_dtype;

/* Shape of the stage.  Requirements (otherwise RC_ERR_UNSUPPORTED):
 *  - hidden % heads == 0; hidden, ffn, seq_len and head_dim = hidden/heads
 *    are multiples of 8;
 *  - bf16 stages: every matrix the matrix-core kernels read through a
 *    buffer descriptor fits its 2^31 - 1 byte range: 2 T max(3 hidden, ffn)
 *    (activation operands, T = micro_batch * seq_len), 2 hidden
 *    max(3 hidden, ffn) (weights) and, without fused attention, 2 seq_len^2
 *    (one head's probabilities).
 * causal = 1 masks keys after the query (GPT). */
typedef struct rc_stage_config {
  int32_t num_layers;
  int32_t hidden;
  int32_t heads;
  int32_t ffn;
  int32_t seq_len;
  int32_t micro_batch;
  int32_t causal;
  int32_t dtype;            /* rc_dtype */
  float ln_eps;             /* LayerNorm epsilon inside the square root */
  int32_t max_stashed_mb;   /* micro-batches that may hold weight-pass intermediates (F..W) at once */
  int32_t max_inflight_mb;  /* micro-batches that may hold forward-only intermediates (F..B) at once; <= max_stashed_mb */
} rc_stage_config;

/* AdamW (Kingma & Ba bias correction, decoupled weight decay).  Weight decay
 * applies to the four linear weight matrices of each layer only. */
typedef struct rc_adam_config {
  float lr, beta1, beta2, eps, weight_decay;
} rc_adam_config;

/* Micro-batch identity: j = id within the iteration, k = original
 * data-parallel pipeline (k != the handle's pipeline_id when re-routed). */
typedef struct rc_mb {
  int32_t j;
  int32_t k;
} rc_mb;

enum { RC_OP_F = 0, RC_OP_B = 1, RC_OP_W = 2, RC_OP_STEP = 3, RC_OP_SKIP = 4, RC_OP_ROLLBACK = 5 };

/* One op-log entry: the op 5-tuple (i=stage, j, k, c=op, k_s) plus the
 * sequence number and the stage-local iteration.  STEP has j = k = -1. */
typedef struct rc_op_record {
  int64_t seq;
  int32_t op;
  int32_t j;
  int32_t k;
  int32_t k_s;
  int32_t stage;
  int32_t reserved;
  int64_t iter;
} rc_op_record;

/* What rc_stage_read copies out (all fp32, the parameter's natural shape). */
enum { RC_READ_PARAM = 0, RC_READ_GRAD = 1, RC_READ_ADAM_M = 2, RC_READ_ADAM_V = 3 };

/* Parameter ids within a layer; linear weights are stored [in, out]
 * (y = x W) and the fused QKV weight [hidden, 3*hidden] has column blocks
 * Q | K | V, head n using columns n*head_dim .. (n+1)*head_dim-1 of each. */
enum {
  RC_P_LN1_G = 0, RC_P_LN1_B = 1, RC_P_W_QKV = 2, RC_P_B_QKV = 3, RC_P_W_O = 4, RC_P_B_O = 5,
  RC_P_LN2_G = 6, RC_P_LN2_B = 7, RC_P_W_1 = 8, RC_P_B_1 = 9, RC_P_W_2 = 10, RC_P_B_2 = 11,
  RC_NUM_PARAMS = 12
};

typedef struct rc_stage rc_stage; /* opaque, library-owned host object */

/* Bytes of the three caller-allocated device arenas:
 *  state: fp32 master weights, fp32 gradients, Adam m and v, bf16 weight copies;
 *  stash: max_stashed_mb weight-pass slots + max_inflight_mb forward-only slots
 *         (the WeightGradStore of section 5; the memory cost the paper names in
 *         section 3.2, "the memory challenge");
 *  work:  per-call scratch reused by every call of the handle.
 * Each arena must be 256-byte aligned.  Pure host function.
 * Errors: RC_ERR_INVALID_ARG (null pointers, inconsistent config),
 *         RC_ERR_UNSUPPORTED (shape outside the requirements above). */
rc_status rc_stage_memory_requirements(const rc_stage_config* cfg, size_t* state_bytes,
                                       size_t* stash_bytes, size_t* work_bytes);

/* Create stage i = stage_index of pipeline k_s = pipeline_id.  The arenas are
 * owned by the caller and must stay valid until rc_stage_destroy; their
 * contents are managed by the library (gradients, m and v are zeroed here,
 * parameters start at zero until loaded).  hip_stream is a hipStream_t (NULL =
 * the null stream); every compute call is enqueued on it.
 * Dry-run handle: pass state_arena == stash_arena == work_arena == NULL.  It
 * performs only the bookkeeping (state machine, stash slots, op log), enqueues
 * nothing and touches no device; it validates op lists on the host.
 * Errors: RC_ERR_INVALID_ARG, RC_ERR_UNSUPPORTED, RC_ERR_HIP. */
rc_status rc_stage_create(const rc_stage_config* cfg, const rc_adam_config* adam,
                          int32_t stage_index, int32_t pipeline_id, void* state_arena,
                          void* stash_arena, void* work_arena, void* hip_stream, rc_stage** out);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): as
 * rc_stage_create, but the work arena is a library-owned array of
 * RC_STATIC_WORK_BYTES in device memory instead of a caller allocation.  Each
 * GPU the library runs on holds one such array from the first use of the
 * library on it until the process ends; the call allocates no device memory.
 * Every handle created this way on one GPU shares that GPU's array, so their
 * calls must not overlap in time (one stream, or ordered by the caller):
 * overlapping calls race on the work memory.  Nothing in it needs to start
 * at zero; it keeps whatever the last call left there.  state_arena and
 * stash_arena are the caller's, as for rc_stage_create (no dry run).  The
 * array belongs to the device that runs hip_stream (NULL: the current device).
 * Errors: RC_ERR_UNSUPPORTED (the configuration needs more work memory than
 *         RC_STATIC_WORK_BYTES, see rc_stage_memory_requirements; device index
 *         above 63), RC_ERR_INVALID_ARG (null arenas, misaligned arenas,
 *         inconsistent config), RC_ERR_HIP. */
#define RC_STATIC_WORK_BYTES (96u * 1024u * 1024u)
rc_status rc_stage_create_static(const rc_stage_config* cfg, const rc_adam_config* adam,
                                 int32_t stage_index, int32_t pipeline_id, void* state_arena,
                                 void* stash_arena, void* hip_stream, rc_stage** out);

/* Waits for the handle's stream, then frees the host object (not the arenas). */
rc_status rc_stage_destroy(rc_stage* st);

/* Copy fp32 host values into parameter (layer, param_id); bf16 weight copies
 * are refreshed (round to nearest even).  Synchronous.  host_src holds the
 * parameter's element count in its natural row-major shape. */
rc_status rc_stage_load_param(rc_stage* st, int32_t layer, int32_t param_id, const float* host_src);

/* Copy parameter / gradient / Adam moment (what = RC_READ_*) of (layer,
 * param_id) to host fp32 memory.  Synchronous (waits for the stream).
 * Gradients are those of the last weight pass, kept until the first weight
 * pass of the next iteration. */
rc_status rc_stage_read(rc_stage* st, int32_t what, int32_t layer, int32_t param_id, float* host_dst);

/* F: y = Stage(x) for micro-batch mb.  x, y: device [micro_batch, seq_len,
 * hidden] row-major in the config dtype; y must not alias x.  The caller owns
 * both and may reuse them once the stream reaches this point.  Takes one
 * stash slot and one forward-only slot.
 * Errors: RC_ERR_BAD_STATE (mb already ran F this iteration),
 *         RC_ERR_OUT_OF_STASH, RC_ERR_INVALID_ARG, RC_ERR_HIP. */
rc_status rc_stage_forward(rc_stage* st, rc_mb mb, const void* x, void* y);

/* B_input: dx = J_x(x)^T dy for micro-batch mb; touches no gradient buffer.
 * dy is copied into the stash; dx may be sent upstream as soon as the stream
 * reaches this point.  Frees the micro-batch's forward-only slot.
 * Errors: RC_ERR_BAD_STATE (mb has not run F, or already ran B),
 *         RC_ERR_INVALID_ARG, RC_ERR_HIP. */
rc_status rc_stage_backward_input(rc_stage* st, rc_mb mb, const void* dy, void* dx);

/* Coupled backward (the conventional reverse pass, B_input and B_weight of
 * mb in one call): dx as rc_stage_backward_input, then mb's gradients as
 * rc_stage_backward_weight; logs a B and a W record.  For micro-batches whose
 * weight pass is not deferred (selective decoupling under a stash limit,
 * section 3.2 "the memory challenge").  Errors: as rc_stage_backward_input. */
rc_status rc_stage_backward(rc_stage* st, rc_mb mb, const void* dy, void* dx);

/* B_weight: add mb's parameter gradients (X^T dY per linear, column sums for
 * biases, sum(dout * xhat) / sum(dout) for LayerNorm) into the fp32 gradient
 * buffers; the first weight pass of an iteration overwrites them.  Any order
 * over micro-batches.  Frees the micro-batch's stash slot.
 * Errors: RC_ERR_BAD_STATE (mb has not run B, or already ran W), RC_ERR_HIP. */
rc_status rc_stage_backward_weight(rc_stage* st, rc_mb mb);

/* B_weight of n micro-batches mbs[0..n) at once (the weight pass is
 * dependence-free once its own B_input ran, so it may be deferred and run in
 * any order and grouping, section 3.2; re-routing leaves the computation, a
 * sum of per-micro-batch gradients, unchanged, section 3.1).  Same result and op-log records as n
 * consecutive rc_stage_backward_weight calls in the given order (fp32 sums
 * in another association order), but each linear's gradient is one product
 * over the n micro-batches' concatenated tokens and each bias / LayerNorm
 * parameter one reduction, so a pass over several deferred micro-batches runs
 * longer, fuller kernels.  mbs: host array of n distinct micro-batches,
 * 1 <= n <= 32; all-or-nothing: no state changes on error.
 * Errors: RC_ERR_INVALID_ARG (n out of range, mbs NULL),
 *         RC_ERR_BAD_STATE (a micro-batch has not run B, already ran W, or is
 *         listed twice), RC_ERR_HIP. */
rc_status rc_stage_backward_weight_many(rc_stage* st, const rc_mb* mbs, int32_t n);

/* AdamW over every parameter of the stage with g = grad_scale * gradient;
 * refreshes the bf16 weight copies; closes the iteration (every micro-batch
 * state is reset, the iteration counter advances).  With no weight pass in
 * the iteration the gradient is zero.
 * Errors: RC_ERR_BAD_STATE (a micro-batch of the iteration has not run W),
 *         RC_ERR_HIP. */
rc_status rc_stage_optimizer_step(rc_stage* st, float grad_scale);

/* Post-step local validation (section 5, the paragraph on bypassing optimizer
 * synchronisation: each stage validates its own gradients after the
 * all-reduce, steps on its own and its upstream stages' results, and rolls
 * back when a downstream stage fails).
 *
 * rc_stage_grad_check: *sumsq = sum of squares of the finite entries of
 * grad_scale * gradient, *nonfinite = number of NaN / Inf entries.  Reads the
 * gradient being accumulated or, while the last call closed an iteration
 * (step / skip / rollback), the gradient that iteration used; zero before
 * the first weight pass of an iteration.  Fixed reduction order (bitwise
 * reproducible).  Synchronises the handle's stream.
 * Errors: RC_ERR_INVALID_ARG (NULL outputs; dry-run handle), RC_ERR_HIP. */
rc_status rc_stage_grad_check(rc_stage* st, float grad_scale, double* sumsq, int64_t* nonfinite);

/* Close the iteration without an update (a failed validation here or
 * upstream): parameters, Adam state and the step count are unchanged; logs
 * RC_OP_SKIP.  Errors: as rc_stage_optimizer_step. */
rc_status rc_stage_optimizer_skip(rc_stage* st);

/* Undo the optimizer step that was this handle's last call (a failed
 * validation downstream).  AdamW is arithmetically reversible: p, m and v
 * before the step are recomputed from their stepped values and the retained
 * gradient, with no saved copy (fp32 rounding: relative error ~1e-7).  The
 * step count goes back by one; the iteration stays closed; logs
 * RC_OP_ROLLBACK with the undone step's iteration.
 * Errors: RC_ERR_BAD_STATE (the last call was not a step, e.g. a second
 * rollback, a skip, or any F/B/W or load_param after the step), RC_ERR_HIP. */
rc_status rc_stage_optimizer_rollback(rc_stage* st);

/* Copy up to cap op-log records into buf (may be NULL when cap == 0); *n
 * receives the total number of records. */
rc_status rc_stage_op_log(rc_stage* st, rc_op_record* buf, int32_t cap, int32_t* n);

/* Stash accounting (the memory change of each op in the schedule MILP,
 * section 4.2.2: F adds the activations kept for the backward pass, B_input
 * swaps them for what the deferred B_weight needs, B_weight frees that).
 * Read as: F +a_f, B_input +(s_w - a_f), B_weight -s_w, coupled backward
 * -a_f.  Byte counts are the logical sizes of the kept tensors (no alignment
 * padding), per micro-batch over all layers:
 *   a_f = L (E (8 T h + 2 T f) + 16 T + attn),  attn = 4 b heads s (fused
 *         attention's row statistics) or E b heads s^2 (probabilities);
 *   s_w = L (E (12 T h + 2 T f) + 16 T);   E = element bytes, T = b s. */
typedef struct rc_stash_account {
  uint64_t a_f;    /* bytes a micro-batch holds from its F to its B_input */
  uint64_t s_w;    /* bytes it holds from its B_input to its B_weight */
  uint64_t live;   /* bytes held by all micro-batches now (between calls) */
  uint64_t peak;   /* maximum of live since create or the last reset */
  uint64_t limit;  /* stash limit, 0 = none */
} rc_stash_account;

/* Fill *out; reset_peak != 0 sets peak = live first.  Works on dry-run handles. */
rc_status rc_stage_stash_account(rc_stage* st, rc_stash_account* out, int32_t reset_peak);

/* Stash limit M_limit (bytes, 0 = none): a forward pass that would raise
 * live above it returns RC_ERR_OUT_OF_STASH with no state change.  Backward
 * calls are never refused; a caller keeps within the limit by running
 * deferred weight passes, or the coupled backward, when deferring would not
 * fit.  Errors: RC_ERR_INVALID_ARG (0 < bytes < a_f). */
rc_status rc_stage_set_stash_limit(rc_stage* st, uint64_t bytes);

/* Number of micro-batches currently holding a stash slot / a forward-only slot. */
rc_status rc_stage_stash_usage(rc_stage* st, int32_t* stashed, int32_t* inflight);

/* Replace the handle's stream (subsequent calls enqueue on it). */
rc_status rc_stage_set_stream(rc_stage* st, void* hip_stream);

/* Kernel classes of the per-kernel profile (the per-op latencies the paper's
 * Profiler collects for its Planner, section 4.1: T_F, T_B_input, T_B_weight,
 * here broken down by kernel). */
enum {
  RC_K_GEMM_FWD = 0,    /* forward linear GEMMs: QKV, out-proj, FC1, FC2 */
  RC_K_GEMM_DGRAD = 1,  /* input-gradient linear GEMMs (B_input) */
  RC_K_GEMM_WGRAD = 2,  /* weight-gradient linear GEMMs (B_weight) */
  RC_K_ATTN_FWD = 3,    /* attention core forward (one region per layer) */
  RC_K_ATTN_BWD = 4,    /* attention core backward (one region per layer) */
  RC_K_LN = 5,          /* LayerNorm forward / input-gradient kernels; the first layer's forward
                           also copies the stage input into the stash, the last layer's LN2
                           backward the upstream gradient */
  RC_K_REDUCE = 6,      /* bias and LayerNorm-affine gradient reductions */
  RC_K_ADAM = 7,        /* fused AdamW */
  RC_K_COPY = 8,        /* separate device copies (none at present: the stash copies of the
                           stage input and upstream gradient ride on the LayerNorm kernels) */
  RC_K_COUNT = 9
};

/* Accumulated profile of one kernel class: number of timed regions, their
 * total device time (HIP events on the handle's stream around each launch or
 * region), and the algorithmic flops and HBM bytes of those regions
 * (operands read + results written once, independent of the kernel design). */
typedef struct rc_kernel_stat {
  int32_t kind;
  int32_t launches;
  double ms;
  double flops;
  double bytes;
} rc_kernel_stat;

/* enable = 1: reset the profile and start recording events around every
 * launch of subsequent calls; enable = 0: stop.  Host-side events only; no
 * device memory.  Errors: RC_ERR_INVALID_ARG (null / dry-run handle), RC_ERR_HIP. */
rc_status rc_stage_profile_enable(rc_stage* st, int32_t enable);

/* Wait for the stream and copy the RC_K_COUNT class profiles into out
 * (out[i].kind == i).  Errors: RC_ERR_INVALID_ARG, RC_ERR_HIP. */
rc_status rc_stage_profile_read(rc_stage* st, rc_kernel_stat* out);

/* Attention kernels the handle's F and B_input run (chosen from the shape
 * and the compute-unit count of the current device):
 *   RC_ATTN_MATERIALISED  scores and probabilities in memory, GEMM + softmax
 *                         kernels (fp32 stages, head_dim != 128);
 *   RC_ATTN_BLOCK         fused online softmax, one workgroup per block of
 *                         128 queries (non-causal, or causal grids that would
 *                         fill the last round of paired workgroups poorly);
 *   RC_ATTN_PAIRED        fused causal, one workgroup per pair of query
 *                         blocks (q, last - q) of equal total length.
 * Host only; works on dry-run handles.  Errors: RC_ERR_INVALID_ARG. */
enum { RC_ATTN_MATERIALISED = 0, RC_ATTN_BLOCK = 1, RC_ATTN_PAIRED = 2 };
rc_status rc_stage_attention_kernels(rc_stage* st, int32_t* kind);

/* Wait for the handle's stream; reports any deferred device error as RC_ERR_HIP. */
rc_status rc_stage_synchronize(rc_stage* st);

/* Message for the last non-OK status on the calling thread ("" if none). */
const char* rc_last_error(void);

/* ---- Schedule side (host only, no device work) ------------------------- */

/* Failure Normalization (section 4.2.1, Algorithm 1): assign `failures`
 * failed workers to pipeline stages so that the estimated extra slots are
 * least; per_stage[i] (length pp) receives the count for stage i, *overhead
 * the estimate.  Per-stage cost of x failures: max(0, 3 mb x - 3 (dp - x)
 * (pp - 1)) (the printed min(0, ...) is read as max); ties go to later
 * stages; at most dp - 1 failures per stage.
 * Errors: RC_ERR_INVALID_ARG (dp < 2, pp < 1, mb < 1, failures < 0 or above
 * pp (dp - 1), NULL outputs). */
rc_status rc_failure_normalization(int32_t dp, int32_t pp, int32_t mb, int32_t failures,
                                   int32_t* per_stage, int64_t* overhead);

#define RC_SIM_MAX_ITER 16

/* Unit-slot schedule simulator of dp data-parallel pipelines of pp stages,
 * mb micro-batches each (sections 3.1-3.3).  F, B_input and B_weight take one
 * slot, a coupled backward two.  Failed workers' micro-batches go round-robin
 * to the alive peers of their stage.  Each worker runs a ready backward first,
 * then a ready forward, then (decoupled) a deferred weight pass, oldest first;
 * ties in (origin pipeline, index) order.  inflight_cap != 0 caps micro-batches
 * between F and B on stage i at pp - i (textbook 1F1B depth).  Iteration n+1
 * starts after every worker finished iteration n, or, staggered, per stage
 * after every worker of that stage did. */
typedef struct rc_sim_config {
  int32_t dp, pp, mb;
  int32_t decoupled;      /* split B into B_input and a deferred B_weight */
  int32_t staggered;      /* per-stage optimizer step */
  int32_t iterations;     /* 1 .. RC_SIM_MAX_ITER */
  int32_t inflight_cap;
  int32_t n_failed;
  const int32_t* failed;  /* n_failed pairs (pipeline k, stage i) */
} rc_sim_config;

typedef struct rc_sim_result {
  int32_t makespan;                  /* slots until the last op ends */
  int32_t workers;                   /* alive workers */
  int32_t busy_max;                  /* most busy slots of any worker */
  int32_t reserved;
  int32_t iter_end[RC_SIM_MAX_ITER]; /* slot at which iteration n's last op ends */
} rc_sim_result;

/* One simulated op: worker (k_s, stage) runs op (RC_OP_F/B/W) of micro-batch
 * (j, origin k) of iteration `iter` in slots [slot, slot + dur). */
typedef struct rc_sim_op {
  int32_t slot, op, iter, stage, j, k, k_s, dur;
} rc_sim_op;

/* Simulate; up to cap ops are written to ops (NULL when cap == 0) in start
 * order, *n_ops receives the total.  Errors: RC_ERR_INVALID_ARG (bad sizes, a
 * stage without an alive worker, a schedule that cannot progress). */
rc_status rc_schedule_simulate(const rc_sim_config* cfg, rc_sim_result* res, rc_sim_op* ops,
                               int32_t cap, int32_t* n_ops);

#ifdef __cplusplus
}
#endif

#endif /* RECYCLE_STAGE_H */
