/*
 * lamb_mi355x.h -- C ABI of the multi-tensor LAMB / LARS optimizer step for
 * AMD Instinct MI355X (gfx950).
 *
 * Method: You et al., "Large Batch Optimization for Deep Learning: Training
 * BERT in 76 minutes" (arXiv:1904.00962). LAMB is Algorithm 2 (Section 3.2),
 * LARS is Algorithm 1 (Section 3.1); the scaling function
 * phi(z) = min(max(z, gamma_l), gamma_u) is defined in Section 3, and a
 * "layer" x^(i) is one block of the parameter vector (Section 2, Notation),
 * here one tensor of the table.
 *
 * Conventions for every entry point:
 *  - Tensor pointers are DEVICE pointers on the device that is current when
 *    the plan is created; host arrays are marked "host".
 *  - All state (x, g, m, v) is owned by the caller. The plan owns only its
 *    own small device buffers (tensor and chunk tables, per-chunk partial
 *    sums, per-tensor step scales), allocated in lamb_plan_create and freed
 *    in lamb_plan_destroy.
 *  - Arguments are validated on the host before any HIP call. A call that
 *    fails validation returns a negative lamb_status, launches nothing and
 *    changes no state. lamb_last_error() then describes the failure.
 *  - Step calls enqueue work on `stream` (a hipStream_t; NULL = the null
 *    stream) and return without synchronising, allocating (beyond one HIP
 *    event per device, created by the first single-pass step) or copying to
 *    the host. Device faults surface at the caller's next synchronisation.
 *    A step that returns LAMB_EHIP after validation may already have
 *    enqueued the kernels before the failed launch, so the state of that
 *    step is then undefined.
 *  - One step may be in flight per plan (its partials buffer is reused);
 *    a plan is not thread-safe. Distinct plans are independent.
 *  - NaN and Inf in the inputs propagate by IEEE rules; nothing is masked.
 */
#ifndef LAMB_MI355X_H
#define LAMB_MI355X_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Entry points are the only symbols the shared library exports. */
#if defined(__GNUC__) || defined(__clang__)
#define LAMB_API __attribute__((visibility("default")))
#else
#define LAMB_API
#endif

typedef enum lamb_status {
    LAMB_OK = 0,
    LAMB_EINVAL = -1,   /* a size or scalar is outside its documented range  */
    LAMB_ENULL = -2,    /* a required pointer is NULL                         */
    LAMB_EALIGN = -3,   /* a tensor pointer is not 16-byte aligned            */
    LAMB_EOVERLAP = -4, /* two tensor buffers of the table overlap            */
    LAMB_EHIP = -5,     /* a HIP runtime call failed                          */
    LAMB_ENOMEM = -6,   /* a host or device allocation failed                 */
    LAMB_EPLAN = -7,    /* the plan was built for the other algorithm         */
    LAMB_ESYNC = -8     /* a single-pass step abandoned a wait (lamb_plan_check) */
} lamb_status;

typedef enum lamb_grad_dtype {
    LAMB_GRAD_F32 = 0,  /* g is float                                         */
    LAMB_GRAD_BF16 = 1  /* g is bfloat16 (raw 16-bit patterns), widened exactly */
} lamb_grad_dtype;

typedef enum lamb_algo {
    LAMB_ALGO_LAMB = 0, /* Algorithm 2: needs m and v                          */
    LAMB_ALGO_LARS = 1  /* Algorithm 1: needs m only; v is ignored            */
} lamb_algo;

/*
 * One layer block x^(i) (Section 2). Every buffer holds `numel` contiguous
 * elements (1 to 2^40) and is 16-byte aligned; no two buffers of a table may
 * overlap.
 *   x  fp32 parameters, updated in place
 *   g  gradient g_t (fp32 or bf16, fixed per plan), read only
 *   m  fp32 first moment (LAMB) / momentum (LARS), updated in place; start at 0
 *   v  fp32 second moment (LAMB), updated in place; start at 0. NULL for LARS.
 *   wd weight-decay mask: 1 applies lambda to this block, 0 uses lambda = 0
 */
typedef struct lamb_tensor {
    float *x;
    const void *g;
    float *m;
    float *v;
    int64_t numel;
    int32_t wd;
    int32_t reserved; /* must be 0 */
} lamb_tensor;

typedef struct lamb_plan lamb_plan; /* opaque */

/* Which algorithm a step runs (lamb_step_ex). */
typedef enum lamb_variant {
    LAMB_VARIANT_LAMB = 0,   /* Algorithm 2 (Section 3.2)                      */
    LAMB_VARIANT_NLAMB = 1,  /* Algorithm 3, N-LAMB (Appendix D)               */
    LAMB_VARIANT_NNLAMB = 2, /* Algorithm 4, NN-LAMB (Appendix D)              */
    LAMB_VARIANT_LARS = 3    /* Algorithm 1 (Section 3.1); needs a LARS plan   */
} lamb_variant;

/* Layer norm used for ||x_i|| and for the update's ||u_i|| (Appendix F: L2
 * is the paper's default; it does not name the others it tried). */
typedef enum lamb_norm {
    LAMB_NORM_L2 = 0,   /* sqrt(sum a^2)                                      */
    LAMB_NORM_L1 = 1,   /* sum |a|                                            */
    LAMB_NORM_LINF = 2  /* max |a| (a NaN element makes it NaN)               */
} lamb_norm;

/*
 * How a plan's direct-mode steps (skip_nonfinite = 0) run.
 *  LAMB_PATH_AUTO      (default) every layer of at most 4 * (compute units)
 *                      tiles takes one single-pass kernel that reads x, g,
 *                      m, v and writes x, m, v once: a persistent grid keeps
 *                      each tile's x and update direction on chip while the
 *                      layer's norms are combined. A tile holds 8192
 *                      elements, or 10240 when that puts more whole layers'
 *                      parameters on the single pass (lamb_tile_schedule):
 *                      one round holds 8M or 10M elements on MI355X. The
 *                      environment variable LAMB_MI355X_TILE_GROUPS (8 or
 *                      10), read by lamb_plan_create, fixes the tile instead;
 *                      tests use it to run the wider tile on small layers
 *                      (any other value fails with LAMB_EINVAL). A larger
 *                      layer puts its last elements on the single pass (as
 *                      many tiles as the plan's largest whole layer takes,
 *                      or one round when no whole layer is on it; its head
 *                      ends at a multiple of 1024 elements) and its head on
 *                      the two-pass kernels: a moment pass and a totals
 *                      kernel before the single pass, which adds the head's
 *                      partial norms into the layer's, and an apply pass
 *                      after it. Needs the device's full occupancy
 *                      for the length of that kernel: the library runs the
 *                      single-pass kernels of one process one at a time
 *                      (a step on another stream than the previous one
 *                      waits for it); steps of other processes on the same
 *                      device, or replays of captured graphs that overlap
 *                      another single-pass kernel, may stall until a wait
 *                      gives up (lamb_plan_check).
 *  LAMB_PATH_TWO_PASS  every layer takes the two-pass kernels: a moment pass
 *                      that reads x, g, m, v and writes m, v; a per-layer
 *                      finalize; an apply pass that reads x, m, v (and g for
 *                      N-LAMB / NN-LAMB) and writes x.
 * skip_nonfinite = 1 on LAMB_PATH_AUTO (with any layer on the single pass)
 * first reads every g once to take the step's verdict, then runs the same
 * kernels as a direct step, which change nothing when the verdict is
 * raised; the single pass reports the verdict (the heads' apply pass after
 * it reads a copy the totals kernel took). On
 * LAMB_PATH_TWO_PASS it takes the deferred two-pass kernels: a read-only
 * moment pass, then an apply pass that writes x, m, v unless the verdict
 * is raised.
 * Both paths give the same m and v bit for bit; the layer norms are summed
 * in a different order, so ratios and x agree to rounding.
 */
typedef enum lamb_path {
    LAMB_PATH_AUTO = 0,
    LAMB_PATH_TWO_PASS = 1
} lamb_path;

/*
 * Hyperparameters of one step (lamb_step_ex). lamb_hparams_init fills the
 * paper's defaults for a variant; change fields afterwards.
 *   variant          lamb_variant
 *   norm             lamb_norm
 *   step             t >= 1 (LAMB family; ignored by LARS)
 *   lr               eta_t, finite
 *   beta1            LAMB family beta1, LARS momentum; in [0, 1)
 *   beta2, eps       LAMB family: beta2 in [0, 1), eps finite >= 0
 *   weight_decay     lambda, finite; applied where the tensor's wd mask is 1
 *   gamma_l, gamma_u phi's clamp, 0 <= gamma_l <= gamma_u (gamma_u may be inf)
 *   trust_coef       LARS only: ratio = trust_coef * phi / ||m||, finite
 *   grad_scale       every gradient element is multiplied by it first, so the
 *                    caller can hand over a sum of per-sample gradients (the
 *                    1/|S_t| of Algorithms 1-2) or a loss-scaled gradient;
 *                    finite
 *   bias_correction  LAMB only: 1 (Algorithm 2) or 0 (Appendix E); must be 1
 *                    for N-LAMB and NN-LAMB
 *   skip_nonfinite   1: if any scaled gradient element (computed in fp32) of
 *                    any tensor is NaN or infinite, the step leaves every x,
 *                    m, v unchanged. The moment pass then writes nothing and
 *                    the apply pass recomputes and writes x, m, v together,
 *                    which costs 2 more bytes per parameter (bf16 g) or 4
 *                    (fp32 g). 0: no check, moments are written in the first
 *                    pass. The ratio and norm outputs of a skipped step are
 *                    unspecified.
 */
typedef struct lamb_hparams {
    int32_t variant;
    int32_t norm;
    int64_t step;
    float lr;
    float beta1;
    float beta2;
    float eps;
    float weight_decay;
    float gamma_l;
    float gamma_u;
    float trust_coef;
    float grad_scale;
    int32_t bias_correction;
    int32_t skip_nonfinite;
    int32_t reserved; /* set to 0 (lamb_hparams_init does) */
} lamb_hparams;

/*
 * Build a plan for a fixed table of blocks (Section 2's decomposition of x).
 * The table is copied; the tensor pointers must stay valid and unchanged for
 * the plan's life (rebuild the plan if the buffers move).
 *   tensors      host array of n_tensors descriptors, n_tensors >= 1
 *   g_dtype      dtype of every g, a lamb_grad_dtype value
 *   algo         which step the plan serves, a lamb_algo value
 * (The enum parameters travel as int32_t so that any value a caller passes
 * is well defined and rejected with LAMB_EINVAL when out of range.)
 *   chunk_elems  elements per work chunk: 0 picks the default, otherwise a
 *                multiple of 8 in [8, 2^30]. Results are deterministic for a
 *                given chunk size and agree across sizes to rounding.
 *   out          receives the plan
 * Errors: LAMB_ENULL (tensors/out/x/g/m, or v for LAMB), LAMB_EINVAL (sizes,
 * dtype, algo, reserved != 0, or a device whose round of single-pass tiles
 * would exceed 2^29 elements, which the kernel's 32-bit offsets cannot
 * address), LAMB_EALIGN, LAMB_EOVERLAP, LAMB_ENOMEM, LAMB_EHIP (device
 * allocation or copy failed).
 */
LAMB_API lamb_status lamb_plan_create(const lamb_tensor *tensors, int32_t n_tensors,
                             int32_t g_dtype, int32_t algo,
                             int32_t chunk_elems, lamb_plan **out);

/* Free the plan's device buffers. NULL is accepted. Waits for nothing: the
 * caller must not destroy a plan whose step is still running. */
LAMB_API lamb_status lamb_plan_destroy(lamb_plan *plan);

/*
 * Attach bf16 working copies of the parameters (for the next forward pass of
 * mixed-precision training): every later step's apply pass also writes
 * copy_i[j] = bf16(x_i[j]) after the update, rounded to nearest with ties to
 * even (NaN becomes 0x7fc0), at 2 more bytes per parameter instead of a
 * separate cast pass.
 *   copies  host array of n_tensors device pointers to numel bf16 each,
 *           16-byte aligned, overlapping no buffer of the plan or each other;
 *           an entry may be NULL (no copy for that tensor); copies = NULL
 *           detaches all.
 * Copies a table to the device synchronously; do not call while a step runs.
 * Errors: LAMB_ENULL (plan), LAMB_EALIGN, LAMB_EOVERLAP, LAMB_EHIP.
 */
LAMB_API lamb_status lamb_plan_set_bf16_copies(lamb_plan *plan, void *const *copies);

/* Sizes of a plan (host outputs; any may be NULL). */
LAMB_API lamb_status lamb_plan_info(const lamb_plan *plan, int32_t *n_tensors,
                           int32_t *n_chunks, int32_t *chunk_elems);

/* Select the plan's path (lamb_path) for later steps. Errors: LAMB_ENULL,
 * LAMB_EINVAL. */
LAMB_API lamb_status lamb_plan_set_path(lamb_plan *plan, int32_t path);

/*
 * The single-pass layout (host outputs; any may be NULL):
 *   tiles_per_tensor  n_tensors entries: the layer's tile count on the
 *                     single pass (of its tail, for a layer of more than one
 *                     round of tiles)
 *   n_tiles           total tiles of the single pass
 *   tile_groups       the tile shape lamb_tile_schedule chose: 8 (tiles of
 *                     8192 elements) or 10 (10240 elements)
 *   single_elems      n_tensors entries: the layer's elements on the single
 *                     pass; the rest (the head of a larger layer) take the
 *                     two-pass kernels
 * Errors: LAMB_ENULL (plan).
 */
LAMB_API lamb_status lamb_plan_tiles(const lamb_plan *plan, int32_t *tiles_per_tensor,
                            int32_t *n_tiles, int32_t *tile_groups, int64_t *single_elems);

/*
 * Wait for `stream` and report whether a single-pass step of the plan gave
 * up a wait (a layer's tiles were not all resident within about a second:
 * 2^22 polls, or the count in the environment variable
 * LAMB_MI355X_SPIN_LIMIT when lamb_plan_create ran, which tests use to
 * exercise this path; a value that is not a positive integer makes
 * lamb_plan_create fail with LAMB_EINVAL, and values above 2^30 count as
 * 2^30).
 * That step's state is then undefined (tiles that finished reading had
 * written new moments without moving x), and from then on every kernel of
 * the plan returns without changing anything, on both paths. To recover,
 * restore x, m and v from a checkpoint and build a new plan (on
 * LAMB_PATH_TWO_PASS if the device cannot be given to the single pass
 * alone). Synchronises the stream. Errors: LAMB_ENULL, LAMB_EHIP,
 * LAMB_ESYNC.
 */
LAMB_API lamb_status lamb_plan_check(lamb_plan *plan, void *stream);

/*
 * Fill `hp` with the paper's defaults for `variant` (Section 4, Appendix H:
 * beta1 0.9, beta2 0.999, eps 1e-6, lambda 0.01; Appendix D for N-LAMB and
 * NN-LAMB: beta1 0.975, eps 1e-8; LARS: momentum 0.9, trust_coef 1), with
 * step 1, lr 1e-3, phi clamp [0, 10], L2 norms, grad_scale 1, bias
 * correction on and no non-finite skip. Errors: LAMB_ENULL, LAMB_EINVAL.
 */
LAMB_API lamb_status lamb_hparams_init(lamb_hparams *hp, int32_t variant);

/*
 * One step of any algorithm over every block of the plan: the single-pass
 * kernel for the layers that take it (lamb_path), then for the other layers
 * a moment pass, a per-tensor finalize (norms, phi, trust ratio) and an
 * apply pass.
 *   hp             host, validated before any HIP call
 *   stream         hipStream_t (NULL = null stream)
 *   ratio_out      device, n_tensors doubles, or NULL
 *   norms_out      device, 2*n_tensors doubles {||x_i||, ||u_i||}, or NULL
 *   nonfinite_out  device int32, or NULL; needs skip_nonfinite = 1; receives 1
 *                  when the step was skipped, else 0
 * Errors: LAMB_ENULL, LAMB_EPLAN (variant and plan disagree), LAMB_EINVAL,
 * LAMB_EHIP.
 */
LAMB_API lamb_status lamb_step_ex(lamb_plan *plan, const lamb_hparams *hp, void *stream,
                         double *ratio_out, double *norms_out, int32_t *nonfinite_out);

/*
 * One LAMB step (Algorithm 2) over every block of the plan, at step t = step:
 *   m <- beta1 m + (1 - beta1) g ;  v <- beta2 v + (1 - beta2) g^2
 *   r  = (m / c1) / (sqrt(v / c2) + eps),  c1 = 1 - beta1^t, c2 = 1 - beta2^t
 *        (c1 = c2 = 1 when bias_correction == 0, Appendix E)
 *   u  = r + lambda_i x,  lambda_i = wd_i ? weight_decay : 0
 *   x <- x - lr * phi(||x_i||) / ||u_i|| * u      per block i
 * A block with ||u_i|| = 0 is left unchanged and reports ratio 0.
 * Scalars: step >= 1; 0 <= beta1, beta2 < 1; eps >= 0; 0 <= gamma_l <=
 * gamma_u (gamma_u may be +inf); lr and weight_decay finite.
 *   ratio_out  device, n_tensors doubles: phi(||x_i||)/||u_i||, or NULL
 *   norms_out  device, 2*n_tensors doubles {||x_i||, ||u_i||}, or NULL
 * Errors: LAMB_ENULL (plan), LAMB_EPLAN (a LARS plan), LAMB_EINVAL, LAMB_EHIP.
 */
LAMB_API lamb_status lamb_step(lamb_plan *plan, float lr, float beta1, float beta2,
                      float eps, float weight_decay, float gamma_l,
                      float gamma_u, int64_t step, int32_t bias_correction,
                      void *stream, double *ratio_out, double *norms_out);

/*
 * One N-LAMB step (Algorithm 3, Appendix D) or, with nesterov_v = 1, one
 * NN-LAMB step (Algorithm 4) over every block of a LAMB plan, at step t:
 *   m <- beta1 m + (1 - beta1) g ;  v <- beta2 v + (1 - beta2) g^2
 *   m_hat = beta1 m / (1 - beta1^(t+1)) + (1 - beta1) g / (1 - beta1^t)
 *   v_hat = beta2 v / (1 - beta2^t)                                  (N-LAMB)
 *   v_hat = beta2 v / (1 - beta2^(t+1)) + (1 - beta2) g^2 / (1 - beta2^t)
 *                                                                    (NN-LAMB)
 *   u = m_hat / (sqrt(v_hat) + eps) + lambda_i x ; x as in lamb_step.
 * The algorithms take a per-step sequence {beta1^t}; this entry point uses
 * the constant sequence beta1^t = beta1 (the paper's setting, beta1 = 0.975),
 * whose running products are the powers above. The apply pass also reads g.
 * Scalars, outputs and errors as lamb_step (nesterov_v must be 0 or 1).
 */
LAMB_API lamb_status nlamb_step(lamb_plan *plan, float lr, float beta1, float beta2,
                       float eps, float weight_decay, float gamma_l,
                       float gamma_u, int64_t step, int32_t nesterov_v,
                       void *stream, double *ratio_out, double *norms_out);

/*
 * One LARS step (Algorithm 1) over every block of the plan:
 *   m <- momentum m + (1 - momentum) (g + lambda_i x)
 *   x <- x - lr * trust_coef * phi(||x_i||) / ||m_i|| * m      per block i
 * trust_coef (kappa) scales the ratio; kappa = 1 is Algorithm 1 as printed.
 * A block with ||m_i|| = 0 is left unchanged and reports ratio 0.
 * Scalars: 0 <= momentum < 1; 0 <= gamma_l <= gamma_u; lr, weight_decay and
 * trust_coef finite.
 *   ratio_out  device, n_tensors doubles kappa phi/||m_i||, or NULL
 *   norms_out  device, 2*n_tensors doubles {||x_i||, ||m_i||}, or NULL
 * Errors: LAMB_ENULL, LAMB_EPLAN (a LAMB plan), LAMB_EINVAL, LAMB_EHIP.
 */
LAMB_API lamb_status lars_step(lamb_plan *plan, float lr, float momentum,
                      float weight_decay, float gamma_l, float gamma_u,
                      float trust_coef, void *stream, double *ratio_out,
                      double *norms_out);

/*
 * Split step, for optimizer state sharded over workers. Section 4.1 trains
 * with synchronous data parallelism: every worker holds the step's averaged
 * gradient g_t. When each worker keeps only a slice of every block's x, m
 * and v, it runs the step on its slices (one plan over them); the layer norms
 * ||x_i|| and ||u_i|| of Algorithms 1-2 then need every slice, so the step
 * splits where those norms are formed:
 *
 *   lamb_step_partials   the moment pass over every block of the plan (the
 *                        two-pass kernels, whatever the plan's path): with
 *                        skip_nonfinite = 0 it writes the new m and v; with
 *                        skip_nonfinite = 1 it only reads, since whether the
 *                        step runs is known once every shard has reported.
 *                        Then each block's partial norms over this plan's
 *                        elements go to `totals`.
 *   (the caller combines the totals of all shards, element by element)
 *   lamb_step_finish     from the combined totals: each block's norms, phi,
 *                        trust ratio and step scale (as lamb_step_ex), then
 *                        the apply pass. With skip_nonfinite = 1 it writes x,
 *                        m and v unless the combined verdict is nonzero, in
 *                        which case nothing changes.
 *
 *   totals   device, 2 * n_tensors + 1 doubles. totals[2 i] and totals[2 i + 1]
 *            are block i's partial norms of x and of the update direction u
 *            (m_t for LARS) over this plan's elements, as raw accumulators:
 *            sums of squares (L2), sums of magnitudes (L1) or maxima of
 *            magnitudes (L-infinity). totals[2 n] is 1.0 when skip_nonfinite
 *            is set and any scaled gradient element of this plan is NaN or
 *            infinite, else 0.0. Combine shards with an element-wise sum (L2,
 *            L1) or maximum that keeps NaN (L-infinity); either keeps
 *            totals[2 n] nonzero when any shard saw a non-finite gradient.
 *            lamb_step_finish only reads it (totals may be the buffer the
 *            combine wrote in place).
 *   hp       the same hyperparameters for both halves of one step, and for
 *            every shard; validated on the host before any HIP call
 *   ratio_out, norms_out, nonfinite_out   as lamb_step_ex (the combined,
 *            whole-block values)
 * Between the two halves the plan runs nothing else. Timing hooks do not
 * record split steps. Errors: LAMB_ENULL (plan, totals), LAMB_EPLAN,
 * LAMB_EINVAL, LAMB_EHIP.
 */
LAMB_API lamb_status lamb_step_partials(lamb_plan *plan, const lamb_hparams *hp, void *stream,
                                        double *totals);
LAMB_API lamb_status lamb_step_finish(lamb_plan *plan, const lamb_hparams *hp, void *stream,
                                      const double *totals, double *ratio_out,
                                      double *norms_out, int32_t *nonfinite_out);

/*
 * Per-tile timeline of the single pass, for measurement. With `trace` a
 * device buffer of 4 * n_tiles 64-bit words (lamb_plan_tiles), every later
 * single-pass step of the plan writes for tile j (its index in the schedule,
 * lamb_tile_schedule): trace[4 j] when the tile starts, [4 j + 1] when its
 * reads and partial norms are done, [4 j + 2] when its layer's step scale is
 * known and [4 j + 3] when its writes are issued, in ticks of the device's
 * constant 100 MHz clock (entries of empty tiles are left as they are). NULL
 * turns it off. The caller owns the buffer and must keep it valid while
 * traced steps run. Errors: LAMB_ENULL (plan), LAMB_EALIGN.
 */
LAMB_API lamb_status lamb_plan_set_trace(lamb_plan *plan, uint64_t *trace);

/*
 * Check of the two-pass path's recomputation (Algorithm 2's last line uses
 * one u for ||u_i|| and for the update; the apply pass recomputes u from the
 * stored moments instead of storing it). enable = 1 allocates one partial-norm
 * pair per chunk of the plan: from then on the apply pass of every step that
 * takes the two-pass kernels without skip_nonfinite (lamb_step_ex on layers
 * outside the single pass, lamb_step_finish) also sums the norms of the x it
 * reads and of the u it recomputes, per chunk, in the moment pass's order,
 * which must give the moment pass's partials bit for bit. enable = 0 frees
 * the buffer. Do not call while a step runs. Errors: LAMB_ENULL, LAMB_EINVAL,
 * LAMB_ENOMEM, LAMB_EHIP.
 */
LAMB_API lamb_status lamb_plan_set_u_check(lamb_plan *plan, int32_t enable);

/*
 * Wait for `stream` and copy, for the last step that ran the check, the
 * moment pass's per-chunk partial norms and the apply pass's re-summed ones
 * to the host: moment_out and apply_out receive *n_out pairs {x, u} each, in
 * the order of that step's chunk table (*n_out = 0, and nothing is copied,
 * when the last step did not run the check). capacity: pairs each array can
 * hold. Errors: LAMB_ENULL, LAMB_EINVAL (capacity too small; *n_out is still
 * set), LAMB_EHIP.
 */
LAMB_API lamb_status lamb_plan_u_partials(lamb_plan *plan, void *stream, int32_t capacity,
                                          double *moment_out, double *apply_out,
                                          int32_t *n_out);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): lamb_step_ex over a table
 * of blocks without a plan. It runs the two-pass kernels (exactly those of a
 * plan on LAMB_PATH_TWO_PASS with the same chunk_elems, with the same results
 * bit for bit) and keeps their tables, per-chunk partial norms, scales and
 * flags in a fixed device array of the library: 10.8 MiB, one per device,
 * held from the library's load on that device until the process ends. A call
 * allocates no device or host memory and copies nothing from the host: the
 * tensor table reaches the device as kernel arguments of ceil(n_tensors / 48)
 * small table kernels, which also clear the array's flag words.
 *   tensors       host array of n_tensors blocks, as lamb_plan_create (v may
 *                 be NULL for LARS); validated on every call
 *   g_dtype       lamb_grad_dtype
 *   chunk_elems   0 (the default) or as lamb_plan_create
 *   hp, stream, ratio_out, norms_out, nonfinite_out   as lamb_step_ex (a
 *                 LARS step is hp->variant = LAMB_VARIANT_LARS; hp selects
 *                 the algorithm, there being no plan)
 * Limits: n_tensors <= 4096, and at most 2^19 chunks of chunk_elems elements
 * over the table (the sum of ceil(numel / chunk_elems)); a larger table fails
 * with LAMB_EINVAL before any HIP call (a larger chunk_elems fits more).
 * Every call on one device shares that device's array, which keeps the last
 * call's contents: calls that overlap in time on one device (on different
 * streams or host threads) race and give undefined results; calls ordered
 * on one stream are safe. Runs on the current device.
 * Errors: as lamb_plan_create and lamb_step_ex (LAMB_EPLAN does not occur).
 */
LAMB_API lamb_status lamb_step_static(const lamb_tensor *tensors, int32_t n_tensors,
                                      int32_t g_dtype, int32_t chunk_elems,
                                      const lamb_hparams *hp, void *stream, double *ratio_out,
                                      double *norms_out, int32_t *nonfinite_out);

/*
 * The chunk table a plan would use (host only, no HIP call). Tensor i is cut
 * into ceil(numel[i] / chunk_elems) chunks in table order; chunk k of it
 * starts at k * chunk_elems and holds min(chunk_elems, numel[i] - start)
 * elements. chunk_elems = 0 picks the default.
 *   numel        host, n_tensors sizes (each in [1, 2^40])
 *   capacity     length of the three host output arrays (may be 0 with NULL
 *                outputs to query the count)
 *   n_chunks     receives the number of chunks
 * Errors: LAMB_ENULL, LAMB_EINVAL (including capacity too small, in which
 * case *n_chunks still receives the count).
 */
LAMB_API lamb_status lamb_chunk_table(const int64_t *numel, int32_t n_tensors,
                             int32_t chunk_elems, int32_t capacity,
                             int32_t *chunk_tensor, int64_t *chunk_start,
                             int32_t *chunk_len, int32_t *n_chunks);

/*
 * The single-pass schedule a plan would use (host only, no HIP call). The
 * single-pass kernel runs a persistent grid of `round` workgroups; workgroup
 * w takes entries w, w + round, ..., so the entry list falls into rounds of
 * `round` entries. A tile holds G blocks of 1024 elements (G = 8 or 10). A
 * layer of n elements takes T = ceil(n / (1024 G)) tiles; if T <= max_round
 * it takes the single pass: its tiles are consecutive entries inside one
 * round, and tile j holds the layer's blocks j, j + T, ..., j + (G - 1) T
 * (those inside the layer). Layers are packed first-fit by decreasing tile
 * count (ties in table order) into the fewest rounds of `max_round`
 * entries; `round` is then the narrowest width that packs into as few
 * rounds, so the rounds come out about equally full. The gap a round leaves
 * is filled with empty entries (tensor -1, length 0). A plan uses
 * max_round = 4 * (compute units) and tile_groups = 0.
 *   numel         host, n_tensors sizes (each in [1, 2^40])
 *   max_round     widest round, >= 1
 *   tile_groups   G: 8, 10, or 0 for a plan's choice, which is 10 only if
 *                 that puts more parameters on the single pass than 8
 *   capacity      length of the three entry arrays (0 with NULL arrays to
 *                 query the count)
 *   entry_tensor  host, layer of each entry or -1
 *   entry_start   host, first element of each entry (of its first block)
 *   entry_len     host, elements each entry holds (0 for an empty entry)
 *   first_tile    host, n_tensors: the layer's first entry (0 if none)
 *   tiles         host, n_tensors: the layer's tile count, 0 when it takes
 *                 the two-pass kernels (more than `max_round` tiles)
 *   n_entries     receives the length of the list
 *   round_out     receives the round width (the single-pass grid)
 *   groups_out    receives G (may be NULL)
 * Errors: LAMB_ENULL, LAMB_EINVAL (including capacity too small, in which
 * case *n_entries, *round_out, *groups_out, first_tile and tiles are still
 * filled).
 */
LAMB_API lamb_status lamb_tile_schedule(const int64_t *numel, int32_t n_tensors,
                               int32_t max_round, int32_t tile_groups, int32_t capacity,
                               int32_t *entry_tensor, int64_t *entry_start, int32_t *entry_len,
                               int32_t *first_tile, int32_t *tiles, int32_t *n_entries,
                               int32_t *round_out, int32_t *groups_out);

/*
 * Per-kernel timing with HIP events, for measurement. max_steps > 0 creates
 * events for that many recorded steps; from then on one step in `every`
 * (the first, then every `every`-th) records events around its kernels on
 * the step's stream, until max_steps steps are recorded. Each
 * recorded step costs a few microseconds of event processing, which
 * sampling (every > 1) spreads thin. max_steps = 0 turns timing off and
 * frees the events. Errors: LAMB_ENULL, LAMB_EINVAL, LAMB_EHIP.
 */
LAMB_API lamb_status lamb_plan_set_timing(lamb_plan *plan, int32_t max_steps, int32_t every);

/*
 * Synchronise on the recorded events and return the summed durations in
 * milliseconds over `steps` recorded steps (host) of: kernel_ms[0] the
 * moment kernel, [1] the finalize (both levels), [2] the apply kernel, [3]
 * the single-pass kernel, [4] the finiteness check (host, 5 entries; 0 for
 * a kernel the steps did not launch). Then start a new recording window.
 */
LAMB_API lamb_status lamb_plan_timing(lamb_plan *plan, double *kernel_ms, int64_t *steps);

/*
 * Host-side learning-rate schedule (Section 4): a polynomially decaying rate
 * eta = eta_0 (1 - tau/T)^power after a linear warmup, in stages that run
 * back to back, so that the second stage of mixed-batch training (Section
 * 4.1) warms up again.
 *   steps         T, iterations in the stage (>= 1)
 *   warmup_steps  W, 0 <= W <= T
 *   peak_lr       eta_0, finite and >= 0
 *   power         decay exponent (1 in the paper), finite and >= 0
 */
typedef struct lamb_lr_stage {
    int64_t steps;
    int64_t warmup_steps;
    double peak_lr;
    double power;
} lamb_lr_stage;

/*
 * Learning rate for step t >= 1 (the t passed to lamb_step). With tau = the
 * number of steps already taken inside the stage holding t:
 *   tau <  W:  eta_0 (tau + 1) / W          (reaches eta_0 on the last warmup step)
 *   tau >= W:  eta_0 (1 - tau / T)^power
 * and 0 after the last stage. Errors: LAMB_ENULL, LAMB_EINVAL (t < 1 or a
 * stage out of range); *lr_out is untouched on error.
 */
LAMB_API lamb_status lamb_lr_at(const lamb_lr_stage *stages, int32_t n_stages, int64_t step,
                       double *lr_out);

/*
 * Square-root learning-rate scaling (Section 4; Tables 4 and 5):
 * lr = base_lr * sqrt(batch / base_batch). Errors: LAMB_ENULL, LAMB_EINVAL
 * (non-positive batch sizes, negative or non-finite base_lr).
 */
LAMB_API lamb_status lamb_sqrt_scaled_lr(double base_lr, int64_t base_batch, int64_t batch,
                                double *lr_out);

/* Static description of a status code. */
LAMB_API const char *lamb_status_str(int32_t status);

/* Detail of the calling thread's last failure ("" if none). */
LAMB_API const char *lamb_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LAMB_MI355X_H */
