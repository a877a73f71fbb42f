/*
 * meq.h - C ABI of the MeqMuon optimizer update for AMD MI355X (gfx950).
 *
 * One call of meq_step updates every parameter of a plan.  A plan holds one kind
 * of parameter (Algorithm "MeqMuon", arxiv 2609.35701, Section "MeqMuon"); all
 * kinds share the momentum and the write-back:
 *
 *   B   <- mu * B + G                                   eq. "momentum"
 *   V   <- B            (or G + mu * B when nesterov)   Section "Experiments"
 *   W   <- (1 - lr * lambda) * W - rho * lr * U~        eq. "meqmuon-update"
 *
 * and differ in U~:
 *   MEQ_PARAM_HIDDEN  2D hidden-layer weight W (m x n, rows = output features):
 *                       U   <- K quintic Newton-Schulz steps on V / ||V||_F   eq. "ns"
 *                       r,c <- row / column RMS of U                          eq. "row-col-rms"
 *                       U~  <- N_r(U) if CV(r) >= CV(c) else N_c(U)           eqs. "cv", "operators", "hidden"
 *                     or, with update_rule MEQ_RULE_MOONLIGHT, the Muon update the paper
 *                     compares with: U~ <- sqrt(max(m, n)) * U               eq. "moonlight-update"
 *   MEQ_PARAM_AUX     remaining 2D parameter (token embedding, LM head; rows = vocabulary):
 *                       U~  <- N_c(N_r(V))                                    eq. "aux"
 *   MEQ_PARAM_VECTOR  1-D parameter (norm weight, bias) of d elements:
 *                       U~  <- V / (||V||_2 / sqrt(d))                        eq. "vector"
 *
 * Conventions shared by every entry point
 *   - Matrices are dense, contiguous, row-major; element (i, j) of an m x n
 *     matrix sits at offset i * n + j.
 *   - "Device pointer" means memory allocated on the HIP device the stream
 *     belongs to (hipMalloc or a torch CUDA/HIP tensor).  The library never
 *     allocates, frees or takes ownership of caller memory.
 *   - Functions that return meq_status validate every argument before any
 *     device work; on an argument error nothing is enqueued and no caller
 *     memory is modified.  HIP failures are reported as MEQ_ERR_HIP.
 *   - A step enqueues many kernels.  When a launch fails part-way (MEQ_ERR_HIP,
 *     MEQ_ERR_NO_MEMORY or MEQ_ERR_INTERNAL from meq_step), the launches before
 *     it stay enqueued and the ones after it are not: some matrices may have
 *     their momenta (and, for a later pass or kernel, parameters) updated while
 *     others do not.  The step is not atomic; a caller that must recover keeps a
 *     copy of the parameters and momenta.
 *   - No entry point blocks the host except meq_get_stats, meq_ns_cv_trace and
 *     meq_get_timing, which synchronize with the given stream.
 *   - A plan is not reentrant: do not run two meq_step calls of one plan (or
 *     two plans sharing one workspace) concurrently on different streams.
 */
#ifndef MEQ_H
#define MEQ_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MEQ_OK = 0,
  MEQ_ERR_INVALID_ARG = -1, /* a null pointer, a bad size or hyperparameter, a count mismatch   */
  MEQ_ERR_UNSUPPORTED = -2, /* a dtype combination or size the library does not implement        */
  MEQ_ERR_HIP = -3,         /* a HIP runtime call or kernel launch failed                          */
  MEQ_ERR_WORKSPACE = -4,   /* the workspace is null, too small or not 256-byte aligned           */
  MEQ_ERR_NO_MEMORY = -5,   /* a host allocation (plan metadata, launch lists) failed; no launch   */
                            /* of the failing call was enqueued after the failure                  */
  MEQ_ERR_INTERNAL = -6     /* an unexpected host-side failure inside the library (a bug); no      */
                            /* launch of the failing call was enqueued after it                    */
} meq_status;

typedef enum { MEQ_F32 = 0, MEQ_BF16 = 1 } meq_dtype;

/* Normalization direction chosen for a matrix (eq. "hidden"). */
typedef enum { MEQ_DIR_ROW = 0, MEQ_DIR_COL = 1 } meq_direction;

/* Parameter kind of a plan (the three branches of Algorithm "MeqMuon"). */
typedef enum { MEQ_PARAM_HIDDEN = 0, MEQ_PARAM_AUX = 1, MEQ_PARAM_VECTOR = 2 } meq_param_kind;

/* Update of hidden weights: MeqMuon's equilibrated update (eq. "hidden"), or the
 * Moonlight-Muon update with the sqrt(max(m, n)) factor and no equilibration
 * (eq. "moonlight-update"), run on the same Newton-Schulz kernels. */
typedef enum { MEQ_RULE_MEQMUON = 0, MEQ_RULE_MOONLIGHT = 1 } meq_update_rule;

/*
 * Hyperparameters of the update (Section "Experiments"; delta from Section
 * "Imbalance patterns").  The learning rate eta_t is passed to each meq_step.
 *   mu             momentum coefficient, 0 <= mu < 1
 *   rho            RMS alignment coefficient, rho > 0
 *   weight_decay   decoupled weight decay lambda >= 0
 *   ns_steps       number K of Newton-Schulz steps, 1 <= K <= 64
 *   ns_a/b/c       quintic coefficients (a, b, c), finite
 *   zero_rms_delta RMS values at or below delta count as zero, delta >= 0
 *   nesterov       0: normalize B_t (Algorithm "MeqMuon");
 *                  1: normalize G_t + mu * B_t (the experiments' hidden weights)
 *   update_rule    meq_update_rule; MEQ_RULE_MOONLIGHT only for MEQ_PARAM_HIDDEN plans
 *   ns_gram_steps  g, 1 <= g <= 3: the most Newton-Schulz steps one Gram-space segment
 *                  covers.  g = 1 runs eq. "ns" as printed: every step forms A = X X^T,
 *                  the polynomial P = a I + b A + c A A and X <- P X.  With g >= 2, a
 *                  matrix whose padded long side is at least twice its padded short side
 *                  runs its K steps in segments of at most g steps: a segment forms
 *                  A = X X^T once, then iterates on s x s matrices only (each step's P is a
 *                  polynomial of A, so A_{k+1} = P_k A_k P_k and the segment's product
 *                  Q = P_last ... P_first are symmetric and commute), and ends with one
 *                  product X <- Q X.  Equal to eq. "ns" in exact arithmetic; it replaces
 *                  most s x l products by s x s ones.  Segments are g steps long, the last
 *                  one takes the remainder (K = 5, g = 3: 3 + 2).  Default 3.  Longer
 *                  segments are not offered: a single segment of 4 or 5 steps loses
 *                  accuracy on rank-deficient inputs.
 *                  Precision in every schedule: fp32 accumulation; X and the matrix that
 *                  multiplies it (P of a printed step, a segment's final Q) in bf16; A = X X^T
 *                  and the other s x s matrices of a segment in fp16 (A scaled by 2^13), whose
 *                  11-bit significand keeps the iteration more accurate than bf16 storage.
 *                  fp16 needs bounded iterates: meq_init bounds the singular values of 64
 *                  steps of the plan's coefficients (each step maps [0, r] into
 *                  [0, max |a x + b x^3 + c x^5| on [0, r]]) and, unless the scaled matrices
 *                  stay below 16384, runs every matrix through the printed iteration with all
 *                  matrices in bf16 (segments are then not used).  The paper's coefficients
 *                  keep every singular value below 1.21 and pass.
 * ns_steps, ns_a/b/c and ns_gram_steps only matter for hidden plans but are validated for
 * every plan.
 */
typedef struct {
  float mu;
  float rho;
  float weight_decay;
  int32_t ns_steps;
  float ns_a;
  float ns_b;
  float ns_c;
  float zero_rms_delta;
  int32_t nesterov;
  int32_t update_rule;
  int32_t ns_gram_steps;
} meq_hparams;

/*
 * One parameter: rows x cols, with its parameter and gradient dtype.
 * Supported (param, grad) pairs: (MEQ_F32, MEQ_F32) and (MEQ_BF16, MEQ_BF16).
 * The momentum is always float32 with the same shape (one value per element,
 * the paper's optimizer-state accounting in Table "experiment-efficiency").
 * Limits by plan kind:
 *   hidden  1 <= rows, cols <= 65536
 *   aux     1 <= rows <= 2^24, 1 <= cols <= 65536, rows * cols < 2^31
 *   vector  rows * cols elements form one vector; 1 <= rows * cols < 2^31
 */
typedef struct {
  int64_t rows;
  int64_t cols;
  int32_t param_dtype; /* meq_dtype */
  int32_t grad_dtype;  /* meq_dtype */
} meq_matrix_desc;

typedef struct meq_plan meq_plan; /* opaque; owns host metadata only */

/* Fill *hp with the paper's defaults: mu 0.95, rho 0.2, lambda 0.1, K 5,
 * (a, b, c) = (3.4445, -4.7750, 2.0315), delta 1e-7, nesterov 0,
 * update_rule MEQ_RULE_MEQMUON, ns_gram_steps 3.  No-op on null. */
void meq_default_hparams(meq_hparams* hp);

/*
 * Validate `count` parameter descriptors of one meq_param_kind and the
 * hyperparameters and build a plan: hidden matrices are grouped by shape for
 * batched Newton-Schulz launches, and the workspace layout is fixed.  Touches no
 * device and may run without a GPU.  count == 0 is allowed (meq_step is then a
 * no-op).  On success *out receives a plan the caller releases with meq_destroy;
 * on failure *out is set to NULL.  An unknown kind, or MEQ_RULE_MOONLIGHT with a
 * kind other than MEQ_PARAM_HIDDEN, is MEQ_ERR_INVALID_ARG.
 */
meq_status meq_init_kind(int32_t kind, const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp,
                         meq_plan** out);

/* meq_init_kind(MEQ_PARAM_HIDDEN, ...). */
meq_status meq_init(const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp, meq_plan** out);

/*
 * meq_init_kind with the plan's workspace held to at most max_workspace_bytes (0: no cap, the
 * same plan as meq_init_kind).  The update is the same: every matrix's arithmetic is the same,
 * and the results are bitwise equal to the uncapped plan's.  A hidden plan keeps its per-matrix
 * statistics for all matrices and one region for the Newton-Schulz buffers
 * (Algorithm "MeqMuon" as written handles one matrix at a time; the memory of the update is the
 * point of the paper's Table "experiment-efficiency"): its shape groups are cut into slices
 * packed into passes that fit the region, and meq_step runs the passes one after the other on
 * the stream (momentum, Newton-Schulz, statistics and write-back of one pass before the next),
 * each reusing the region.  Fewer matrices per launch fill the GPU less, so a small cap costs
 * time.  Aux and vector plans are not sliced; their workspace must fit the cap as planned.
 * MEQ_ERR_WORKSPACE when the per-matrix part alone, or one matrix's Newton-Schulz buffers,
 * exceed the cap; other errors as meq_init_kind.
 */
meq_status meq_init_capped(int32_t kind, const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp,
                           size_t max_workspace_bytes, meq_plan** out);

/* Bytes of device workspace meq_step needs for this plan (0 for a null plan). */
size_t meq_workspace_bytes(const meq_plan* plan);

/*
 * Enqueue one update of every matrix of the plan on `stream` (0 = the null
 * stream of the current device).
 *   params[i]   device pointer, rows x cols of param_dtype; updated in place
 *   grads[i]    device pointer, rows x cols of grad_dtype; read only
 *   momenta[i]  device pointer, rows x cols float32; updated in place; zero
 *               before the first step (B_{-1} = 0)
 *   lr          learning rate eta_t of this step (finite, >= 0)
 *   workspace   device pointer, 256-byte aligned, at least workspace_bytes bytes,
 *               >= meq_workspace_bytes(plan); its contents need not be preserved
 *               between calls, but it must not be used by anything else while
 *               the step runs.  It also holds the statistics read by
 *               meq_get_stats until the next meq_step.
 * The three pointer arrays are host arrays of `count` entries (count as given to
 * meq_init) and are only read during the call.  Parameters, gradients and
 * momenta of different matrices must not overlap each other or the workspace.
 * Returns after enqueuing; the update is complete when the stream reaches it.
 */
meq_status meq_step(meq_plan* plan, void* const* params, const void* const* grads, float* const* momenta,
                    float lr, void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Copy the last step's per-matrix statistics from the workspace to host arrays
 * of `count` entries (any of them may be null): gamma_r, gamma_c are the row
 * and column CVs of U (eq. "cv", computed in double precision), dir the chosen
 * meq_direction.  Synchronizes with `stream`.  Only hidden plans with
 * MEQ_RULE_MEQMUON compute these; other plans return MEQ_ERR_UNSUPPORTED.
 */
meq_status meq_get_stats(const meq_plan* plan, const void* workspace, double* gamma_r, double* gamma_c,
                         int32_t* dir, hipStream_t stream);

/*
 * Diagnostics: the row and column CVs of X_k for k = 0 .. kmax (eq. "cv" of the row/column
 * RMS of eq. "row-col-rms"), where X_0 = V / ||V||_F is formed from inputs[i] (device
 * pointer, rows x cols of the matrix's param dtype, read only) and X_k follows eq. "ns" with
 * the plan's coefficients; the replay behind the paper's CV trajectories of the NS
 * iterations (Section "Imbalance patterns").  Runs on the plan's own kernels, uses the
 * workspace (its statistics are overwritten) and touches no parameters or momenta.
 * gamma_r and gamma_c are host arrays of count * (kmax + 1) doubles, matrix-major
 * (entry i * (kmax + 1) + k).  A hidden plan only; 0 <= kmax <= 64.  Synchronizes with
 * `stream` once per k.
 */
meq_status meq_ns_cv_trace(meq_plan* plan, const void* const* inputs, int32_t kmax, void* workspace,
                           size_t workspace_bytes, double* gamma_r, double* gamma_c, hipStream_t stream);

/*
 * Bytes of the device scratch array meq_step_static uses as its workspace: one array per GPU the
 * library runs on, allocated with the library's code object and held until the process ends.
 */
#define MEQ_STATIC_SCRATCH_BYTES ((size_t)256 << 20)

/*
 * meq_step without a caller workspace, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  Same
 * arguments and update as meq_step; the workspace is the library's scratch array on the current
 * device (the stream must belong to the current device).  Nothing is allocated or freed: no
 * hipMalloc, hipFree or allocating library routine is called, only hipGetDevice and, once per
 * device, hipGetSymbolAddress.  A plan whose meq_workspace_bytes exceeds
 * MEQ_STATIC_SCRATCH_BYTES is rejected with MEQ_ERR_WORKSPACE before any device work; build such
 * plans with meq_init_capped(..., MEQ_STATIC_SCRATCH_BYTES, ...).  Every call on one GPU shares
 * that GPU's array and leaves its contents behind (nothing in it needs to start at zero: a step
 * writes every workspace byte it reads); calls that overlap on one GPU, on any streams or plans,
 * race on it and must be serialized by the caller.  The statistics meq_get_stats reads stay in
 * the library's array, so they are not available after this variant.
 */
meq_status meq_step_static(meq_plan* plan, void* const* params, const void* const* grads, float* const* momenta,
                           float lr, hipStream_t stream);

/* Release a plan (null is a no-op).  Pending timing events are destroyed. */
void meq_destroy(meq_plan* plan);

/* A static, human-readable description of a status code. */
const char* meq_status_string(meq_status s);

/* ----------------------------------------------------------------------------
 * Introspection (host only, no device work)
 * ------------------------------------------------------------------------- */

/* Number of Newton-Schulz shape groups (matrices with equal (min, max) dims); in a plan from
 * meq_init_capped a shape group cut into slices counts once per slice.  0 for aux and vector
 * plans. */
int32_t meq_plan_num_groups(const meq_plan* plan);

/* Number of passes a hidden plan's step runs (1 without a workspace cap; 0 for an empty plan and
 * for aux and vector plans). */
int32_t meq_plan_num_passes(const meq_plan* plan);

/* Shape group g: short side s, long side l (after transposing tall matrices to
 * wide orientation) and its number of matrices. */
meq_status meq_plan_group(const meq_plan* plan, int32_t g, int64_t* s, int64_t* l, int32_t* count);

/* Newton-Schulz schedule of shape group g: *nsegs receives the number of segments and
 * segs[0 .. min(*nsegs, max_segs) - 1] their lengths in steps (they sum to ns_steps; all
 * ones is the iteration of eq. "ns" as printed, see ns_gram_steps).  segs may be null
 * when max_segs is 0. */
meq_status meq_plan_group_schedule(const meq_plan* plan, int32_t g, int32_t* segs, int32_t max_segs,
                                   int32_t* nsegs);

/* Buffers of the workspace that tests may inspect after a step.
 * Hidden plans: all six.  Aux plans: MEQ_BUF_ROW_RMS (r of V), MEQ_BUF_COL_RMS
 * (c of N_r(V)).  Vector plans: MEQ_BUF_NORMSQ (||V||_2^2).  Other pairs are
 * MEQ_ERR_INVALID_ARG. */
typedef enum {
  MEQ_BUF_X0 = 0,      /* bf16 V (not yet divided by ||V||_F), wide orientation s x l, ld = padded l;
                          still intact after a step only when the matrix's Newton-Schulz schedule
                          has one segment (meq_plan_group_schedule; later segments reuse the
                          buffer) and the matrix is in the plan's last pass                       */
  MEQ_BUF_U = 1,       /* bf16 Newton-Schulz output U, wide orientation s x l, ld = padded l; after a
                          step of a plan with several passes only for matrices of the last pass    */
  MEQ_BUF_NORMSQ = 2,  /* double ||V||_F^2, 1 x 1                                                    */
  MEQ_BUF_ROW_RMS = 3, /* double r of U in the matrix's own orientation, 1 x rows                      */
  MEQ_BUF_COL_RMS = 4, /* double c of U in the matrix's own orientation, 1 x cols                      */
  MEQ_BUF_SCALE = 5    /* float per-row (dir row, 1 x rows) or per-column (1 x cols) scale of U~ = U*s;
                          with MEQ_RULE_MOONLIGHT every row's entry is sqrt(max(m, n))              */
} meq_buffer_kind;

/*
 * Locate buffer `kind` of matrix `matrix` inside the workspace: byte *offset from
 * the workspace start, logical *rows x *cols and leading dimension *ld in elements.
 * For MEQ_BUF_SCALE the extent depends on the direction chosen at run time; the
 * region returned covers max(rows, cols) entries.  Any output may be null.
 */
meq_status meq_debug_region(const meq_plan* plan, int32_t matrix, int32_t kind, size_t* offset, int64_t* rows,
                            int64_t* cols, int64_t* ld);

/* ----------------------------------------------------------------------------
 * Per-kernel timing with HIP events on the launch stream
 * ------------------------------------------------------------------------- */

typedef enum {
  MEQ_K_MOMENTUM = 0, /* momentum + ||V||^2 partials + bf16 V in wide orientation            */
  MEQ_K_NORM = 1,     /* ||V||_F^2 finalization                                                */
  MEQ_K_GRAM = 2,     /* A = X X^T and the Gram-space products P A, P T, P Q (symmetric tiles;  */
                      /* one launch may carry both)                                            */
  MEQ_K_POLY = 3,     /* P = a I + b A + c A A (symmetric tiles)                               */
  MEQ_K_APPLY = 4,    /* X <- P X, or X <- Q X at the end of a Gram-space segment              */
  MEQ_K_ROWCOL = 5,   /* row and column sums of squares of U                                    */
  MEQ_K_SELECT = 6,   /* CVs, direction, scale vector                                           */
  MEQ_K_UPDATE = 7,   /* decoupled weight decay + normalized update write-back                   */
  MEQ_K_AUX_ROWS = 8,   /* aux: momentum + row RMS of V                                         */
  MEQ_K_AUX_COLS = 9,   /* aux: column RMS of N_r(V) (partials + finalization)                   */
  MEQ_K_AUX_UPDATE = 10, /* aux: decoupled weight decay + two-sided normalized update            */
  MEQ_K_VECTOR = 11,    /* vector: momentum, global RMS and write-back in one kernel             */
  MEQ_K_COUNT = 12
} meq_kernel_kind;

/* Bracket every launch of the kinds in `kind_mask` (bit k = meq_kernel_kind k)
 * with HIP events on the launch stream from the next meq_step on; 0 turns timing off. */
meq_status meq_set_timing(meq_plan* plan, uint32_t kind_mask);

/* Synchronize the recorded events, add their durations to the plan's totals and
 * report, for kernel kind `kind`, the accumulated milliseconds and launch count
 * since the last reset (reset != 0 clears the totals after reading). */
meq_status meq_get_timing(meq_plan* plan, int32_t kind, double* total_ms, int64_t* launches, int32_t reset);

#ifdef __cplusplus
}
#endif

#endif /* MEQ_H */
