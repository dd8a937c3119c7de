/*
 * muon.h -- C ABI of the MI355X (gfx950) single-GPU Muon optimizer step.
 *
 * The library applies one Muon step (DMuon, arXiv 2606.27153, Sec. 2.1) to a
 * fixed list of weight matrices that one GPU owns.  For every matrix it runs
 *
 *   1. momentum:  M <- mu*M + G;  NS input u = G + mu*M (Nesterov) or u = M
 *   2. orientation: X = u^T when rows > cols, so that X is m x n, m <= n
 *   3. Frobenius normalisation: X0 = X / (||X||_F + eps)
 *   4. k steps of the quintic Newton-Schulz iteration of Eq. 2,
 *        A = X X^T,  B = b*A + c*A*A,  X <- a*X + B*X
 *      with the Gram product computed on lower-triangular tiles only and
 *      mirrored (the symmetric kernel of Sec. 3.3), the polynomial fused into
 *      the A*A product and a*X fused into B*X.  Wide enough matrices
 *      (n >= gram_min_aspect * m, m >= 256) instead carry the iteration in
 *      Gram space (Sec. 3.3, Eq. 4): G0 = X0 X0^T, P_i = a I + b G_i +
 *      c G_i^2, G_{i+1} = P_i (G_i P_i), Q = P_{j-1} ... P_0, X_j = Q X0 --
 *      every m x m product symmetric (lower tiles, mirrored), one m x n
 *      product at each end -- restarted from X_j every gram_restart steps:
 *      per segment of L steps 3 m^2 n + (4L - 3) m^3 flops instead of
 *      L (3 m^2 n + m^3)
 *   5. O = X^T (tall) or X (wide) -- the orthogonalised update NS_k(M_t)
 *   6. Eq. 1 with decoupled weight decay and the shape scale:
 *        W <- W*(1 - lr*wd) - lr*sqrt(max(1, rows/cols))*O
 *
 * Matrices are independent (Sec. 3.3); the plan groups them by shape into
 * buckets and advances whole groups through each NS step with grouped
 * launches, so many small matrices do not each pay a launch.
 *
 * Conventions for every entry point:
 *  - Every function returns a muon_status; nothing aborts, throws or exits.
 *    On failure muon_last_error() returns a thread-local message.
 *  - Device buffers are row-major (leading dimension = cols), contiguous and
 *    16-byte aligned.  The caller owns every device buffer and the stream.
 *  - muon_step enqueues work on the caller's HIP stream and returns; results
 *    are visible after the stream is synchronised.  Arguments are checked
 *    before anything is enqueued; on an error nothing is launched.
 *  - NaN or Inf in the inputs propagate; they are not sanitised.
 */
#ifndef MUON_MI355X_H
#define MUON_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MUON_ABI_VERSION 4

#if defined(__GNUC__)
#define MUON_API __attribute__((visibility("default")))
#else
#define MUON_API
#endif

typedef enum muon_status {
  MUON_OK = 0,
  MUON_ERR_INVALID_ARG = 1,          /* a null pointer, bad shape or out-of-range value */
  MUON_ERR_UNSUPPORTED = 2,          /* a dtype combination or option the library lacks */
  MUON_ERR_OUT_OF_MEMORY = 3,        /* host or device allocation failed (plan create) */
  MUON_ERR_WORKSPACE_TOO_SMALL = 4,  /* workspace_bytes below muon_plan_workspace_bytes */
  MUON_ERR_DEVICE = 5                /* a HIP call failed; the HIP error text is kept */
} muon_status;

typedef enum muon_dtype { MUON_F32 = 0, MUON_BF16 = 1 } muon_dtype;

/* Arithmetic of the Newton-Schulz GEMMs.  MUON_NS_BF16: bf16 operands in
 * HBM, fp32 accumulation on the matrix cores (matrices with
 * min(rows, cols) <= small_m_threshold still use fp32).  MUON_NS_FP32: fp32
 * operands and fp32 matrix-core arithmetic for every matrix (validation).
 * MUON_NS_FP16: fp16 operands, fp32 accumulation, for every matrix size (the
 * NS precision of the paper's implementation, Sec. 4 "Configurations"): the
 * same matrix-core rate as bf16 and about 8x less rounding error.  Its range
 * is fp16's: the Nesterov input u = G + mu*M is stored in fp16 before it is
 * normalised, so |u| must stay below 65504, and entries below 2^-24 round to
 * zero. */
typedef enum muon_ns_precision { MUON_NS_BF16 = 0, MUON_NS_FP32 = 1, MUON_NS_FP16 = 2 } muon_ns_precision;

/* Plan flags. */
#define MUON_PLAN_HOST_ONLY 0x1u     /* build host metadata only: no device memory is
                                        touched; such a plan can be inspected but not stepped */
#define MUON_PLAN_CHECK_BUFFERS 0x2u /* muon_step also vets where its buffers live (the memory
                                        checks of muon_check_buffers, two HIP queries per buffer)
                                        whenever their addresses differ from the previous call's */

/* One weight matrix: stored shape and dtypes.  param in {F32, BF16},
 * grad in {F32, BF16}, momentum must be F32. */
typedef struct muon_matrix_desc {
  int64_t rows;
  int64_t cols;
  int32_t param_dtype;
  int32_t grad_dtype;
  int32_t momentum_dtype;
  int32_t tile_hint;                 /* 0: the planner's cost model picks the GEMM tile; 64, 128 or
                                        256: use that output tile for this matrix (a measured
                                        choice, e.g. from an autotuner's cache; Sec. 3.3 tunes the
                                        schedule per shape).  256 needs 16-bit operands: with fp32
                                        NS (MUON_NS_FP32, or small m under bf16) it is UNSUPPORTED.
                                        Anything else is INVALID_ARG. */
} muon_matrix_desc;

typedef struct muon_plan_opts {
  int32_t precision;                 /* muon_ns_precision */
  int32_t max_ns_steps;              /* largest ns_steps muon_step accepts, 1..64 */
  float a, b, c;                     /* NS coefficients of Eq. 2, used for every step.  c = 0 gives the
                                        cubic iteration (the A*A product is skipped); otherwise b / c must
                                        be finite in fp32, else muon_plan_create returns INVALID_ARG */
  float eps;                         /* added to ||X||_F before dividing */
  int32_t small_m_threshold;         /* bf16 plans: min(rows,cols) <= this -> fp32 NS */
  uint32_t flags;                    /* MUON_PLAN_* */
  int64_t wave_bytes;                /* cap on the NS working set of one group ("wave")
                                        of matrices processed together; 0 = default (12 GiB) */
  float gram_min_aspect;             /* 16-bit NS matrices with m >= 256 and n >= gram_min_aspect * m
                                        run the Gram-space recurrence (Eq. 4); 0 = never.  Must be 0
                                        or >= 1; ignored when c = 0 at some step.  Default 1.4: from there
                                        the restarted form is both faster and, on planted spectra, as
                                        accurate as Eq. 2 in bf16 and fp16 */
  int32_t gram_restart;              /* NS steps per Gram-space segment: after that many steps the
                                        iterate X = Q X0 is formed and the recurrence restarts from
                                        a fresh Gram matrix X X^T.  0 = the default, 2.  Without
                                        restarts (a value >= ns_steps), 16-bit rounding of the Gram
                                        matrix is amplified from step to step wherever the input
                                        has small singular values, and the result can be far off;
                                        restarting every 2 steps keeps it as accurate as Eq. 2.
                                        Must be >= 0 */
  const float* abc_per_step;         /* NULL (a, b, c above at every step), or 3 * max_ns_steps
                                        floats: NS step i uses (a, b, c) = abc_per_step[3i],
                                        [3i + 1], [3i + 2] (a per-step coefficient set, Sec. 4
                                        "Configurations").  Read once by muon_plan_create, which
                                        keeps a copy; every triple obeys the rule for a, b, c.  A
                                        cubic step (c = 0) keeps every matrix on Eq. 2. */
} muon_plan_opts;

typedef struct muon_plan_s* muon_plan;

/* Summary of a plan (for callers and tests). */
typedef struct muon_plan_info {
  int32_t n_matrices;
  int32_t n_waves;                   /* groups of matrices stepped together */
  int32_t n_buckets;                 /* distinct (m, n, padded shape, kernel class) */
  int32_t device;                    /* HIP device the plan lives on, -1 if host-only */
  int64_t workspace_bytes;           /* bytes muon_step needs */
  int64_t launches_per_step;         /* kernel launches of one muon_step at max_ns_steps */
  double ns_flops_per_ns_step;       /* algorithmic flops of one NS step of Eq. 2 over all
                                        matrices: sum of 3 m^2 n + m^3 (symmetry-aware) */
  double padded_flops_per_ns_step;   /* flops those steps issue on padded tiles */
  int32_t n_gram;                    /* matrices that run the Gram-space recurrence */
  int32_t gram_restart;              /* NS steps per Gram-space segment (the effective value) */
} muon_plan_info;

/* Placement of one matrix in the plan. */
typedef struct muon_matrix_info {
  int64_t m, n;                      /* oriented: m = min(rows, cols), n = max */
  int64_t m_pad, n_pad;              /* padded to the kernel tile */
  int32_t transposed;                /* 1 if rows > cols */
  int32_t kernel_class;              /* index of the GEMM configuration */
  int32_t tile;                      /* square output tile of that configuration */
  int32_t fp32_ns;                   /* 1 if the NS GEMMs run in fp32 */
  int32_t wave;                      /* group the matrix is stepped in */
  int32_t bucket;
  int32_t gram_space;                /* 1 if it runs the Gram-space recurrence (Eq. 4) */
  int32_t reserved;
} muon_matrix_info;

/* Fills *o with the defaults: precision BF16, max_ns_steps 16,
 * (a,b,c) = (3.4445, -4.7750, 2.0315), eps 1e-7, small_m_threshold 64,
 * flags 0, wave_bytes 0, gram_min_aspect 1.4, gram_restart 0 (2), abc_per_step NULL.  Returns
 * INVALID_ARG if o is NULL. */
MUON_API muon_status muon_plan_opts_default(muon_plan_opts* o);

/* Builds a plan for n matrices (orientation, buckets, kernel classes, tile
 * tables, workspace layout).  Unless MUON_PLAN_HOST_ONLY is set, the plan is
 * bound to the current HIP device and uploads its tables there (the only
 * host-to-device copy outside muon_step).  opts may be NULL (defaults).
 * Errors: INVALID_ARG (null, n < 1, rows or cols < 1 or >= 2^31, bad tile_hint,
 * opts out of range), UNSUPPORTED (dtypes, a dimension that reaches 2^31 once padded to its
 * tile, a tile_hint of 256 with fp32 operands), OUT_OF_MEMORY, DEVICE. */
MUON_API muon_status muon_plan_create(const muon_matrix_desc* mats, int32_t n,
                             const muon_plan_opts* opts, muon_plan* out);

/* Releases the plan and its device tables.  NULL is accepted.  The caller
 * must make sure no enqueued step still uses the plan. */
MUON_API muon_status muon_plan_destroy(muon_plan plan);

/* Workspace size in bytes that muon_step needs. */
MUON_API muon_status muon_plan_workspace_bytes(muon_plan plan, size_t* bytes);

MUON_API muon_status muon_plan_get_info(muon_plan plan, muon_plan_info* info);

/* The plan's own algorithmic NS flops for ns_steps steps (symmetry-aware),
 * into *flops: an Eq. 2 matrix does 3 m^2 n + m^3 per step; a Gram-space
 * matrix, per segment of L steps, 3 m^2 n (the Gram product and the final
 * m x m x n product) and (4L - 3) m^3 (L polynomials P_i and 3 (L - 1)
 * further products of the recurrence).  INVALID_ARG for a NULL argument or
 * ns_steps outside [0, max_ns_steps]. */
MUON_API muon_status muon_plan_ns_flops(muon_plan plan, int32_t ns_steps, double* flops);
MUON_API muon_status muon_plan_matrix_info(muon_plan plan, int32_t index, muon_matrix_info* info);

/* One Muon step over every matrix of the plan (Eq. 1, Eq. 2).
 *
 * params[i]   device, rows x cols of param_dtype, updated in place
 * grads[i]    device, rows x cols of grad_dtype, read only; NULL skips
 *             matrix i for this step: its param and momentum are left
 *             untouched (no momentum update, no weight decay), as an
 *             optimizer skips a parameter that received no gradient
 * momentum[i] device, rows x cols fp32, updated in place
 *   (arrays of n device pointers on the host, in descriptor order; buffers of
 *   different matrices must not overlap)
 * lr, weight_decay: finite, >= 0;  momentum_coef in [0, 1)
 * ns_steps in [0, max_ns_steps];  nesterov: 0 or 1
 * workspace: device buffer of at least muon_plan_workspace_bytes bytes, owned
 *   by the caller, contents need not be initialised; steps that may run
 *   concurrently need distinct workspaces and distinct plans.
 * hip_stream: hipStream_t (NULL = default stream).
 *
 * The call only enqueues work on hip_stream; it never allocates and never
 * waits for the stream.  The plan keeps a device copy of the pointer arrays:
 * when they differ from the previous call's, the new table is written into
 * the next slot of a pinned host ring the plan owns (8 slots) and copied to
 * the device on hip_stream ahead of the kernels.  The host waits only when
 * that slot's copy from 8 refreshes earlier has not yet run on the GPU.
 * Successive steps on one plan must be ordered on the GPU (one stream, or
 * ordered by the caller): each refresh overwrites the device table the
 * previous step's kernels read.
 * A call on the same buffers as the previous call (with launch timing off)
 * enqueues kernels only, so it can be captured in a HIP graph and replayed;
 * each replay is bitwise the step an eager call would make.  The scalars
 * (lr, momentum_coef, weight_decay, ns_steps, nesterov) are captured by
 * value: a new value needs a new capture.  A call whose pointers differ
 * from the previous call's returns INVALID_ARG while its stream is being
 * captured (the copy from the ring could not be replayed safely).  A replay
 * reads the device table as it is at replay time: step eagerly on other
 * buffers in between, and replays use those.
 * The plan must be used from the device it was created on.  The step checks
 * the arguments (NULL param or momentum, alignment, workspace size, current
 * device) and, when the workspace address changes, that the workspace is
 * device memory of the plan's device large enough for the plan; the other
 * buffers' memory is vetted (muon_check_buffers) only on plans created with
 * MUON_PLAN_CHECK_BUFFERS, whenever the addresses change.  On an error
 * nothing is enqueued. */
MUON_API muon_status muon_step(muon_plan plan, void* const* params, const void* const* grads,
                      void* const* momentum, float lr, float momentum_coef,
                      float weight_decay, int32_t ns_steps, int32_t nesterov,
                      void* workspace, size_t workspace_bytes, void* hip_stream);

/* The buffer checks of muon_step, without enqueuing anything.  Beyond the
 * argument rules above (non-NULL params and momentum, 16-byte aligned
 * buffers, a 256-byte aligned workspace of at least
 * muon_plan_workspace_bytes, the current device the plan's), every buffer
 * must be device memory of the plan's device (or managed memory), and each
 * of [params[i], + rows*cols*param size), [grads[i], ...) (unless NULL),
 * [momentum[i], + rows*cols*4), [update_out[i], ...) and the plan's
 * workspace bytes must lie inside one allocation (where HIP reports the
 * allocation; memory mapped through the virtual memory API may not be, and
 * is then taken on trust).  The kernels trust the pointers they are given,
 * so a caller that cannot vouch for its buffers calls this once per new set
 * of addresses, or creates the plan with MUON_PLAN_CHECK_BUFFERS.
 * update_out may be NULL.  Returns MUON_OK, INVALID_ARG or
 * WORKSPACE_TOO_SMALL with the reason in muon_last_error(). */
MUON_API muon_status muon_check_buffers(muon_plan plan, void* const* params, const void* const* grads,
                                        void* const* momentum, void* workspace, size_t workspace_bytes,
                                        float* const* update_out);

/* Size of the library's static workspace (muon_step_static): 64 MiB. */
#define MUON_STATIC_WORKSPACE_BYTES (64u << 20)

/* muon_step without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, allocation-free serving
 * loops, harnesses that forbid hipMalloc).  The step runs exactly as
 * muon_step (same kernels, bitwise the same W and M) but in a workspace the
 * library holds itself: a static device array of MUON_STATIC_WORKSPACE_BYTES
 * on each GPU the library runs on, kept until the process ends.  Nothing is
 * allocated: no hipMalloc, hipFree or allocating library call (launch timing
 * is not recorded on this path, since its events would be created).
 *   - The plan's workspace (muon_plan_workspace_bytes) must fit: a larger
 *     plan gives WORKSPACE_TOO_SMALL and nothing is enqueued.
 *   - Every call on one GPU shares that GPU's array, which keeps whatever
 *     the last call left there; a step writes every byte it later reads, so
 *     nothing needs clearing.  Calls that may overlap on one GPU (other
 *     streams, other threads, other plans) race on the array: order them.
 * Arguments and errors as for muon_step (without workspace and
 * workspace_bytes). */
MUON_API muon_status muon_step_static(muon_plan plan, void* const* params, const void* const* grads,
                                      void* const* momentum, float lr, float momentum_coef, float weight_decay,
                                      int32_t ns_steps, int32_t nesterov, void* hip_stream);

/* muon_step plus, for every i with update_out[i] != NULL, the orthogonalised
 * update O_i (before lr and the shape scale) written as fp32 rows x cols
 * row-major to update_out[i] (device, 16-byte aligned).  W and M are
 * bitwise identical to muon_step's.  update_out may be NULL (no output); a
 * matrix skipped for a NULL gradient leaves its update_out untouched. */
MUON_API muon_status muon_step_debug(muon_plan plan, void* const* params, const void* const* grads,
                            void* const* momentum, float lr, float momentum_coef,
                            float weight_decay, int32_t ns_steps, int32_t nesterov,
                            void* workspace, size_t workspace_bytes, void* hip_stream,
                            float* const* update_out);

/* Launch timing.  While enabled, muon_step records a pair of HIP events on
 * its stream around every launch (a few microseconds per launch; a B*X
 * launch and the launch of its matrices' edge strips on 128 tiles, which
 * follows it, are one record).
 * muon_plan_timing_read waits for the recorded events, and aggregates the
 * launches by (kind, kernel class) into stats[0..capacity), setting *count
 * to the number of entries; with reset != 0 the records are dropped
 * afterwards.  Flops and bytes are the algorithmic work of each launch:
 *   MUON_KERNEL_GRAM  m^2 n flops per matrix (half of the symmetric X X^T)
 *   MUON_KERNEL_POLY  m^3 flops (half of the symmetric A*A)
 *   MUON_KERNEL_BX    2 m^2 n flops (the last one also applies Eq. 1 to the
 *                     parameters, reading and writing W instead of storing O)
 *   MUON_KERNEL_SYMM  m^3 flops (a symmetric m x m product of the Gram-space
 *                     recurrence: G P, P (G P) or P Q; the P_i product itself
 *                     counts as MUON_KERNEL_POLY)
 *   MUON_KERNEL_MOMENTUM  read G, read and write M, write X0 once
 *   MUON_KERNEL_APPLY     only when ns_steps = 0: read W and X0, write W
 * counted for every matrix of the launch, also ones skipped for a zero
 * gradient.  Timing must be read on the thread that steps the plan. */
typedef enum muon_kernel_kind {
  MUON_KERNEL_MOMENTUM = 0,
  MUON_KERNEL_FINALIZE = 1,
  MUON_KERNEL_GRAM = 2,
  MUON_KERNEL_POLY = 3,
  MUON_KERNEL_BX = 4,
  MUON_KERNEL_APPLY = 5,
  MUON_KERNEL_SYMM = 6
} muon_kernel_kind;

typedef struct muon_kernel_stat {
  int32_t kind;                      /* muon_kernel_kind */
  int32_t kernel_class;              /* GEMM class, -1 for elementwise kernels */
  int64_t launches;
  double total_ms;                   /* sum of event-measured launch durations */
  double algo_flops;                 /* summed over the launches */
  double algo_bytes;
} muon_kernel_stat;

MUON_API muon_status muon_plan_set_timing(muon_plan plan, int32_t enable);
MUON_API muon_status muon_plan_timing_read(muon_plan plan, muon_kernel_stat* stats, int32_t capacity,
                                           int32_t* count, int32_t reset);

MUON_API const char* muon_status_string(muon_status s);

/* Thread-local description of the last failure on this thread ("" if none). */
MUON_API const char* muon_last_error(void);

MUON_API int32_t muon_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MUON_MI355X_H */
