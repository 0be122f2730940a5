/*
 * pgc.h -- C ABI of one pipelined-gradient-coding (PGC) training step with all
 * n simulated workers on one gfx950 GPU.
 *
 * Method: Pipelined Gradient Coding (Su and Li).  n workers each hold c = s + 1
 * of the n dataset partitions (fractional repetition, FR, or cyclic repetition,
 * CR; Sec. III).  At step t >= 1 each worker evaluates the gradient of ONE of
 * its partitions, the one in slot (t - 1) mod c, keeps the latest gradient of
 * every partition it holds, and sends one coded gradient built from them
 * (Sec. IV-A for FR, Sec. V-B for CR).  The master ignores up to s stragglers,
 * decodes the survivors' coded gradients and takes a gradient step (Sec. III).
 * Step t = 0 evaluates every held partition (the pipeline warm-up, Sec. IV-A).
 *
 * Conventions for every call:
 *   - Every function returns a pgc_status (0 = success) unless stated.  No
 *     exception or abort crosses the ABI.  On failure pgc_last_error(ctx)
 *     gives a human-readable reason.
 *   - "device pointer" = memory on the GPU the context runs on (e.g. a torch
 *     tensor's data_ptr()); "host pointer" = ordinary CPU memory.
 *   - The library never allocates GPU memory and never frees caller memory.
 *     All device scratch lives in a caller-provided workspace, except the
 *     fixed static array of pgc_step_noalloc.
 *   - A context is not thread-safe; use one context per stream.
 *   - Device work is enqueued on the context's stream and is not synchronised;
 *     device pointers must stay valid until the stream has passed the work.
 */
#ifndef PGC_H
#define PGC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pgc_ctx pgc_ctx;

/* Placement / coding scheme. */
enum pgc_scheme {
  PGC_FR = 0,      /* PGC-FR, Sec. IV-A: groups of c workers share c partitions; needs c | n */
  PGC_CR = 1,      /* PGC-CR, Sec. V-B: cyclic placement, unit coefficients, scale 1/(|J| c) */
  PGC_CR_REAL = 2, /* naive pipelined CR, Sec. V-A: real coefficients, exact-sum decode */
  PGC_IS_SGD = 3   /* ignore-straggler SGD, Sec. VI-A: c = 1, mean of the survivors' gradients */
};

/* Model whose per-partition gradient is evaluated. */
enum pgc_model {
  PGC_LOGISTIC = 0, /* f = log(1 + e^z) - y z, z = x . w, y in {0, 1}; X fp32, y fp32 */
  PGC_LSQ = 1,      /* f = (z - y)^2 / 2; X fp32, y fp32 */
  PGC_MLP = 2       /* d_in -> hidden (ReLU) -> classes, softmax cross-entropy; X bf16, y int32 */
};

enum pgc_status {
  PGC_OK = 0,
  PGC_EINVAL = -1,      /* bad argument: sizes, null pointer, unknown enum, alignment */
  PGC_ESTRAGGLERS = -2, /* more than s = c - 1 stragglers, or an FR group with no survivor */
  PGC_ESINGULAR = -3,   /* the real-valued code cannot decode (residual above 1e-9) */
  PGC_EDEVICE = -4,     /* a HIP runtime error (asynchronous faults surface on a later call) */
  PGC_ESTATE = -5       /* calls out of order (e.g. pgc_step before pgc_bind_workspace) */
};

/* Straggler-mask policies of pgc_make_mask. */
enum pgc_mask_policy {
  PGC_POLICY_EXACT = 0,         /* exactly `cap` stragglers, uniformly chosen */
  PGC_POLICY_UNIFORM_COUNT = 1, /* count uniform in {0..cap}, then uniformly chosen */
  PGC_POLICY_BERNOULLI = 2,     /* each worker with probability p, at most `cap` kept */
  PGC_POLICY_SLOWEST = 3        /* the `cap` slowest under i.i.d. exponential delays: worker i
                                   draws u_i (its delay is -mean ln(1 - u_i)); the `cap`
                                   largest u_i straggle, lower index first on ties */
};

/* Kernels whose GPU time pgc_kernel_time reports. */
enum pgc_kernel {
  PGC_KERNEL_GRADIENT = 0,    /* linear models: per-partition gradient, one HBM pass over the rows */
  PGC_KERNEL_REDUCE = 1,      /* MLP: head partial sums -> ring slots */
  PGC_KERNEL_CODE = 2,        /* encode + masked decode + update (linear models: also folds the
                                 gradient kernel's partial sums into the ring first) */
  PGC_KERNEL_MLP_CAST = 3,    /* MLP: bf16 copies of W1 and W2 */
  PGC_KERNEL_MLP_FORWARD = 4, /* MLP: H = relu(X W1 + b1), bf16 MFMA GEMM */
  PGC_KERNEL_MLP_HEAD = 5,    /* MLP: logits, softmax, dZ2, dZ1 and the small-layer gradients */
  PGC_KERNEL_MLP_WGRAD = 6,   /* MLP: dW1 = X^T dZ1 per partition, bf16 MFMA GEMM */
  PGC_KERNEL_COUNT = 7
};

#define PGC_MAX_N 256           /* largest number of workers */
/* MLP shape limits: d_in % 8 == 0, d_in <= 2^20, hidden % 256 == 0, hidden <= 1024,
 * 1 <= classes <= 16. */
#define PGC_MLP_MAX_D_IN 1048576
#define PGC_MLP_MAX_HIDDEN 1024
#define PGC_MLP_MAX_CLASSES 16
#define PGC_MAX_LINEAR_D 32768  /* largest feature count of the linear models (d % 4 == 0) */
#define PGC_MAX_LINEAR_D_UNALIGNED 8192 /* ... when d % 4 != 0 or X is not 16-byte aligned */

typedef struct pgc_config {
  int32_t model;      /* enum pgc_model */
  int32_t d_in;       /* features per sample: equals d of pgc_init for the linear models */
  int64_t N;          /* samples; N > 0 and N % n == 0 (partition k = rows [k N/n, (k+1) N/n)) */
  int32_t hidden;     /* MLP hidden width (0 for linear models) */
  int32_t classes;    /* MLP classes (0 for linear models) */
  uint64_t code_seed; /* PGC_CR_REAL: seed of the random matrix defining the code; else ignored */
} pgc_config;

/* Create a context for `scheme` with n workers (= partitions), c partitions per
 * worker (s = c - 1 tolerated stragglers) and a parameter vector of length d.
 * Requires 1 <= c <= n <= PGC_MAX_N, d >= 1, c | n for PGC_FR and c = 1 for
 * PGC_IS_SGD (which ignores up to n - 1 stragglers).
 * Sec. III (placements), Sec. IV-A, Sec. V-A, Sec. V-B.  Touches no GPU.
 * *out receives the handle (NULL on failure; reason via pgc_strerror). */
int pgc_init(pgc_ctx** out, int scheme, int n, int c, int64_t d);

/* Fix the model and dataset shape.  For the linear models d_in must equal d;
 * for PGC_MLP d must equal d_in*hidden + hidden + hidden*classes + classes and
 * the shape must meet the PGC_MLP_* limits.
 * For PGC_CR_REAL this builds the n x n real-valued encoding matrix from
 * code_seed (PGC_ESINGULAR if a row's defining system is singular).
 * Resets the step counter to 0 and invalidates a bound workspace.  Host only. */
int pgc_configure(pgc_ctx* ctx, const pgc_config* cfg);

/* Pipelining on (1, the default: PGC) or off (0: gradient coding).  With it
 * off every step evaluates all c partitions each worker holds at the current
 * w, as the warm-up step does, so the coded gradients are current (GC,
 * Sec. III / IV-A); with FR or PGC_CR_REAL the decode then recovers the full
 * gradient exactly and the run coincides with distributed gradient descent.
 * Takes effect from the next pgc_step.  Host only. */
int pgc_set_pipelining(pgc_ctx* ctx, int enabled);

/* Stream (a hipStream_t, NULL = the null stream) on which pgc_step and the
 * pgc_read_* calls enqueue work.  Default: the null stream.  When the stream
 * changes, the call first synchronises the old stream, so the next step sees
 * everything earlier steps wrote; if either stream is being captured into a
 * graph it does not (that would end the capture) and the caller must order
 * the two streams itself. */
int pgc_set_stream(pgc_ctx* ctx, void* hip_stream);

/* Bytes of device workspace the configured context needs (256-byte aligned). */
int pgc_workspace_bytes(const pgc_ctx* ctx, size_t* bytes);

/* Bind caller-owned device memory of at least pgc_workspace_bytes bytes,
 * 256-byte aligned, used until the context is destroyed or rebound.  It holds
 * the gradient ring, the coded and decoded gradients and per-block partial
 * sums.  Synchronises the context stream (work enqueued before may still use
 * the old workspace), then uploads the encoding table with a synchronous copy.
 * Resets t to 0. */
int pgc_bind_workspace(pgc_ctx* ctx, void* dev_workspace, size_t bytes);

/* One PGC step at the context's current step t, then t += 1.
 *   X    device; row-major N x d_in: fp32 (linear models) or bf16 bit patterns (MLP).
 *   y    device; N labels: fp32 {0,1} (logistic), fp32 (least squares), int32 class (MLP).
 *        MLP classes lie in [0, classes); the kernels only compare a label with
 *        class indices, so another value indexes no memory: its row's one-hot
 *        target is all zero.
 *   w    device; fp32 parameter vector of length d, updated in place:
 *        w <- w - lr * ghat, ghat the decoded gradient (Sec. III).  MLP layout:
 *        W1[d_in][hidden] row-major, b1[hidden], W2[hidden][classes], b2[classes].
 *   straggler_mask  host; n bytes, nonzero = worker straggles this step.  Read
 *        before the call returns.  Stragglers still evaluate and store; only
 *        their coded gradients are left out of the decode (Sec. V-B).
 * t = 0 is the warm-up: every worker evaluates all c held partitions at w
 * (Sec. IV-A).  For t >= 1 worker i evaluates its slot (t - 1) mod c.
 * lr must be finite (PGC_EINVAL otherwise).
 * Errors (PGC_EINVAL, PGC_ESTRAGGLERS, PGC_ESINGULAR, PGC_ESTATE) are detected
 * before any work is enqueued: a rejected step has no effect and t does not
 * advance.  Returns without synchronising the stream. */
int pgc_step(pgc_ctx* ctx, const void* X, const void* y, float* w,
             const uint8_t* straggler_mask, float lr);

/* Size of the fixed device array pgc_step_noalloc keeps its scratch in. */
#define PGC_NOALLOC_SCRATCH_BYTES (32u << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * step as pgc_step, same arguments, checks, errors and results bit for bit,
 * for the linear models (PGC_LOGISTIC, PGC_LSQ) only, with the gradient
 * kernel's per-block partial sums in a library-owned static device array of
 * PGC_NOALLOC_SCRATCH_BYTES bytes (one per GPU, held until the process ends)
 * instead of the bound workspace.  The workspace still holds the ring, the
 * coded and decoded gradients (its partial-sum region is not used).
 * Calls no hipMalloc, hipFree or other allocating routine (with kernel timing
 * off; pgc_set_timing creates its events on first use).
 * The array used is the one of the current device, which must be the GPU of
 * the context's stream (as for any launch on that stream); its address is
 * looked up on the first call on each device.
 * Errors: PGC_EINVAL for the MLP, or when the configured shape's partial sums
 * exceed PGC_NOALLOC_SCRATCH_BYTES (at most 1024 gradient blocks of d floats);
 * PGC_EDEVICE if the array's device address cannot be found.  Every call on a
 * GPU uses that GPU's one array: calls that overlap on one GPU (contexts on
 * different streams) race and must be ordered by the caller.  The array keeps
 * the last call's contents; every step overwrites what it reads. */
int pgc_step_noalloc(pgc_ctx* ctx, const void* X, const void* y, float* w,
                     const uint8_t* straggler_mask, float lr);

/* Decode coefficients of `straggler_mask` (host, n bytes) for this context
 * (IS_SGD: d = 1 for every survivor, scale 1/|J|):
 * survivors_out[0..*n_survivors_out) = the non-stragglers J in ascending order;
 * d_out[m] = the unscaled weight of coded gradient J[m]; *scale_out = the
 * common scale; decoded gradient = scale * sum_m d[m] * coded_{J[m]}.
 *   FR:      d = 1 for the lowest-index survivor of each group, else 0; scale 1/n.
 *   CR:      d = 1 for every survivor; scale 1/(|J| c), i.e. 1/(n mu) (Sec. V-B).
 *   CR_REAL: minimum-norm solution of B_J^T d = 1 (fp64); scale 1/n (Sec. V-A).
 * d_out and survivors_out must hold n entries.  Host only; needs pgc_configure. */
int pgc_decode_coeffs(const pgc_ctx* ctx, const uint8_t* straggler_mask,
                      double* d_out, double* scale_out,
                      int32_t* survivors_out, int32_t* n_survivors_out);

/* Placement (host, n*c int32, row-major): out[i*c + l] = partition worker i
 * holds in slot l.  FR: (i / c) * c + l; CR: (i + l) mod n (Sec. III). */
int pgc_placement(const pgc_ctx* ctx, int32_t* out);

/* Partition evaluated by each worker at step t >= 1 (host, n int32):
 * out[i] = placement[i][(t - 1) mod c] (Sec. IV-A, Sec. V-B).  t = 0
 * evaluates every slot (see pgc_placement) and is rejected with PGC_EINVAL. */
int pgc_schedule(const pgc_ctx* ctx, int64_t t, int32_t* out);

/* Encoding matrix (host, n*n fp64, row-major): out[j*n + k] = coefficient of
 * partition k's gradient in worker j's coded gradient.  0/1 for FR and CR;
 * the real-valued matrix for CR_REAL (needs pgc_configure). */
int pgc_encoding_matrix(const pgc_ctx* ctx, double* out);

/* Number of distinct coded gradients kept on the device: n / c for FR (a
 * group's members send identical words), n for CR and CR_REAL. */
int pgc_num_coded(const pgc_ctx* ctx, int32_t* out);

/* Straggler mask of step t (host, n bytes of 0/1) drawn from SplitMix64 seeded
 * with `seed` under `policy` (enum pgc_mask_policy) with cap `cap` and, for
 * PGC_POLICY_BERNOULLI, probability p.  Independent of any context. */
int pgc_make_mask(uint64_t seed, int64_t t, int policy, int n, int cap, double p,
                  uint8_t* out);

/* One step of the simulated straggler model of Sec. VI-B (independent of any
 * context; host only).  Worker i draws u_i (draw i of step t of the SplitMix64
 * stream `seed`, as for pgc_make_mask) and finishes after
 * compute_seconds + delay_i with the exponential delay
 * delay_i = -mean_delay * ln(1 - u_i).  The master waits for the n - s fastest
 * workers: `mask` (n bytes) marks the s others (identical to pgc_make_mask with
 * PGC_POLICY_SLOWEST and cap s), `*step_seconds` is the (n - s)-th smallest
 * finish time (s = 0: the slowest worker, as DGD waits for).  `delays` (n
 * doubles, may be NULL) receives every delay_i.  compute_seconds is the
 * worker's compute time for the step, equal across workers.  PGC_EINVAL when
 * n is outside [1, PGC_MAX_N], s outside [0, n - 1], t < 0, mean_delay or
 * compute_seconds negative or not finite, or mask / step_seconds is NULL. */
int pgc_delay_step(uint64_t seed, int64_t t, int n, int s, double mean_delay,
                   double compute_seconds, uint8_t* mask, double* delays, double* step_seconds);

/* Output `index` (0-based) of the SplitMix64 stream seeded with `seed`. */
int pgc_splitmix64(uint64_t seed, uint64_t index, uint64_t* out);

/* Copy device-resident state to a device buffer of d floats, on the context
 * stream (asynchronous).  Ring: the gradient of the partition worker `worker`
 * holds in slot `slot` as last evaluated; coded: the coded gradient of
 * `index` (a group for FR, a worker for CR); decoded: the last step's ghat. */
int pgc_read_ring(const pgc_ctx* ctx, int worker, int slot, float* dev_out);
int pgc_read_coded(const pgc_ctx* ctx, int index, float* dev_out);
int pgc_read_decoded(const pgc_ctx* ctx, float* dev_out);

/* Checkpoint and resume of the pipeline.  A pipelined step reads the latest
 * gradient of every partition a worker holds, most of them computed at
 * earlier steps (Sec. IV-A, Sec. VI-A), so a run resumes on the same
 * trajectory only if those copies come back; starting over would repeat the
 * warm-up (Sec. IV-A) at the current w and change every later step.  The saved
 * state is the step counter t and the gradient ring.  The parameter vector w
 * is the caller's own and is checkpointed by the caller.
 *
 * pgc_state_bytes: bytes of a saved state for this configured context (a
 *   256-byte header, then c planes of n gradient copies for CR and CR_REAL,
 *   one for FR and IS_SGD).  Host only.
 * pgc_save_state: writes the state into caller-owned device memory
 *   (`bytes` >= pgc_state_bytes, 16-byte aligned) on the context stream,
 *   asynchronously, as of the work enqueued before the call.  Needs a bound
 *   workspace.
 * pgc_load_state: restores a state saved by a context of the same scheme, n,
 *   c, model shape and (CR_REAL) code seed: the ring, and t.  Synchronises the
 *   context stream to read and check the header first; a buffer that is not a
 *   saved state, or one from another configuration, is rejected with
 *   PGC_EINVAL before anything changes.  Pipelining on or off is not part of
 *   the state. */
int pgc_state_bytes(const pgc_ctx* ctx, size_t* bytes);
int pgc_save_state(const pgc_ctx* ctx, void* dev_out, size_t bytes);
int pgc_load_state(pgc_ctx* ctx, const void* dev_in, size_t bytes);

/* Current step counter t (the number of completed pgc_step calls since configure/bind). */
int pgc_get_step(const pgc_ctx* ctx, int64_t* t);

/* Per-kernel GPU timing with HIP events recorded around each launch on the
 * context stream.  pgc_set_timing(ctx, mask) times the kernels whose bit
 * (1 << enum pgc_kernel) is set in `mask` (0 disables timing, -1 times all)
 * and clears the totals; pgc_kernel_time synchronises on the recorded events
 * and returns the summed milliseconds and launch count of `kernel` since. */
int pgc_set_timing(pgc_ctx* ctx, int kernel_mask);
int pgc_kernel_time(pgc_ctx* ctx, int kernel, double* total_ms, int64_t* launches);

/* Time only one launch in `period` of each selected kernel (the first, then
 * every period-th; default 1 = every launch), so that the ~6 us an event pair
 * adds to a step is paid on a sample only.  pgc_kernel_time then reports the
 * sampled launches.  Restarts the sampling count; PGC_EINVAL if period < 1. */
int pgc_set_timing_period(pgc_ctx* ctx, int64_t period);

/* Text of a status code; last error message of a context (never NULL). */
const char* pgc_strerror(int status);
const char* pgc_last_error(const pgc_ctx* ctx);

/* Release the context (host memory and timing events only). NULL is allowed. */
int pgc_destroy(pgc_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* PGC_H */
