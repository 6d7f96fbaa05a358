/*
 * curvadion.h — C ABI of the CurvaDion optimizer step on AMD Instinct MI355X
 * (gfx950).
 *
 * One call performs one step of the paper's Algorithm 2 (CurvaDion, Sec. 2.2)
 * for one weight matrix ("layer") or for a group of layers:
 *
 *   B = M + G                                   buffer update
 *   RMMC = |‖B‖_F - prev| / (prev + eps); prev = ‖B‖_F     (Eq. 1 as executed)
 *   g = max over the layers of RMMC;  sync = g > tau      gate
 *   sync:  P~ = B Q;  P = Orthogonalize(P~);  R = B^T P   power iteration
 *          M = B - (1 - mu) P R^T                     error feedback
 *          Q = ColumnNormalize(R)
 *          X = X - eta sqrt(m/n) P Q^T                weight update
 *   local: M = B;  X = X - eta_local G                (Q unchanged)
 *
 * The sync branch is the Dion step of Algorithm 1 (Sec. 1.1).  With one GPU
 * the data-parallel all-reduces of both algorithms are identities.
 *
 * Memory: every matrix argument is a DEVICE pointer into the memory of the GPU
 * that is current when the layer is created, row-major and contiguous
 * (leading dimension = number of columns), 16-byte aligned.  The caller owns
 * G (read only), M, X (m x n fp32, updated in place) and Q (n x r fp32,
 * updated in place on sync steps).  The library owns its workspace (the
 * P~/P/R panels, Gram and factor matrices, partial sums) and the per-layer
 * prev_norm; both live until cd_destroy.
 *
 * Ordering: all work is ordered on the HIP stream passed to a step call
 * (NULL = the default stream).
 *
 * Blocking and asynchronous steps.  A step call that asks for a result on
 * the host (`out`, or `rmmc_per_layer` of a group step, not NULL) blocks the
 * calling host thread once, after the RMMC gate, until the gate's output has
 * reached the host (the gate kernel writes it into pinned host memory; this
 * single device-to-host crossing stands in for the max all-reduce).  Under
 * the RMMC policy the branch is enqueued after that read, as it depends on
 * it; the other policies fix the branch in advance and enqueue it before the
 * read, so the GPU does not idle through the round trip.  A step call with no
 * host output is asynchronous: it enqueues the whole step and returns without
 * waiting for anything.  The gate then leaves its decision in device memory,
 * and under the RMMC policy both branches are enqueued, each of their kernels
 * returning at once when its branch was not taken (a few microseconds per
 * kernel on the GPU's timeline: the price of not waiting).  The results are
 * bit-identical to those of blocking steps over the same inputs.
 * cd_layer_last_result / cd_group_last_result read the outcome of the last
 * step later (and report CD_ENONFINITE and CD_ERANKDEF).
 *
 * The call returns once the branch is enqueued.  In a group with layers of several shapes (or
 * more than 32 layers of one shape) the sync branch runs each batch of layers
 * of one shape on its own stream: the caller's stream and up to three streams
 * the group owns (default priority), which wait for the caller's stream before
 * they start and which the caller's stream waits for before anything enqueued
 * after the step; the caller sees one ordered stream either way.  Read M, X, Q
 * only after synchronising the stream.  The sync branch's kernels may still
 * run when the call returns, so the next step of the same layer or group must
 * go to the same stream (or the caller orders the two streams); the library's
 * workspace and the caller's M, X, Q are shared between consecutive steps.
 *
 * Errors: arguments are checked before anything is enqueued; CD_EINVAL leaves
 * every buffer and the layer state untouched.  The library cannot see the
 * extent of a device buffer: a buffer smaller than the sizes above is read or
 * written out of bounds.  A HIP failure (CD_EHIP) after the gate has run
 * leaves the step half done (prev_norm and the step counter advanced, the
 * branch partly enqueued); restore M, X, Q and the layer state from a
 * checkpoint before going on.  No C++ exception crosses this interface.
 * cd_last_error() returns a thread-local message for the last failing call on
 * the calling thread.
 *
 * Threads: calls on different layers and groups may come from different host
 * threads; one layer (or a group, or groups that share a layer) must not be
 * stepped from two threads at once.
 */
#ifndef CURVADION_H
#define CURVADION_H

#ifdef __cplusplus
extern "C" {
#endif

#define CD_ABI_VERSION 3

typedef enum cd_status {
  CD_OK = 0,
  CD_EINVAL = -1,      /* invalid argument; nothing was enqueued */
  CD_ENOMEM = -2,      /* device or host allocation failed */
  CD_EHIP = -3,        /* a HIP runtime call failed; see cd_last_error() */
  CD_ENONFINITE = -4,  /* some ‖B‖ was NaN/Inf; the step still ran (local branch) */
  CD_ERANKDEF = -5     /* from cd_*_last_result: the last step synced and some
                          layer's P~ was numerically rank deficient; every
                          output was still written (see cd_layer_rank_deficient) */
} cd_status;

typedef enum cd_dtype { CD_F32 = 0, CD_BF16 = 1 } cd_dtype;

/* How the branch is chosen (Algorithm 2 gate, or a fixed policy). */
typedef enum cd_policy {
  CD_POLICY_RMMC = 0,         /* sync iff max_l RMMC_l > tau (Algorithm 2) */
  CD_POLICY_ALWAYS_SYNC = 1,  /* every step syncs: Dion, Algorithm 1 */
  CD_POLICY_NEVER_SYNC = 2,   /* every step takes the local branch */
  CD_POLICY_EVERY_H = 3       /* sync on steps H, 2H, ...: Scheduled Sync Dion (Sec. 4.3) */
} cd_policy;

typedef struct cd_layer_desc {
  int m;                    /* rows of the weight matrix (and of P) */
  int n;                    /* columns (rows of Q and R) */
  int r_max;                /* largest rank any step of this layer will use;
                               1 <= r_max <= min(m, n); sizes the workspace */
  cd_dtype grad_dtype;      /* element type of G: fp32 or bf16 */
  double tau;               /* gate threshold (strict >) */
  double eps;               /* RMMC denominator guard; the paper leaves it
                               unstated, 1e-8 is the usual choice; >= 0 */
  double eta_local_scale;   /* eta_local = eta_local_scale * eta; >= 0 */
  cd_policy policy;
  int H;                    /* period for CD_POLICY_EVERY_H (>= 1), else ignored */
  double weight_decay;      /* decoupled weight decay lambda >= 0: each step first
                               scales X by (1 - eta * lambda), in either branch;
                               M is untouched.  0 = Algorithm 2 exactly.  (The
                               experiments of Sec. 4 use 0.01 without stating the
                               form; this is the decoupled reading.) */
} cd_layer_desc;

typedef struct cd_result {
  double rmmc;       /* the gate statistic: max over the layers of RMMC */
  int sync_flag;     /* 1 = the sync branch ran, 0 = the local branch ran */
} cd_result;

typedef struct cd_layer cd_layer;
typedef struct cd_group cd_group;

/* Create one layer on the current device: allocates the workspace for
 * (m, n, r_max), sets prev_norm = 0 and the step counter to 0 (Algorithm 2
 * initialisation).  CD_EINVAL for a NULL pointer, a non-positive size,
 * r_max > min(m, n), an unknown dtype or policy, eps < 0, tau NaN, a negative
 * or non-finite weight_decay, or H < 1 under CD_POLICY_EVERY_H. */
cd_status cd_layer_create(const cd_layer_desc* desc, cd_layer** out);

/* One step for one layer (Algorithm 2 with the max taken over this layer
 * alone).  G: m x n of desc.grad_dtype; M, X: m x n fp32; Q: n x r fp32.
 * mu in [0, 1], eta finite and >= 0, 1 <= r <= r_max.  `stream` is a
 * hipStream_t (NULL = default stream).  `out` (host) receives the statistic
 * and the branch taken; NULL makes the step asynchronous (see the top of this
 * header).  Returns CD_OK, or CD_ENONFINITE after a blocking step whose norm
 * was not finite, or an error before any work. */
cd_status cd_step(cd_layer* layer, const void* G, float* M, float* X, float* Q,
                  float mu, float eta, int r, void* stream, cd_result* out);

/* Free the layer and its workspace.  Destroy any group that refers to the
 * layer first.  NULL is accepted (no-op). */
cd_status cd_destroy(cd_layer* layer);

/* For callers that cannot allocate memory while they step (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): one
 * step of one layer as cd_step computes it, that allocates nothing.  Every
 * buffer the step needs besides its inputs and outputs lives in one fixed
 * array of CD_STATIC_SCRATCH_BYTES per device, which the library holds from
 * its first use on a device until the process ends; the first call on a
 * device looks up that array's address.
 *
 * There is no layer object: `desc` describes the layer (as for
 * cd_layer_create; r <= desc->r_max), and the caller owns its state,
 * `prev_norm` (a DEVICE pointer to one double, 0 before the first step, read
 * and written by the step) and `*step` (host, the number of steps taken,
 * incremented).  G, M, X, Q, mu, eta, r, stream and out as for cd_step.  The
 * call blocks the host until the gate's output has been copied back
 * (hipMemcpyAsync into the call's stack, then a stream synchronisation), then
 * enqueues the branch and returns.  Without state between calls there is no
 * branch prediction: under CD_POLICY_RMMC the skip update is a pass of its
 * own (fixed policies fuse it as cd_step does), so results match cd_step's
 * to within an fp32 rounding of X.  Rank deficiency is handled as in cd_step
 * but not reported.
 *
 * CD_EINVAL (nothing enqueued) for the descriptor and argument errors of
 * cd_layer_create and cd_step, a NULL or misaligned prev_norm, a NULL step,
 * and for a layer whose workspace at rank r exceeds CD_STATIC_SCRATCH_BYTES
 * (the message gives both sizes; such layers need cd_step).
 *
 * Every call on one device uses that device's one array, whose contents the
 * next call overwrites: calls whose work overlaps on one device (different
 * streams, or different host threads on streams not ordered with each other)
 * race, and must be ordered by the caller.  Calls from several host threads
 * are serialised on the host. */
#define CD_STATIC_SCRATCH_BYTES (64u << 20)
cd_status cd_step_static(const cd_layer_desc* desc, double* prev_norm, long long* step, const void* G,
                         float* M, float* X, float* Q, float mu, float eta, int r, void* stream,
                         cd_result* out);

/* Group layers so that one step takes the max of RMMC over all of them before
 * any layer branches (Algorithm 2).  All layers must share grad_dtype, tau,
 * policy, H and device; the group refers to (does not own) the layers, and
 * copies the pointer array.  n_layers >= 1. */
cd_status cd_group_create(cd_layer* const* layers, int n_layers, cd_group** out);

/* One step for every layer of the group.  G, M, X, Q are HOST arrays of
 * n_layers DEVICE pointers, in the order the group was created with; shapes as
 * for cd_step with each layer's (m, n) and the common rank r (1 <= r <= every
 * layer's r_max).  `rmmc_per_layer` (host, may be NULL) receives n_layers
 * values of RMMC_l.  With both `rmmc_per_layer` and `out` NULL the step is
 * asynchronous.  Returns CD_OK, or CD_ENONFINITE after a blocking step, or an
 * error before any work. */
cd_status cd_group_step(cd_group* group, const void* const* G, float* const* M,
                        float* const* X, float* const* Q, float mu, float eta, int r,
                        void* stream, double* rmmc_per_layer, cd_result* out);

cd_status cd_group_destroy(cd_group* group);

/* The outcome of the group's last step (of the layer's last cd_step): waits
 * until that step's work has finished on the device (its completion event;
 * other work on the device is not waited for), then writes the gate
 * statistic and the branch taken to `out` and, for a group, the n_layers
 * values of RMMC_l to `rmmc_per_layer` (both host, may be NULL).  Returns
 * CD_OK, CD_ENONFINITE (some ‖B‖ was not finite: the local branch ran),
 * CD_ERANKDEF (the step synced and some layer's P~ was numerically rank
 * deficient; the outputs were still written), or CD_EINVAL before the first
 * step. */
cd_status cd_group_last_result(cd_group* group, double* rmmc_per_layer, cd_result* out);
cd_status cd_layer_last_result(cd_layer* layer, cd_result* out);

/* Checkpoint support: the library-owned state of a layer is prev_norm (the
 * last ‖B‖_F) and the step counter; M, X and Q belong to the caller.  These
 * calls synchronise the device. */
cd_status cd_layer_get_state(const cd_layer* layer, double* prev_norm, long long* step);
cd_status cd_layer_set_state(cd_layer* layer, double prev_norm, long long step);

/* Device pointers to the orthonormal P (m x r) and to R = B^T P (n x r) of
 * the layer's last sync step, row-major, owned by the library and valid until
 * its next step or cd_destroy.  For inspection and tests. */
cd_status cd_layer_last_factors(const cd_layer* layer, const float** P, const float** R);

/* Waits until the layer's last step has finished on the device (the
 * completion event of the group that took it, not the whole device), then
 * sets *flag = 1 if the last sync step found P~ numerically rank deficient (a
 * Cholesky pivot at or below 1e-13 times the largest Gram diagonal).  M, X and Q were still written and P
 * still has orthonormal columns: past the numerical rank it is completed with
 * fixed pseudo-random directions orthonormalised against the other columns
 * (as a Householder QR factor is completed), so those columns, and the
 * matching columns of R and Q, are not unique.  *flag = 0 otherwise. */
cd_status cd_layer_rank_deficient(const cd_layer* layer, int* flag);

/* Kernel timing, for measurement.  While timing is on, every kernel launch of
 * the group's steps is bracketed by two HIP events recorded on the launch
 * stream.  While every kind is bracketed (the default), the sync branch runs
 * its batches one after another on the caller's stream, so that each interval
 * times its kernel alone; with a narrower selection (see below) the schedule
 * is the untimed one, and a bracketed sync-branch launch also counts the time
 * it waits for CUs that kernels of other batches hold.  cd_group_kernel_times() waits for the last recorded event, then
 * returns one entry per kernel kind that ran since timing was switched on (or
 * since the previous query): launch count, summed event time, and the
 * algorithmic bytes and flops of those launches (compulsory traffic of the
 * inputs and outputs each kernel must touch, and the flops of its arithmetic
 * as written in the method; neither counts re-reads or padding).  Records are
 * cleared by each query.  *count receives the number of kinds available even
 * when it exceeds max_kinds. */
typedef struct cd_kernel_time {
  char name[32];
  int launches;
  double total_ms;
  double bytes;
  double flops;
} cd_kernel_time;
cd_status cd_group_set_timing(cd_group* group, int enable);
cd_status cd_group_kernel_times(cd_group* group, cd_kernel_time* out, int max_kinds, int* count);

/* Restricts the bracketing to the kernel kinds named in `kinds`, a
 * comma-separated list of the names cd_group_kernel_times() reports (NULL or
 * "" = every kind, the default).  The events cost several microseconds of
 * idle time at each bracketed launch, so a measurement of whole steps
 * brackets only the kernel it reports.  Applies from the next step; the
 * setting survives cd_group_set_timing().  CD_EINVAL for an unknown name
 * (the previous setting is then kept). */
cd_status cd_group_set_timing_kinds(cd_group* group, const char* kinds);

/* Thread-local text of the last error on this thread ("" if none). */
const char* cd_last_error(void);

/* CD_ABI_VERSION of the built library. */
int cd_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CURVADION_H */
