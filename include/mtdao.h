/*
 * mtdao.h -- C ABI of the MT-DAO optimizer hot path on MI355X (gfx950).
 *
 * MT-DAO ("Multi-timescale Distributed Adaptive Optimizers with Local
 * Updates"): every worker m keeps its own parameters x^m, N first-moment
 * EMAs u^{j,m} with their own decay rates beta_{1,j}, and (Adam and ADOPT
 * forms) one second moment v^m.  A local step combines the current gradient
 * and the N moments quasi-hyperbolically with weights (1 - sum_j omega_j)
 * and omega_j (Section 2.3, Algorithm 1 = Adam form; Algorithm 2 = ADOPT
 * form; Algorithm 3 = SGDM form).  Periodically each state is replaced by
 * its mean over the workers, every state on its own period K_x, K_j, K_v
 * (the "t mod K" conditions of the same algorithms, OuterOpt = averaging).
 *
 * On one GPU the M workers (called K "replicas" here) are K resident rows
 * of every state buffer, and the averaging is an on-device mean over the
 * replica axis.
 *
 * Memory layout (all device buffers are caller-owned, e.g. torch tensors):
 *   x      [K][P]  params, fp32 or bf16 (row m = worker m)
 *   u[j]   [K][P]  fp32, j = 0..N-1 (first moments, paper u^{j+1})
 *   v      [K][P]  fp32 (Adam, ADOPT only; NULL for SGDM)
 *   grads  [K][P]  fp32 or bf16, one gradient row per worker per step
 * P is the total element count of one replica's flat multi-tensor buffer
 * (all tensors of the model concatenated); every call covers all tensors of
 * all replicas.  Rows are contiguous with stride P.  Every pointer must be
 * 16-byte aligned.
 *
 * Step numbering: s counts local updates; the k-th call of
 * mtdao_local_step performs update s = start_step + k (1-based).  State S is
 * due for averaging after update s iff its period H_S > 0 and s mod H_S ==
 * 0 (period 0 = never).  This is Algorithm 1's schedule; Algorithms 2 and 3
 * print the same rule with a one-step phase difference for u and v, which
 * is read as a slip (the unified strategy of the wall-clock appendix syncs
 * parameters and all optimizer states together every K steps).
 *
 * Readings where the paper is silent (Algorithm 1's caption omits the bias
 * correction; the clip types are not spelled out):
 *   - Adam bias correction (bias_correction = 1): u_j / (1 - beta_{1,j}^s) and
 *     v / (1 - beta_2^s) with the global s, never reset by averaging; the
 *     gradient term is uncorrected.  ADOPT and SGDM have no correction.
 *   - clip(g, rho): per-replica global L2 norm over all P elements,
 *     scale = min(1, rho / ||g^m||), 1 when the norm is 0.  Adam's v squares
 *     the clipped gradient.
 *   - ADOPT clip(g_hat, c_t): element-wise clamp to [-c_t, c_t], c_t passed
 *     per call.  adopt_order PREV normalises by v from before this step and
 *     the first update (s == 1) only sets v = g^2 (ADOPT as published); CUR
 *     normalises by the freshly updated v, literally as Algorithm 2 prints.
 *
 * Concurrency: calls on one handle must be serialised by the caller; all
 * work is enqueued on the HIP stream passed to each call (NULL = the null
 * stream).  mtdao_local_step and mtdao_sync only enqueue; mtdao_read_state
 * waits for the stream.
 *
 * Errors: every int32_t-returning call returns MTDAO_OK (0) or a negative
 * code; validation happens on the host before anything is enqueued, so a
 * failing call leaves the device state untouched.  mtdao_last_error gives a
 * human-readable message.
 */
#ifndef MTDAO_H
#define MTDAO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MTDAO_MAX_N 4            /* max number of first moments N          */
#define MTDAO_MAX_REPLICAS 1024  /* max K                                   */
#define MTDAO_SYNC_AUTO 0xFFFFFFFFu

/* forms: Algorithm 1 / Algorithm 2 / Algorithm 3 */
enum { MTDAO_ADAM = 0, MTDAO_ADOPT = 1, MTDAO_SGDM = 2 };
/* storage types of params and gradients (moments are always fp32) */
enum { MTDAO_F32 = 0, MTDAO_BF16 = 1 };
/* ADOPT normalisation order */
enum { MTDAO_ADOPT_PREV = 0, MTDAO_ADOPT_CUR = 1 };
/* Where the averaging of a first moment sits within a step:
 *   MTDAO_SYNC_AFTER_STEP      the step uses each worker's own u^j; the mean
 *                              is the base of the next step (Algorithms 1-3)
 *   MTDAO_SYNC_MOMENTA_IN_STEP the mean of a due u^j replaces it before this
 *                              step's direction uses it (the probabilistic
 *                              variant, Algorithm 4; SGDM form only).  Its
 *                              moment averaging happens inside
 *                              mtdao_step_sync; mtdao_sync then accepts only
 *                              the x bit. */
enum { MTDAO_SYNC_AFTER_STEP = 0, MTDAO_SYNC_MOMENTA_IN_STEP = 1 };
/* OuterOpt at an averaging event of x (the Require blocks' OuterOpt,
 * averaging by default):
 *   MTDAO_OUTER_AVERAGE   every worker restarts from the mean E_m[x^m]
 *   MTDAO_OUTER_NESTEROV  outer Nesterov step on the outer parameters xo
 *                         (fp32 [P]) with outer momentum b (fp32 [P]):
 *                         d = xo - E_m[x^m]; b = mu b + d;
 *                         xo = xo - outer_lr (d + mu b); every worker
 *                         restarts from xo.  outer_lr = 1, mu = 0 is
 *                         averaging.  Needs sync_order AFTER_STEP.  The
 *                         outer step runs at most once per step s: a
 *                         later averaging of x at the same s (mtdao_sync
 *                         after mtdao_step_sync, a repeated mtdao_sync,
 *                         mtdao_sync_stats after mtdao_sync) only averages
 *                         rows that are already equal, so it changes
 *                         nothing. */
enum { MTDAO_OUTER_AVERAGE = 0, MTDAO_OUTER_NESTEROV = 1 };
/* State ids of mtdao_read_state beyond the per-worker states
 * (0 = x, 1..N = u^j, N+1 = v): the outer parameters and momentum of the
 * Nesterov OuterOpt (fp32, one row: replica must be 0). */
#define MTDAO_STATE_X_OUTER 6
#define MTDAO_STATE_OUTER_MOM 7

/* Averaging diagnostics (mtdao_sync_stats), per averaged state, from its
 * values before averaging, over all P elements (Section 4.1, other
 * metrics).  The vectors are c^m = S^m, or, for x under the Nesterov
 * OuterOpt, the pseudo-gradients c^m = x_outer - x^m; cbar is their mean:
 *   [MTDAO_STAT_MEAN_SQ]      ||cbar||^2
 *   [MTDAO_STAT_VARIANCE]     (1/K) sum_m ||c^m - cbar||^2  (cross-worker variance)
 *   [MTDAO_STAT_OUTER_SQ]     ||x_outer||^2 before the outer step (x under
 *                             Nesterov; 0 otherwise); the relative change
 *                             of the model over the round is
 *                             sqrt(MEAN_SQ / OUTER_SQ)
 *   [MTDAO_STAT_WORKER_SQ + m]  ||c^m||^2
 *   [MTDAO_STAT_WORKER_DOT + m] <c^m, cbar>   (cosine = DOT / sqrt(SQ * MEAN_SQ))
 * Workers m < K; K <= MTDAO_STATS_MAX_REPLICAS. */
#define MTDAO_STATS_MAX_REPLICAS 16
#define MTDAO_STATS_STRIDE 36
#define MTDAO_STAT_MEAN_SQ 0
#define MTDAO_STAT_VARIANCE 1
#define MTDAO_STAT_OUTER_SQ 2
#define MTDAO_STAT_WORKER_SQ 4
#define MTDAO_STAT_WORKER_DOT 20
/* status codes */
enum {
  MTDAO_OK = 0,
  MTDAO_ERR_INVALID_ARG = -1, /* bad config value, NULL pointer, bad state id */
  MTDAO_ERR_ALIGN = -2,       /* a device pointer is not 16-byte aligned     */
  MTDAO_ERR_HIP = -3,         /* a HIP runtime call failed (message kept)     */
  MTDAO_ERR_RANGE = -4,       /* offset/count/replica out of range           */
  MTDAO_ERR_WORKSPACE = -5    /* workspace missing or smaller than required  */
};

/* Mask bits of mtdao_sync / mtdao_schedule: bit 0 = x, bit j (1..N) = u^j,
 * bit N+1 = v.  State ids of mtdao_read_state use the same numbering. */

/* Optimizer configuration: the Require block of Algorithms 1-3. */
typedef struct mtdao_config {
  int32_t form;             /* MTDAO_ADAM / MTDAO_ADOPT / MTDAO_SGDM               */
  int32_t replicas;         /* K >= 1: workers (the paper's M)                       */
  int32_t n_moments;        /* N, 1..MTDAO_MAX_N                                     */
  int32_t param_dtype;      /* MTDAO_F32 / MTDAO_BF16 storage of x                   */
  int32_t grad_dtype;       /* MTDAO_F32 / MTDAO_BF16 storage of the gradients       */
  int32_t adopt_order;      /* MTDAO_ADOPT_PREV (default) / MTDAO_ADOPT_CUR          */
  int32_t bias_correction;  /* Adam only: 1 = bias-correct u^j and v, 0 = none       */
  float beta1[MTDAO_MAX_N]; /* beta_{1,j} in [0,1)                                   */
  float omega[MTDAO_MAX_N]; /* omega_j in [0,1], sum <= 1 (+1e-6)                    */
  float beta2;              /* beta_2 in [0,1) (Adam, ADOPT)                         */
  float eps;                /* epsilon >= 0 (Adam, ADOPT)                            */
  float clip_rho;           /* rho > 0: global-norm clip (Adam, SGDM); <= 0: off     */
  int32_t period_x;         /* K_x >= 0 (0 = never)                                  */
  int32_t period_u[MTDAO_MAX_N]; /* K_j >= 0                                         */
  int32_t period_v;         /* K_v >= 0 (ignored by SGDM)                            */
  int64_t start_step;       /* updates already applied (0 fresh; s for a resume)     */
  int64_t numel;            /* P >= 0: elements per replica                          */
  int32_t n_tensors;        /* entries of tensor_numel (0: one tensor of P elements) */
  const int64_t* tensor_numel; /* host array, sums to P; copied by mtdao_init        */
  int32_t sync_order;       /* MTDAO_SYNC_AFTER_STEP (default) / _MOMENTA_IN_STEP    */
  int32_t outer_opt;        /* MTDAO_OUTER_AVERAGE (default) / MTDAO_OUTER_NESTEROV  */
  float outer_lr;           /* Nesterov: outer learning rate > 0                     */
  float outer_momentum;     /* Nesterov: outer momentum mu in [0,1)                  */
} mtdao_config;

/* Device state buffers (caller-owned, [K][P] each, see layout above). */
typedef struct mtdao_buffers {
  void* x;                  /* params                                                */
  float* u[MTDAO_MAX_N];    /* first moments u^1..u^N (entries >= N ignored)         */
  float* v;                 /* second moment (NULL for SGDM)                         */
  int32_t init_states;      /* 0: x row 0 is broadcast to all rows, u and v zeroed,  */
                            /*    x_outer = x row 0 (fp32), x_outer_mom = 0          */
                            /* 1: all given states are kept as they are (resume)     */
  float* x_outer;           /* Nesterov OuterOpt: outer parameters, fp32 [P]         */
  float* x_outer_mom;       /* Nesterov OuterOpt: outer momentum, fp32 [P]           */
} mtdao_buffers;

typedef struct mtdao_handle mtdao_handle;

/* Device workspace (bytes) that mtdao_init needs for this configuration:
 * with clip_rho > 0 (Adam, SGDM) the K clip factors (padded to 256 bytes)
 * and one fp64 partial sum of the gradient-norm reduction per 8192
 * elements of every row, about K * P / 1024 bytes; 0 otherwise.
 * Host-only; no GPU needed. */
int32_t mtdao_workspace_bytes(const mtdao_config* cfg, size_t* bytes);

/* Validate cfg and build a handle over the caller's buffers.  With
 * init_states == 0 it enqueues the broadcast of x_0 (row 0) to every
 * replica and zero-fills u and v (the initial u_{-1} = v_{-1} = 0), as the
 * Require block's single x_0 and the "initialize" line of Algorithms 1-3
 * state.  workspace: device buffer of at least mtdao_workspace_bytes
 * (may be NULL when that is 0), caller-owned, must outlive the handle.
 * The handle is library-owned: release it with mtdao_destroy. */
int32_t mtdao_init(const mtdao_config* cfg, const mtdao_buffers* bufs, void* workspace,
                   size_t workspace_bytes, void* hip_stream, mtdao_handle** out);

/* One local update of every replica (the body of Algorithms 1-3 for all
 * workers in parallel): s += 1, then for every replica m and element i the
 * form's update of u^j, v and x from grads[m][i].
 *   grads       device [K][P] in cfg.grad_dtype, read only
 *   lr          eta_t of this update
 *   adopt_clip  ADOPT's c_t for this update (<= 0: no clamp); ignored otherwise
 * With clip_rho > 0 it first reduces ||grads[m]||_2 per replica (one extra
 * read of the gradient) in a fixed order, so results are deterministic. */
int32_t mtdao_local_step(mtdao_handle* h, const void* grads, float lr, float adopt_clip,
                         void* hip_stream);

/* Replica averaging E_m[.] of the states selected by mask, after the last
 * local update (step s = mtdao_step_count).  mask = MTDAO_SYNC_AUTO applies
 * the schedule (states whose period divides s); any other value is taken as
 * the explicit set of states to average (e.g. the Bernoulli draws of the
 * probabilistic variant, Algorithm 4, made by the caller).  Every element of
 * every selected state becomes S^0 + (sum_{m>=1} (S^m - S^0)) / K, the
 * differences summed in fp64 and the result rounded once to the storage
 * type, and is written to all K rows, so averaging identical rows is an
 * exact no-op and a repeated call at the same s changes nothing (also under
 * the Nesterov OuterOpt, whose outer step runs once per s).
 * applied_mask (may be NULL) receives the set actually averaged. */
int32_t mtdao_sync(mtdao_handle* h, uint32_t mask, uint32_t* applied_mask, void* hip_stream);

/* mtdao_local_step followed by mtdao_sync(mask) in one pass over memory:
 * same arguments and same results, bit for bit (mask = MTDAO_SYNC_AUTO is
 * the schedule at the new step s).  When states are due, the K replica rows
 * of every element are updated and averaged within one workgroup and the
 * mean is written straight to all rows, so the separate averaging pass
 * (read and write of K rows per due state) is not needed.  applied_mask (may be NULL)
 * receives the set averaged.  Nothing is enqueued and the step counter does
 * not move when an argument is rejected. */
int32_t mtdao_step_sync(mtdao_handle* h, const void* grads, float lr, float adopt_clip, uint32_t mask,
                        uint32_t* applied_mask, void* hip_stream);

/* The update count kept in device memory, for capture into a HIP graph:
 * a replayed window of mtdao_step_sync_device calls forms the
 * step-dependent scalars of every update (eta_t, c_t, Adam's bias
 * corrections) from the device-side count instead of values frozen at
 * capture.  Caller-owned device memory, 16-byte aligned. */
typedef struct mtdao_device_step {
  int64_t s;                /* update count as of the last set or advance */
  int64_t reserved;
} mtdao_device_step;

/* Enqueue d->s = s; the host side records the handle's current step count
 * as the base of later offsets (typically s = mtdao_step_count).  No memset
 * is recorded. */
int32_t mtdao_device_step_set(mtdao_handle* h, mtdao_device_step* d, int64_t s, void* hip_stream);

/* mtdao_step_sync whose update number is taken on the device: the k-th
 * call since the last set or advance performs update s = d->s + k, with
 * eta_t = lr_table[s - 1] and c_t = clip_table[s - 1] (or off when
 * clip_table is NULL; the last entries for s > table_len) and the bias
 * corrections of Algorithm 1 formed from this s by the kernels.  The
 * tables are caller-owned device fp32 arrays; the kernels read them (and
 * d) as constants, so they must not be written while a launch of this
 * call runs (writes enqueued on the same stream before or after are
 * ordered with it).  Results equal
 * mtdao_step_sync's with the same eta_t and c_t, bit for bit (the scalars
 * are formed by the same code on host and device).  k, the mask
 * (MTDAO_SYNC_AUTO: the schedule at the handle's step count + 1) and the
 * launch configuration are fixed at call time: a captured window replays
 * the masks of the captured steps, so it equals eager calls when it spans
 * a whole number of every period.  The handle's host step count advances
 * per call as in mtdao_step_sync.  ADOPT's first update (previous-v order,
 * s = 1) is rejected: it sets v only, through mtdao_local_step or
 * mtdao_step_sync. */
int32_t mtdao_step_sync_device(mtdao_handle* h, const void* grads, mtdao_device_step* d, const float* lr_table,
                               const float* clip_table, int64_t table_len, uint32_t mask, uint32_t* applied_mask,
                               void* hip_stream);

/* Enqueue d->s += n, n = the mtdao_step_sync_device calls since the last
 * set or advance (fixed at call time, so a window captured with its
 * advance moves d->s on by the window at every replay); nothing when
 * n = 0. */
int32_t mtdao_device_step_advance(mtdao_handle* h, mtdao_device_step* d, void* hip_stream);

/* Device scratch (bytes) that mtdao_sync_stats needs for this
 * configuration: the 3 + 2K fp64 sums of every workgroup of the
 * diagnostics pass (one workgroup per 1024 fp32 or 2048 bf16 elements of a
 * row) for up to N + 2 states, about (N + 2) (3 + 2K) P / 128 bytes, plus
 * their chunk sums and the finalized rows.  Host-only. */
int32_t mtdao_stats_scratch_bytes(const mtdao_config* cfg, size_t* bytes);

/* mtdao_sync(mask) that also returns the averaging diagnostics of every
 * averaged state, computed in the same pass from the values before they are
 * averaged (the averaged values are bit-identical to mtdao_sync's).
 *   scratch     device buffer of mtdao_stats_scratch_bytes, 256-byte aligned,
 *               caller-owned (contents are scratch between calls)
 *   host_stats  caller-owned host array of (MTDAO_MAX_N + 2) *
 *               MTDAO_STATS_STRIDE doubles, indexed [state id][stat]; the
 *               rows of states not averaged are NaN
 * Needs K <= MTDAO_STATS_MAX_REPLICAS.  Waits for the stream. */
int32_t mtdao_sync_stats(mtdao_handle* h, uint32_t mask, uint32_t* applied_mask, void* scratch, size_t scratch_bytes,
                         double* host_stats, void* hip_stream);

/* mtdao_sync_stats without a caller scratch buffer, for callers that
 * cannot allocate device memory (serving loops and harnesses that forbid
 * allocation).  The partial sums live in a static device array of
 * MTDAO_STATIC_SCRATCH_BYTES that every GPU the library runs on holds until
 * the process ends, shared by all calls on that GPU: calls that overlap on
 * one GPU (other streams, other threads, other handles) race and must be
 * serialised by the caller.  Every scratch word a call reads is written
 * earlier in the same call, so nothing is cleared between calls.  Same
 * results as mtdao_sync_stats, bit for bit.  MTDAO_ERR_WORKSPACE (nothing
 * enqueued) when mtdao_stats_scratch_bytes exceeds the static size, about
 * K P (N + 2)(3 + 2K) / 128 bytes: e.g. up to 156M parameters at K = 4,
 * N = 3.  The handle's device must be current.  Calls no allocator; waits
 * for the stream. */
#define MTDAO_STATIC_SCRATCH_BYTES (64u << 20)
int32_t mtdao_sync_stats_static(mtdao_handle* h, uint32_t mask, uint32_t* applied_mask, double* host_stats,
                                void* hip_stream);

/* The schedule alone: states due after update s for this configuration.
 * Host-only; no GPU needed. */
int32_t mtdao_schedule(const mtdao_config* cfg, int64_t s, uint32_t* mask);

/* Copy count elements of one state row to host memory and wait for it:
 *   state    0 = x (cfg.param_dtype), 1..N = u^j, N+1 = v (fp32),
 *            MTDAO_STATE_X_OUTER / MTDAO_STATE_OUTER_MOM (fp32, Nesterov)
 *   replica  0..K-1 (0 for the outer states);  offset, count within [0, P]
 *   host_dst caller-owned, count * element-size bytes
 * Enqueued on hip_stream after earlier work; returns when the copy is done. */
int32_t mtdao_read_state(mtdao_handle* h, int32_t state, int32_t replica, int64_t offset,
                         int64_t count, void* host_dst, void* hip_stream);

/* Number of local updates applied so far (start_step + calls). -1 for NULL. */
int64_t mtdao_step_count(const mtdao_handle* h);

/* Message of the last failing call on h; with h == NULL, of the last
 * failing call that had no handle (init, workspace_bytes, schedule) on this
 * thread.  Never NULL; "" when there was no error. */
const char* mtdao_last_error(const mtdao_handle* h);

/* Release the handle (never the caller's buffers).  NULL is a no-op. */
void mtdao_destroy(mtdao_handle* h);

#ifdef __cplusplus
}
#endif

#endif /* MTDAO_H */
