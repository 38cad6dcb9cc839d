/*
 * edit_outer.h -- C ABI of the EDiT layer-wise outer synchronization step
 * on one AMD Instinct MI355X (gfx950).
 *
 * The operation (EDiT, arXiv 2412.07210, Sec. 3.2 "Pseudo Gradient Penalty",
 * Eq. 1-5, and the Sync() procedure of the appendix, Algorithm 2):
 * K workers each hold a replica r_j of one module's parameters after their
 * local steps; theta is the module's last synchronized value.  One call
 *   1. forms the pseudo gradients Delta_j = r_j - theta and their norms
 *      G_j = ||Delta_j||_2 over the whole module,
 *   2. flags anomalous workers by an EMA z-test on G_j (Eq. 1; no flags
 *      during a warm-up of `ema_warmup_rounds` rounds) and updates the EMA
 *      mean/std of the unflagged workers,
 *   3. rolls every replica back to theta when all workers are flagged,
 *   4. otherwise weights the unflagged workers by a softmax of -G_j (Eq. 2),
 *      averages Delta_bar = sum_j w_j Delta_j (Eq. 3), clips it by
 *      beta = min(phi / (||Delta_bar|| + eps), 1) (Eq. 4-5),
 *   5. applies the outer optimizer, SGD with Nesterov momentum on the outer
 *      gradient g = -beta*Delta_bar (Sec. 4.1):
 *        b' = rho*b + g;   theta' = theta - nu*(g + rho*b'),
 *   6. writes theta' back to every replica (all K, flagged ones included).
 *
 * Precision: theta and the momentum b are stored in fp32; replicas in fp32
 * or bf16 (round-to-nearest-even of the fp32 theta').  All arithmetic from
 * the pseudo gradients on is fp64 (norms, Gram matrix, EMA state, weights,
 * clip factor and the elementwise update), rounded once when stored.
 *
 * All pointers to tensor data are DEVICE pointers on the device that was
 * current when the handle was created (except theta and momentum of
 * edit_outer_step_round_host, which are pinned HOST memory); the caller owns
 * them.  The library
 * owns the handle, the EMA state, its scratch memory and its events.
 * Every function returns an edit_status_t; nothing is thrown across the ABI.
 * On failure, edit_outer_last_error() returns a message for the calling
 * thread.  A handle is used from one host thread at a time (calls on
 * different handles may come from different threads).
 */
#ifndef EDIT_OUTER_H
#define EDIT_OUTER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Largest number of workers per sync group (the K of Sec. 3.1's model sync
 * group; the paper fixes no upper bound).  Kernels are specialised for every
 * K in 1..EDIT_MAX_K: the Gram pass keeps the K(K+1)/2 pairwise sums in
 * fp64 vector registers up to K = 8 and uses the fp64 matrix cores above. */
#define EDIT_MAX_K 32

/* Penalty components; clearing all three gives the DiLoCo outer step
 * (the ablations of Sec. 4.5). */
#define EDIT_AE 1u /* anomaly elimination (EMA z-test, rollback)  */
#define EDIT_WA 2u /* norm-based weighted averaging (Eq. 2)        */
#define EDIT_GC 4u /* pseudo-gradient clip (Eq. 4-5)               */

/* One-pass mean step, allowed only with AE, WA and GC all clear (the
 * "w/o ALL" ablation of Sec. 4.5, i.e. the DiLoCo outer step): the weights
 * are then 1/K whatever the norms are, so the average, Nesterov and the
 * write-back run in a single pass over theta, b and the replicas (48 bytes
 * per element at K = 8, bf16, against 68 for the two-pass step).  The norms
 * G_j and ||Delta_bar|| are still computed on the way and reported by
 * edit_outer_state_get.  Unlike the two-pass step, a worker with a
 * non-finite norm is NOT left out (there is no norm before the average): its
 * NaN/Inf reaches theta and shows in its reported G_j.  The Gram entry
 * points (edit_outer_gram_layer / _apply_layer) are not available in this
 * mode. */
#define EDIT_ONE_PASS 8u

typedef struct edit_outer *edit_outer_t; /* opaque, library-owned */

/* Status of every call; nothing is thrown across the ABI. */
typedef enum {
  EDIT_OK = 0,
  EDIT_EINVAL = -1, /* bad argument: index, size, NULL, alignment, aliasing  */
  EDIT_ENOMEM = -2, /* host or device allocation failed                      */
  EDIT_EHIP = -3,   /* a HIP runtime call or a kernel launch failed           */
  EDIT_ESTATE = -4, /* not valid now (e.g. state_get before any step)         */
  EDIT_ENODEV = -5  /* the current device is not a gfx950 GPU                 */
} edit_status_t;

/* Element type of the K replicas (the paper states no precision; theta and
 * the momentum are always fp32). */
typedef enum { EDIT_F32 = 0, EDIT_BF16 = 1 } edit_dtype_t;

/* Hyper-parameters of the outer step (Sec. 3.2 and the training settings of
 * Sec. 4.1), the sync units and the replica type. */
typedef struct {
  int32_t num_workers;        /* K, 1..EDIT_MAX_K                              */
  int32_t num_layers;         /* L sync units (modules), >= 1                  */
  const int64_t *layer_numel; /* [L] elements per unit (>= 0); copied at init  */
  int32_t replica_dtype;      /* edit_dtype_t of the K replicas                */
  uint32_t flags;             /* EDIT_AE | EDIT_WA | EDIT_GC, or EDIT_ONE_PASS */
  double outer_lr;            /* nu  (paper: 0.8 or 1.0)                       */
  double momentum;            /* rho (paper: 0.85 or 0.8)                      */
  double clip_threshold;      /* phi of Eq. 4 (paper: 10)                      */
  double clip_eps;            /* eps of Eq. 4, > 0                             */
  double ema_alpha;           /* alpha of Eq. 1 (paper: 0.02), in (0, 1]       */
  double z_threshold;         /* delta of the z-test (paper: 3)                */
  int64_t ema_warmup_rounds;  /* rounds per unit with no anomaly flagging, at  */
                              /* least edit_outer_min_warmup(alpha, delta)      */
                              /* when EDIT_AE is set (see there)                */
} edit_outer_config_t;

/* Per-unit state and the decision of its most recent step (host memory):
 * the EMA mean and std of each worker's pseudo-gradient norm (Eq. 1, kept
 * per worker and module as Sec. 3.2 describes), the norms G_j, the anomaly
 * mask, the weights w_j of Eq. 2, ||Delta_bar|| and the clip factor beta of
 * Eq. 4. */
typedef struct {
  int64_t round;               /* completed outer rounds of this unit         */
  int32_t num_workers;         /* K                                           */
  int32_t rolled_back;         /* 1 if every worker was flagged               */
  int32_t z_tested;            /* 1 if the z-test was applied (after warm-up) */
  int32_t reserved;
  double ema_mean[EDIT_MAX_K]; /* mu_j after the last step                    */
  double ema_std[EDIT_MAX_K];  /* sigma_j after the last step                 */
  double norm[EDIT_MAX_K];     /* G_j of the last step                        */
  double weight[EDIT_MAX_K];   /* w_j of the last step (0 when flagged)       */
  uint8_t anomalous[EDIT_MAX_K];
  double synced_norm;          /* ||Delta_bar|| of the last step              */
  double clip_coef;            /* beta of the last step (0 on rollback)       */
} edit_layer_state_t;

/* Create a handle on the current device for L sync units, each holding the
 * state Sec. 3.2 keeps per module: the EMA mean and std of Eq. 1 for each of
 * the K workers, zero at the start (the paper gives no initial value), and a
 * round counter.  Validates cfg (K in 1..EDIT_MAX_K, L >= 1, numel >= 0,
 * dtype, 0 < alpha <= 1, eps > 0, and with EDIT_AE a warm-up of at least
 * edit_outer_min_warmup rounds), allocates the state, per-unit scratch and
 * events.  EDIT_EINVAL for a bad config, EDIT_ENODEV off gfx950,
 * EDIT_ENOMEM. */
edit_status_t edit_outer_init(const edit_outer_config_t *cfg, edit_outer_t *out);

/* The shortest EMA warm-up, in rounds, after which a worker whose norm G_j
 * is the same every round passes the z-test of Eq. 1 (G_j - mu_j > delta *
 * sigma_j flags it) when the EMA starts from zero: mu after k updates is
 * G (1 - (1-alpha)^k), so it lags G, and sigma is small.  With a shorter
 * warm-up every such worker is flagged at its first tested round, and since
 * a flagged worker's EMA state is not updated (Sec. 3.2), the unit stays
 * masked or rolled back from then on.  6 for the paper's alpha = 0.02 and
 * delta = 3.  -1 when no warm-up suffices (delta <= 0) or alpha is outside
 * (0, 1].  Host-only; no device needed. */
int64_t edit_outer_min_warmup(double alpha, double delta);

/* One outer step of unit `layer` (Sec. 3.2, Algorithm 2), enqueued on
 * `stream` (a hipStream_t; NULL = the default stream).  No host
 * synchronisation; the norm/Gram pass, the one-block decision kernel and the
 * update pass run in stream order.
 *   theta    [n] fp32, in: theta_t, out: theta_{t+1} (unchanged on rollback)
 *   momentum [n] fp32, in/out: outer momentum b (zero-initialised by caller)
 *   replicas host array of K device pointers, each [n] of replica_dtype;
 *            in: the workers' parameters, out: theta_{t+1} in that dtype
 * Device pointers must be 16-byte aligned and the K+2 ranges disjoint
 * (else EDIT_EINVAL).  Steps of one unit must be ordered by the caller
 * (same stream or events); different units may run concurrently on
 * different streams.  n = 0 is allowed (NULL pointers accepted). */
edit_status_t edit_outer_step_layer(edit_outer_t h, int32_t layer, float *theta,
                                    float *momentum, void *const *replicas, void *stream);

/* One outer round: `count` distinct units, stepped in the given (forward)
 * order on `stream` (the layer-wise synchronization of Sec. 3.1), with the
 * same results bit for bit as calling edit_outer_step_layer for each of them
 * in that order.  Up to K = 8 each unit's one-block decision runs inside
 * the next pass-1 launch (an extra block), and its update pass follows that
 * launch; two consecutive units (not the round's last) share one pass-1
 * launch, whose partial sums are those of their own launches.  Above K = 8
 * a unit's update pass follows its own pass 1 and decision.  A unit of at
 * most 256 16-byte vectors (2,048 bf16 or 1,024 fp32 elements) is stepped
 * whole by one block of a small launch that carries up to four such units.
 * Units that kernel timing (edit_outer_set_profiling) covers keep launches
 * of their own.
 *   layers   [count] unit indices, each at most once (else EDIT_EINVAL)
 *   theta    [count] device pointers, as in edit_outer_step_layer
 *   momentum [count] device pointers
 *   replicas [count * K] device pointers, unit i's K replicas at i*K
 * Arguments are checked for every unit before anything is enqueued. */
edit_status_t edit_outer_step_round(edit_outer_t h, int32_t count, const int32_t *layers,
                                    float *const *theta, float *const *momentum,
                                    void *const *replicas, void *stream);

/* One outer round, as edit_outer_step_round, with theta_t and the outer
 * momentum b kept in HOST memory: the memory-saving placement of the outer
 * optimizer state that the paper describes (Sec. 3.2), so that the device
 * holds only the K replicas plus a staging ring of three units' theta and b
 * (allocated on the first call and kept until edit_outer_destroy).  Per unit,
 * on two library-owned copy streams: theta and b are copied in while the
 * previous unit computes, the step runs on `stream` from the staging slot,
 * and theta' and b' are copied back while the next unit computes.  The
 * kernels are those of the resident step, so results are the same bit for
 * bit.  The host link bounds it: 8 bytes per element each way.
 *   theta_host    [count] host pointers to [n] fp32 theta_t -> theta_{t+1}
 *   momentum_host [count] host pointers to [n] fp32 b -> b'
 *                 both must be page-locked (hipHostMalloc), else EDIT_EINVAL
 *   replicas      [count * K] device pointers, as in edit_outer_step_round
 * Everything is enqueued behind `stream`'s earlier work, and `stream` waits
 * for the last copy back: after synchronising `stream` the host arrays hold
 * theta_{t+1} and b'.  The caller must not touch them before that.  Rounds on
 * one handle must be issued from one stream. */
edit_status_t edit_outer_step_round_host(edit_outer_t h, int32_t count, const int32_t *layers,
                                         float *const *theta_host, float *const *momentum_host,
                                         void *const *replicas, void *stream);

/* A module whose parameters are sharded over several devices (the model-shard
 * group of Sec. 3.1) still takes its penalty on norms of the WHOLE module
 * (Sec. 3.2): each shard contributes partial sums, which the shards add up
 * before deciding.  The two calls below split edit_outer_step_layer at that
 * point.  Each shard is a unit of its own handle (its own layer_numel); the
 * caller adds the shards' Gram vectors (e.g. an all-reduce) and hands the
 * same sum to every shard, whose decisions and EMA states then agree bit for
 * bit.  For an unsplit unit, gram_layer followed by apply_layer with that
 * Gram gives the same results bit for bit as edit_outer_step_layer.
 *
 * The Gram vector holds the K(K+1)/2 sums sum_i Delta_j[i] Delta_k[i] over
 * the unit's elements, Delta_j = replica_j - theta, for j <= k, row by row:
 * (0,0), (0,1), ..., (0,K-1), (1,1), ..., (K-1,K-1); fp64, device memory,
 * 8-byte aligned, owned by the caller.  Its diagonal holds the squared norms
 * G_j^2, and the norm of the weighted average of Eq. 3 follows from it as
 * sqrt(w^T Gram w).
 *
 * gram_layer: pass 1 of unit `layer` only, enqueued on `stream`; writes
 *   `gram` and changes no state.  theta and the replicas are only read.
 * apply_layer: the decision (anomaly test, EMA update, weights, clip) from
 *   `gram`, then the update pass, on `stream`; state and outputs as in
 *   edit_outer_step_layer.  theta and the replicas must be unchanged since
 *   the Gram was taken.
 * Checks as in edit_outer_step_layer (gram_layer needs no momentum), plus
 * `gram` non-NULL, 8-byte aligned and disjoint from the other buffers;
 * EDIT_EINVAL on a handle made with EDIT_ONE_PASS. */
edit_status_t edit_outer_gram_layer(edit_outer_t h, int32_t layer, const float *theta,
                                    void *const *replicas, double *gram, void *stream);
edit_status_t edit_outer_apply_layer(edit_outer_t h, int32_t layer, const double *gram,
                                     float *theta, float *momentum, void *const *replicas,
                                     void *stream);

/* Copy unit `layer`'s EMA state (Eq. 1: mu_j and sigma_j of every worker,
 * the per-module state of Sec. 3.2) and last decision (G_j, mask, w_j of
 * Eq. 2, ||Delta_bar||, beta of Eq. 4) to *out (host memory), after waiting
 * for that unit's last enqueued step.  EDIT_ESTATE if the unit never stepped
 * and no state was set. */
edit_status_t edit_outer_state_get(edit_outer_t h, int32_t layer, edit_layer_state_t *out);

/* Restore unit `layer`'s EMA state of Eq. 1 (ema_mean, ema_std and the
 * round counter that the warm-up of Sec. 3.2 counts; other fields ignored),
 * e.g. when resuming from a checkpoint.  EDIT_EINVAL for a non-finite mean,
 * a negative or non-finite std or a negative round.  Waits for that unit's
 * last enqueued step first. */
edit_status_t edit_outer_state_set(edit_outer_t h, int32_t layer, const edit_layer_state_t *in);

/* Release everything the handle owns: the per-unit state of Sec. 3.2, the
 * scratch memory and the events (waits for its pending work first). */
void edit_outer_destroy(edit_outer_t h);

/* A static string naming status s. */
const char *edit_outer_strerror(edit_status_t s);

/* Message of the last failure on the calling thread ("" if none). */
const char *edit_outer_last_error(void);

/* ---- a step that allocates nothing ------------------------------------ */

/* Bytes of the fixed device array edit_outer_step_layer_noalloc works in. */
#define EDIT_NOALLOC_SCRATCH_BYTES (1u << 20)

/* For callers that cannot allocate device memory when they step (code under
 * HIP graph capture, serving loops, harnesses that forbid hipMalloc): the
 * step of edit_outer_step_layer, with the same kernels and the same results
 * bit for bit, except that the per-block partial sums of its Gram pass live
 * in a fixed array of EDIT_NOALLOC_SCRATCH_BYTES that the library keeps on
 * each GPU for the life of the process (set up by edit_outer_init) instead
 * of the handle's scratch memory.  The call allocates nothing: no hipMalloc,
 * no hipFree, no event creation; kernel timing (edit_outer_set_profiling)
 * does not apply to it.  The handle (made earlier, outside any capture)
 * still holds the unit's EMA state and decision record.
 * Arguments, ownership and errors as in edit_outer_step_layer, plus
 * EDIT_EINVAL when the handle was made with EDIT_ONE_PASS, or when the
 * unit's partials exceed the array: K(K+1)/2 doubles per Gram-pass block,
 * whose count grows with the unit up to one block per CU above K = 8 (255
 * on MI355X), so only K = 32 units of more than 63,488 16-byte vectors
 * (507,904 bf16 or 253,952 fp32 elements) are refused there.
 * All calls on one GPU share that GPU's array, which keeps the last call's
 * partials (nothing in it needs clearing: a call writes every partial it
 * reads).  Calls on one GPU must therefore not overlap: order them on one
 * stream or with events, also across handles and host threads; overlapping
 * calls race.  The call enqueues three kernels and one event record and
 * makes no synchronising call, so it can be captured into a HIP graph and
 * replayed; after a replay, once the caller has synchronised,
 * edit_outer_state_get reports that replay's step. */
edit_status_t edit_outer_step_layer_noalloc(edit_outer_t h, int32_t layer, float *theta,
                                            float *momentum, void *const *replicas, void *stream);

/* ---- one worker of a sync group on its own GPU ------------------------- */

/* In EDiT a module's K replicas belong to the K workers of a model sync
 * group, one per GPU, and every worker runs Sync() (appendix, Algorithm 2)
 * on its own copy: its pseudo gradient Delta_i and norm G_i, its z-test
 * against its own EMA state (Eq. 1), an exchange of the K norms (the
 * "sync the pseudo gradient norms" step), the weights (Eq. 2), the sum
 * Delta_bar = sum_j w_j Delta_j over the group (Eq. 3), the clip (Eq. 4-5)
 * and OuterOpt.  A group handle is one worker's (rank's) share of that on
 * its GPU; the two exchanges between the calls are the caller's collectives
 * (for instance RCCL over xGMI), which this library does not make:
 *
 *   edit_group_norm      Delta_rank = replica - theta in fp64: G_rank, this
 *                        worker's z-test and EMA update, Delta_rank exported
 *                        to `delta` in fp32, and {G_rank, flag} to `norm_out`
 *   [caller] all-gather of every rank's norm_out, in rank order
 *   edit_group_weights   the group's decision from the gathered pairs (mask,
 *                        rollback, w_j; the same on every rank), w_rank to
 *                        `weight_out`, and `delta` cleared when this worker
 *                        is flagged (its Delta may be NaN; w_rank is then 0)
 *   [caller] all-reduce sum over the group of w_j * delta_j (e.g. a
 *            pre-multiplied sum with w_rank as this rank's factor) into dbar
 *   edit_group_apply     Gbar = ||dbar||, beta, Nesterov on theta and the
 *                        momentum, and this rank's replica set to theta'; on
 *                        a rollback the replica is set to theta only
 *
 * Each call is enqueued on `stream` and reads what the previous call wrote
 * through the caller's collectives on the same stream order.  The pseudo
 * gradient's norm is exact (fp64); the collective's payload is fp32, so
 * Delta_bar carries one fp32 rounding per term (relative 2^-24) against the
 * single-GPU step.
 *
 * cfg is validated as by edit_outer_init (num_workers = K, the group size;
 * EDIT_ONE_PASS is not accepted); 0 <= rank < K.  All tensor pointers are
 * device pointers on the handle's device, 16-byte aligned (the 2-double
 * norm_out / 2K-double gathered / 1-double weight_out: 8-byte aligned), with
 * n = layer_numel[layer] elements: theta, momentum, delta and dbar fp32,
 * replica of cfg->replica_dtype.  theta, momentum, replica and delta must not
 * overlap each other; dbar may be `delta` itself (an in-place all-reduce)
 * but must not overlap theta, momentum or the replica.  The EMA state of a
 * group handle is this worker's only: edit_group_state_get reports it at
 * index `rank` of ema_mean / ema_std (0 elsewhere), and the norms, mask and
 * weights of every worker from the last decision. */
typedef struct edit_group *edit_group_t; /* opaque, library-owned */

edit_status_t edit_group_init(const edit_outer_config_t *cfg, int32_t rank, edit_group_t *out);
edit_status_t edit_group_norm(edit_group_t h, int32_t layer, const float *theta, const void *replica,
                              float *delta, double *norm_out, void *stream);
edit_status_t edit_group_weights(edit_group_t h, int32_t layer, const double *gathered,
                                 double *weight_out, float *delta, void *stream);
edit_status_t edit_group_apply(edit_group_t h, int32_t layer, const float *dbar, float *theta,
                               float *momentum, void *replica, void *stream);
/* As edit_outer_state_get / _set, for this worker (see above); state_set
 * takes ema_mean[rank], ema_std[rank] and round.  Both wait for the unit's
 * last edit_group_apply; after a norm or weights call that no apply has
 * followed yet they synchronise the whole device instead. */
edit_status_t edit_group_state_get(edit_group_t h, int32_t layer, edit_layer_state_t *out);
edit_status_t edit_group_state_set(edit_group_t h, int32_t layer, const edit_layer_state_t *in);
void edit_group_destroy(edit_group_t h);

/* ---- measurement helpers (not part of the method) ---------------------- */

/* every > 0: steps of units whose index is a multiple of `every` record HIP
 * events around their two passes (each event costs a few microseconds of
 * stream time, so a benchmark samples a subset of units); 0 turns it off.
 * EDIT_EINVAL for every < 0. */
edit_status_t edit_outer_set_profiling(edit_outer_t h, int32_t every);

/* Durations in ms of the last profiled step of `layer`: ms[0] its norm/Gram
 * pass plus its decision kernel (in a round: its own norm/Gram launch, which
 * up to K = 8 also carries the decisions of the one or two units before it),
 * ms[1] its update pass.  With EDIT_ONE_PASS: ms[0] the fused pass, ms[1]
 * the record reduction when the unit was stepped alone (0 in a round, which
 * reduces all units in one launch at its end).  Waits for it. */
edit_status_t edit_outer_kernel_times(edit_outer_t h, int32_t layer, float ms[2]);

/* The memory traffic of unit `layer`'s update pass with no arithmetic: a
 * kernel with the update pass's grid, block order and 16-byte accesses reads
 * theta, the momentum and all K replicas and writes them back unchanged
 * (16 + 2K R bytes per element, the update pass's bytes when every worker
 * contributes), so its time is the floor this access pattern sets for that
 * pass.  Elements past the last whole 16-byte replica vector are not
 * touched.  Arguments and checks as in edit_outer_step_layer; the EMA state
 * and records are untouched. */
edit_status_t edit_outer_update_probe(edit_outer_t h, int32_t layer, float *theta, float *momentum,
                                      void *const *replicas, void *stream);

/* Plain device-to-device copy kernel of nbytes (a multiple of 16, 16-byte
 * aligned, non-overlapping pointers; one 16-byte vector per thread), used to
 * calibrate HBM traffic counters and as the bandwidth reference. */
edit_status_t edit_outer_copy_probe(void *dst, const void *src, int64_t nbytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* EDIT_OUTER_H */
