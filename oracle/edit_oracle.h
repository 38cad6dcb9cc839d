/*
 * edit_oracle.h -- CPU oracle of EDiT's layer-wise outer synchronization step.
 *
 * TEST INFRASTRUCTURE ONLY.  This header and edit_oracle.c are the plain,
 * slow, fp64 statement of what the outer step computes (EDiT, Sec. 3.2
 * "Pseudo Gradient Penalty", Eq. 1-5, and the Sync() procedure of the
 * appendix, Algorithm 2).  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it; the product library never
 * does, and the two share no code, header, table or constant.
 *
 * Parity pins: every function below is pinned by the CPU tests
 * (closed forms, invariants, a brute-force transcription on tiny inputs,
 * torch's SGD-Nesterov and softmax).  The full composition of a step has no
 * printed reference value in the paper; beyond the pins it is "parity
 * unpinned" as a whole and is checked only through its parts.
 */
#ifndef EDIT_ORACLE_H
#define EDIT_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORACLE_MAX_K 64

/* Penalty components (the ablation switches of the paper's Sec. 4.5:
 * anomaly elimination, weighted averaging, gradient clip). */
#define ORACLE_AE 1u
#define ORACLE_WA 2u
#define ORACLE_GC 4u

typedef struct {
  double outer_lr;       /* nu: outer learning rate of OuterOpt            */
  double momentum;       /* rho: Nesterov momentum coefficient              */
  double clip_threshold; /* phi of Eq. 4                                    */
  double clip_eps;       /* epsilon of Eq. 4                                */
  double ema_alpha;      /* alpha of Eq. 1                                  */
  double z_threshold;    /* delta of the z-test                             */
  int64_t warmup_rounds; /* rounds during which no worker is flagged        */
  uint32_t flags;        /* ORACLE_AE | ORACLE_WA | ORACLE_GC               */
} oracle_cfg_t;

/* EMA statistics of one module (Eq. 1), one pair per worker, plus the
 * number of completed outer rounds of that module. */
typedef struct {
  double mu[ORACLE_MAX_K];
  double sigma[ORACLE_MAX_K];
  int64_t round;
} oracle_ema_t;

/* What one step decided, for comparison. */
typedef struct {
  double norm[ORACLE_MAX_K];     /* G_j = ||Delta_j||_2 (before masking)     */
  uint8_t anomalous[ORACLE_MAX_K];
  double weight[ORACLE_MAX_K];   /* w_j, 0 for masked workers               */
  double margin[ORACLE_MAX_K];   /* relative distance of the z-test from a
                                    tie; +inf where no test was taken       */
  double synced_norm;            /* Gbar = ||sum_j w_j Delta_j||_2          */
  double clip_coef;              /* beta of Eq. 4                           */
  int32_t rolled_back;           /* 1 when every worker was anomalous       */
  int32_t z_tested;              /* 1 when the z-test was applied           */
} oracle_record_t;

/*
 * One outer step of one module, in place.
 *   theta    [n] fp32   last synchronized parameters theta_t -> theta_{t+1}
 *   momentum [n] fp32   outer momentum buffer b -> b'
 *   replicas [K] pointers to [n] elements, fp32 (replica_is_bf16 = 0) or
 *            bf16 bit patterns (uint16_t, replica_is_bf16 = 1);
 *            in: theta_{t,tau} of each worker; out: theta_{t+1} cast to
 *            the replica type (every worker, masked ones included)
 *   ema      in/out EMA state and round counter of this module
 *   rec      out: the decision record (may be NULL)
 * Returns 0, or -1 for bad arguments (K outside 1..ORACLE_MAX_K, n < 0,
 * NULL pointers), or -2 when scratch memory cannot be allocated.
 */
int oracle_step(const oracle_cfg_t *cfg, int K, int64_t n, int replica_is_bf16,
                float *theta, float *momentum, void *const *replicas,
                oracle_ema_t *ema, oracle_record_t *rec);

/*
 * The decision of one step taken from a given Gram matrix of the K pseudo
 * gradients, Gram_jk = <Delta_j, Delta_k> (Sec. 3.2, Eq. 1-4), without the
 * elementwise update: G_j = sqrt(Gram_jj); the mask, EMA update and weights
 * exactly as in oracle_step; Gbar^2 = sum_jk w_j w_k Gram_jk over the
 * unflagged workers (taken as 0 if rounding makes it negative); beta.
 *   gram  [K(K+1)/2] fp64, the upper triangle row by row:
 *         (0,0), (0,1), ..., (0,K-1), (1,1), ..., (K-1,K-1)
 *   ema   in/out EMA state and round counter of the module
 *   rec   out: the decision record (may be NULL)
 * Returns 0, or -1 for bad arguments.
 */
int oracle_decide_gram(const oracle_cfg_t *cfg, int K, const double *gram, oracle_ema_t *ema,
                       oracle_record_t *rec);

/* Round-to-nearest-even of an fp32 value to bfloat16 (bit pattern). */
uint16_t oracle_f32_to_bf16(float x);

/* Exact widening of a bfloat16 bit pattern to fp32. */
float oracle_bf16_to_f32(uint16_t h);

#ifdef __cplusplus
}
#endif

#endif /* EDIT_ORACLE_H */
