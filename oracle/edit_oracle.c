/*
 * edit_oracle.c -- CPU oracle of EDiT's layer-wise outer synchronization step.
 *
 * TEST INFRASTRUCTURE ONLY (see edit_oracle.h).  Plain loops in fp64, one
 * thread, no blocking, no fusion beyond what the equations state, in the
 * order of the paper's Sync() procedure (appendix, Algorithm 2):
 *
 *   pseudo gradients and their norms        Sec. 3.2, Algorithm 2
 *   anomaly elimination (EMA z-test)         Sec. 3.2, Eq. 1
 *   rollback when every worker is anomalous  Sec. 3.2, Algorithm 2
 *   weighted averaging                       Eq. 2, Eq. 3
 *   pseudo-gradient clip                     Eq. 4, Eq. 5
 *   OuterOpt = Nesterov momentum             Sec. 4.1 (after DiLoCo)
 *   write-back to every worker               Algorithm 2
 *
 * oracle_decide_gram takes the same decision from a given Gram matrix of the
 * pseudo gradients (norms from its diagonal, Gbar^2 = w^T Gram w).
 *
 * Readings taken where the paper is silent (each listed in the design notes):
 *   - OuterOpt consumes the outer gradient g = -Delta_hat, in the form of
 *     SGD with Nesterov momentum: b' = rho*b + g; theta' = theta - nu*(g + rho*b').
 *   - The z-test z > delta is evaluated as (G - mu) > delta*sigma, against the
 *     state before this round's update; the EMA state starts at zero.
 *   - A non-finite norm always counts as anomalous, even in the warm-up.
 *   - The softmax of Eq. 2 is evaluated after subtracting the smallest
 *     unmasked norm (identical to Eq. 2 unless every exp(-G) underflows).
 *   - A rollback leaves theta, the momentum and the EMA state unchanged and
 *     only resets the replicas; the round counter still advances.
 *   - A quadratic form w^T Gram w that rounding takes below zero is a squared
 *     norm and counts as 0.
 */
#include "edit_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ bf16 */

float oracle_bf16_to_f32(uint16_t h) {
  /* bfloat16 is the upper half of an fp32 word: widening is exact. */
  uint32_t bits = (uint32_t)h << 16;
  float x;
  memcpy(&x, &bits, sizeof x);
  return x;
}

/* Value of an fp32 bit pattern as a double; the pattern just past the
 * largest finite magnitude stands for 2^128 (the IEEE overflow point). */
static double pattern_value(uint32_t bits) {
  if ((bits & 0x7FFFFFFFu) == 0x7F800000u) {
    double big = ldexp(1.0, 128);
    return (bits & 0x80000000u) ? -big : big;
  }
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

uint16_t oracle_f32_to_bf16(float x) {
  /* Round to nearest, ties to even, by comparing distances to the two
   * bfloat16 neighbours of x (bfloat16 keeps 8 significand bits). */
  uint32_t bits;
  memcpy(&bits, &x, sizeof bits);
  if (isnan(x)) return (uint16_t)(((bits >> 16) & 0x8000u) | 0x7FC0u);
  if (isinf(x)) return (uint16_t)(bits >> 16);
  uint32_t toward_zero = bits & 0xFFFF0000u;
  if (toward_zero == bits) return (uint16_t)(bits >> 16);
  uint32_t away = toward_zero + 0x00010000u; /* one bf16 step further out */
  double d_toward = fabs((double)x - pattern_value(toward_zero));
  double d_away = fabs(pattern_value(away) - (double)x);
  if (d_toward < d_away) return (uint16_t)(toward_zero >> 16);
  if (d_away < d_toward) return (uint16_t)(away >> 16);
  return ((toward_zero >> 16) & 1u) ? (uint16_t)(away >> 16)
                                    : (uint16_t)(toward_zero >> 16);
}

/* ------------------------------------------------------ pseudo gradient */

/* Delta_j[i] = theta_{t,tau}^{(j)}[i] - theta_t[i]  (Sec. 3.2, Algorithm 2). */
static double pseudo_gradient(const void *replica, int is_bf16, const float *theta,
                              int64_t i) {
  double r = is_bf16 ? (double)oracle_bf16_to_f32(((const uint16_t *)replica)[i])
                     : (double)((const float *)replica)[i];
  return r - (double)theta[i];
}

/* G_j = ||Delta_j||_2 over the whole module (Sec. 3.2). */
static double pseudo_gradient_norm(const void *replica, int is_bf16,
                                   const float *theta, int64_t n) {
  double s = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    double d = pseudo_gradient(replica, is_bf16, theta, i);
    s += d * d;
  }
  return sqrt(s);
}

/* ------------------------------------------------- anomaly elimination */

/* IsAnomaly(G_j): z = (G - mu)/sigma > delta, with the state before this
 * round's update; not applied during the warm-up (Sec. 3.2). */
static int is_anomaly(double G, double mu, double sigma, double delta,
                      double *margin) {
  double lhs = G - mu;
  double rhs = delta * sigma;
  double scale = fmax(fmax(fabs(G), fabs(mu)), rhs);
  *margin = scale > 0.0 ? fabs(lhs - rhs) / scale : 0.0;
  return lhs > rhs;
}

/* Eq. 1: mu' = alpha*G + (1-alpha)*mu;
 *        sigma' = sqrt((1-alpha)*sigma^2 + alpha*(G - mu')^2). */
static void ema_update(double G, double alpha, double *mu, double *sigma) {
  double mu_new = alpha * G + (1.0 - alpha) * (*mu);
  double dev = G - mu_new;
  double sigma_new = sqrt((1.0 - alpha) * (*sigma) * (*sigma) + alpha * dev * dev);
  *mu = mu_new;
  *sigma = sigma_new;
}

/* ------------------------------------------------------------ the step */

/* Every worker takes the same value: theta_{t+1}[i] in the replica type. */
static void write_back_all(void *const *replicas, int K, int is_bf16, int64_t i, float value) {
  if (is_bf16) {
    uint16_t h = oracle_f32_to_bf16(value);
    for (int j = 0; j < K; ++j) ((uint16_t *)replicas[j])[i] = h;
  } else {
    for (int j = 0; j < K; ++j) ((float *)replicas[j])[i] = value;
  }
}

/* Eq. 4: beta = min(phi / (Gbar + eps), 1) with the clip on, else 1. */
static double clip_coefficient(const oracle_cfg_t *cfg, double gbar) {
  if (!(cfg->flags & ORACLE_GC)) return 1.0;
  return fmin(cfg->clip_threshold / (gbar + cfg->clip_eps), 1.0);
}

/* The decision from the norms G_j, shared by the step and by the decision
 * on a given Gram matrix: anomaly elimination (Sec. 3.2; a flagged worker's
 * norm counts as infinite, so it drops out of Eq. 2 and its EMA update is
 * skipped), the EMA update of Eq. 1, and the weights of Eq. 2 (1/|U| each
 * without weighted averaging).  Fills the record's norms, mask, margins and
 * weights; returns the number of unflagged workers (0: rollback). */
static int decide_weights(const oracle_cfg_t *cfg, int K, const double *G, oracle_ema_t *ema,
                          oracle_record_t *r, int *anomalous, double *w) {
  const int ae = (cfg->flags & ORACLE_AE) != 0;
  const int wa = (cfg->flags & ORACLE_WA) != 0;
  for (int j = 0; j < K; ++j) r->norm[j] = G[j];

  const int z_test = ae && ema->round >= cfg->warmup_rounds;
  r->z_tested = z_test;
  for (int j = 0; j < K; ++j) {
    r->margin[j] = INFINITY;
    anomalous[j] = !isfinite(G[j]);
    if (z_test && !anomalous[j])
      anomalous[j] = is_anomaly(G[j], ema->mu[j], ema->sigma[j], cfg->z_threshold,
                                &r->margin[j]);
    r->anomalous[j] = (uint8_t)anomalous[j];
  }
  if (ae)
    for (int j = 0; j < K; ++j)
      if (!anomalous[j]) ema_update(G[j], cfg->ema_alpha, &ema->mu[j], &ema->sigma[j]);

  int n_ok = 0;
  for (int j = 0; j < K; ++j) n_ok += !anomalous[j];
  if (n_ok == 0) return 0;

  if (wa) {
    double g0 = INFINITY;
    for (int j = 0; j < K; ++j)
      if (!anomalous[j] && G[j] < g0) g0 = G[j];
    double gamma = 0.0;
    for (int j = 0; j < K; ++j) {
      w[j] = anomalous[j] ? 0.0 : exp(-(G[j] - g0));
      gamma += w[j];
    }
    for (int j = 0; j < K; ++j) w[j] /= gamma;
  } else {
    for (int j = 0; j < K; ++j) w[j] = anomalous[j] ? 0.0 : 1.0 / (double)n_ok;
  }
  for (int j = 0; j < K; ++j) r->weight[j] = w[j];
  return n_ok;
}

int oracle_step(const oracle_cfg_t *cfg, int K, int64_t n, int replica_is_bf16,
                float *theta, float *momentum, void *const *replicas,
                oracle_ema_t *ema, oracle_record_t *rec) {
  if (!cfg || !ema || K < 1 || K > ORACLE_MAX_K || n < 0) return -1;
  if (n > 0 && (!theta || !momentum || !replicas)) return -1;
  for (int j = 0; j < K && n > 0; ++j)
    if (!replicas[j]) return -1;

  const int bf16 = replica_is_bf16 != 0;

  oracle_record_t r;
  memset(&r, 0, sizeof r);

  /* Pseudo gradient norms. */
  double G[ORACLE_MAX_K];
  for (int j = 0; j < K; ++j) G[j] = pseudo_gradient_norm(replicas[j], bf16, theta, n);

  /* Anomaly elimination, the EMA update and the weights of Eq. 2. */
  int anomalous[ORACLE_MAX_K];
  double w[ORACLE_MAX_K];
  const int n_ok = decide_weights(cfg, K, G, ema, &r, anomalous, w);

  if (n_ok == 0) {
    /* Rollback: every worker returns to the last synchronized theta_t. */
    for (int64_t i = 0; i < n; ++i) write_back_all(replicas, K, bf16, i, theta[i]);
    r.rolled_back = 1;
    ema->round += 1;
    if (rec) *rec = r;
    return 0;
  }

  /* Eq. 3: Delta_bar = sum_j w_j Delta_j, materialised. */
  double *dbar = NULL;
  if (n > 0) {
    dbar = (double *)malloc((size_t)n * sizeof(double));
    if (!dbar) return -2;
  }
  for (int64_t i = 0; i < n; ++i) {
    double s = 0.0;
    for (int j = 0; j < K; ++j)
      if (!anomalous[j]) s += w[j] * pseudo_gradient(replicas[j], bf16, theta, i);
    dbar[i] = s;
  }

  /* Eq. 4: Gbar = ||Delta_bar||_2, beta = min(phi / (Gbar + eps), 1). */
  double ss = 0.0;
  for (int64_t i = 0; i < n; ++i) ss += dbar[i] * dbar[i];
  const double gbar = sqrt(ss);
  const double beta = clip_coefficient(cfg, gbar);
  r.synced_norm = gbar;
  r.clip_coef = beta;

  /* Eq. 5 and OuterOpt (Nesterov momentum on the outer gradient -Delta_hat),
   * then every worker takes theta_{t+1}. */
  const double nu = cfg->outer_lr, rho = cfg->momentum;
  for (int64_t i = 0; i < n; ++i) {
    double delta_hat = beta * dbar[i];
    double g = -delta_hat;
    double b_new = rho * (double)momentum[i] + g;
    double th_new = (double)theta[i] - nu * (g + rho * b_new);
    theta[i] = (float)th_new;
    momentum[i] = (float)b_new;
    write_back_all(replicas, K, bf16, i, theta[i]);
  }
  free(dbar);

  ema->round += 1;
  if (rec) *rec = r;
  return 0;
}

/* ------------------------------------------------ decision from a Gram */

int oracle_decide_gram(const oracle_cfg_t *cfg, int K, const double *gram, oracle_ema_t *ema,
                       oracle_record_t *rec) {
  if (!cfg || !ema || !gram || K < 1 || K > ORACLE_MAX_K) return -1;

  /* Entry (j, k), j <= k, of the row-major upper triangle. */
#define GRAM_AT(j, k) gram[(j) * K - ((j) * ((j) - 1)) / 2 + ((k) - (j))]

  oracle_record_t r;
  memset(&r, 0, sizeof r);

  /* G_j = ||Delta_j||_2 = sqrt(<Delta_j, Delta_j>). */
  double G[ORACLE_MAX_K];
  for (int j = 0; j < K; ++j) G[j] = sqrt(GRAM_AT(j, j));

  int anomalous[ORACLE_MAX_K];
  double w[ORACLE_MAX_K];
  const int n_ok = decide_weights(cfg, K, G, ema, &r, anomalous, w);
  if (n_ok == 0) {
    r.rolled_back = 1;
    ema->round += 1;
    if (rec) *rec = r;
    return 0;
  }

  /* Eq. 3-4: ||sum_j w_j Delta_j||^2 = sum_j sum_k w_j w_k <Delta_j, Delta_k>
   * over the unflagged workers (a flagged worker's entries may be
   * non-finite and have weight 0).  The sum is a squared norm, so a value
   * that rounding took below zero counts as zero. */
  double q = 0.0;
  for (int j = 0; j < K; ++j) {
    if (anomalous[j]) continue;
    for (int k = 0; k < K; ++k) {
      if (anomalous[k]) continue;
      q += w[j] * w[k] * (j <= k ? GRAM_AT(j, k) : GRAM_AT(k, j));
    }
  }
#undef GRAM_AT
  const double gbar = sqrt(q > 0.0 ? q : 0.0);
  r.synced_norm = gbar;
  r.clip_coef = clip_coefficient(cfg, gbar);

  ema->round += 1;
  if (rec) *rec = r;
  return 0;
}
