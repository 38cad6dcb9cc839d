"""Brute-force twin of the outer step for tiny inputs (pins the oracle).

Pure Python floats and math.fsum, following the Sync() procedure of the
paper's appendix (Algorithm 2) in its own literal form, independently of
oracle/edit_oracle.c:

  * an anomalous worker's norm is *set to infinity* and the EMA update is
    skipped for infinite norms (Sec. 3.2);
  * gamma = sum_k exp(-G_k) and the rollback test is literally gamma == 0;
  * w_j = exp(-G_j) / gamma without any shift (Eq. 2);
  * the z-score is a division, z = (G - mu) / sigma > delta; for sigma = 0
    the reading "flag iff G > mu" is used (the limit of the division);
  * sums are correctly rounded (math.fsum), not sequential.

Replica values are taken as Python floats; bf16 rounding of the write-back
uses torch's own float->bfloat16 conversion.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np
import torch

AE, WA, GC = 1, 2, 4


def _f32(x: float) -> float:
    return float(np.float32(x))


def _bf16(x: float) -> float:
    return float(torch.tensor([x], dtype=torch.float32).to(torch.bfloat16).to(torch.float32)[0])


def brute_sync(theta: Sequence[float], mom: Sequence[float], reps: Sequence[Sequence[float]],
               mu: Sequence[float], sigma: Sequence[float], round_: int, cfg: dict,
               bf16: bool = False) -> Tuple[List[float], List[float], List[List[float]],
                                            List[float], List[float], dict]:
    """One outer step; returns (theta', mom', reps', mu', sigma', record)."""
    K, n = len(reps), len(theta)
    flags = cfg.get("flags", AE | WA | GC)
    mu, sigma = list(mu), list(sigma)

    delta = [[reps[j][i] - theta[i] for i in range(n)] for j in range(K)]
    G = [math.sqrt(math.fsum(d * d for d in delta[j])) for j in range(K)]
    raw_G = list(G)

    anomalous = [False] * K
    for j in range(K):
        if not math.isfinite(G[j]):
            anomalous[j] = True
        elif flags & AE and round_ >= cfg["warmup_rounds"]:
            if sigma[j] > 0:
                z = (G[j] - mu[j]) / sigma[j]
                anomalous[j] = z > cfg["z_threshold"]
            else:
                anomalous[j] = G[j] > mu[j]
        if anomalous[j]:
            G[j] = math.inf

    if flags & AE:
        a = cfg["ema_alpha"]
        for j in range(K):
            if math.isinf(G[j]):
                continue  # the EMA update is skipped for an infinite norm
            mu[j] = a * G[j] + (1 - a) * mu[j]
            sigma[j] = math.sqrt((1 - a) * sigma[j] ** 2 + a * (G[j] - mu[j]) ** 2)

    gamma = math.fsum(math.exp(-g) for g in G)
    rec = {"norm": raw_G, "anomalous": anomalous}
    if gamma == 0.0:
        new_reps = [[(_bf16(t) if bf16 else t) for t in theta] for _ in range(K)]
        rec.update(weight=[0.0] * K, rolled_back=True, synced_norm=0.0, clip_coef=0.0)
        return list(theta), list(mom), new_reps, mu, sigma, rec

    if flags & WA:
        w = [math.exp(-g) / gamma for g in G]
    else:
        m = sum(1 for g in G if not math.isinf(g))
        w = [0.0 if math.isinf(g) else 1.0 / m for g in G]
    dbar = [math.fsum(w[j] * delta[j][i] for j in range(K) if w[j] != 0.0) for i in range(n)]
    gbar = math.sqrt(math.fsum(x * x for x in dbar))
    beta = min(cfg["clip_threshold"] / (gbar + cfg["clip_eps"]), 1.0) if flags & GC else 1.0

    nu, rho = cfg["outer_lr"], cfg["momentum"]
    new_theta, new_mom = [], []
    for i in range(n):
        g = -(beta * dbar[i])
        b = rho * mom[i] + g
        new_mom.append(_f32(b))
        new_theta.append(_f32(theta[i] - nu * (g + rho * b)))
    new_reps = [[(_bf16(t) if bf16 else t) for t in new_theta] for _ in range(K)]
    rec.update(weight=w, rolled_back=False, synced_norm=gbar, clip_coef=beta)
    return new_theta, new_mom, new_reps, mu, sigma, rec
