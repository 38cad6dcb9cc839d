"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test names the passage it follows.  None of them re-types the oracle's
formulas: they use closed forms, invariants, library routines (torch's
SGD with Nesterov momentum, torch.softmax, torch's bfloat16 cast) and the
independent brute-force transcription in brute_sync.py.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import AE, GC, WA, OracleConfig, OracleUnit, f32_to_bf16_bits
from brute_sync import brute_sync

HERE = os.path.dirname(os.path.abspath(__file__))


def ulp32(x):
    return np.spacing(np.abs(np.asarray(x, dtype=np.float32))).astype(np.float64)


def assert_f32_within_ulps(a, b, ulps=1):
    a = np.asarray(a, dtype=np.float32).astype(np.float64)
    b = np.asarray(b, dtype=np.float32).astype(np.float64)
    tol = ulps * np.maximum(ulp32(a), ulp32(b))
    assert np.all(np.abs(a - b) <= tol), np.max(np.abs(a - b) - tol)


def make_inputs(rng, K, n, theta_std=0.02, delta_std=1e-3, scales=None):
    theta = rng.normal(0, theta_std, n).astype(np.float32)
    mom = np.zeros(n, dtype=np.float32)
    scales = np.ones(K) if scales is None else np.asarray(scales, dtype=np.float64)
    reps = [(theta.astype(np.float64) + scales[j] * rng.normal(0, delta_std, n)).astype(np.float32)
            for j in range(K)]
    return theta, mom, reps


def bf16_bits(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float32)).to(torch.bfloat16).view(torch.int16) \
        .numpy().view(np.uint16)


def bits_to_f32(h):
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------- constants


def test_paper_constants_are_the_defaults():
    """Sec. 3.2 (alpha, delta), Sec. 4.1 (phi), appendix A.2 (nu, rho on FineWeb-Edu)."""
    with open(os.path.join(HERE, "golden", "paper_hyperparameters.json")) as f:
        paper = json.load(f)
    cfg = OracleConfig()
    assert cfg.ema_alpha == paper["ema_alpha"]["value"]
    assert cfg.z_threshold == paper["z_threshold"]["value"]
    assert cfg.clip_threshold == paper["clip_threshold"]["value"]
    assert cfg.outer_lr == paper["fineweb_edu"]["outer_lr"]
    assert cfg.momentum == paper["fineweb_edu"]["outer_momentum"]


# ------------------------------------------------------- pseudo gradients


@pytest.mark.parametrize("bf16", [False, True])
def test_norm_closed_form(bf16):
    """Sec. 3.2: G_j = ||r_j - theta||_2.  With r_j = theta + c_j on every
    element (dyadic values, exact in fp32/bf16) G_j = |c_j| * sqrt(n) exactly."""
    n, K = 64, 4  # sqrt(64) = 8
    rng = np.random.default_rng(1)
    theta = (rng.integers(-64, 64, n) / 256.0).astype(np.float32)  # 8-bit dyadic: bf16-exact
    c = [0.0, 2.0 ** -6, -3 * 2.0 ** -7, 2.0 ** -3]
    reps = [(theta + np.float32(cj)).astype(np.float32) for cj in c]
    if bf16:
        reps = [bf16_bits(r) for r in reps]
        assert all(np.array_equal(bits_to_f32(r), (theta + np.float32(cj))) for r, cj in zip(reps, c))
    unit = OracleUnit(K, OracleConfig(warmup_rounds=100))
    rec = unit.step(theta.copy(), np.zeros(n, np.float32), [r.copy() for r in reps])
    assert list(rec["norm"]) == [abs(cj) * 8.0 for cj in c]


def test_identical_replicas_zero_update():
    """Eq. 2-5: identical replicas give Delta = 0, Gbar = 0, so with b = 0
    the parameters do not move (and every weight is 1/K)."""
    rng = np.random.default_rng(2)
    n, K = 1000, 5
    theta = rng.normal(0, 0.02, n).astype(np.float32)
    reps = [theta.copy() for _ in range(K)]
    th, b = theta.copy(), np.zeros(n, np.float32)
    rec = OracleUnit(K).step(th, b, reps)
    assert np.array_equal(th, theta) and not b.any()
    assert all(np.array_equal(r, theta) for r in reps)
    assert np.all(rec["norm"] == 0) and rec["synced_norm"] == 0 and rec["clip_coef"] == 1.0
    assert np.all(rec["weight"] == 1.0 / K)


def test_identical_replicas_with_momentum_moves_by_rho2_b():
    """With Delta_hat = 0 the Nesterov step still applies the old momentum:
    b' = rho*b and theta' = theta - nu*rho*b' (nu = rho = 0.5: dyadic, exact)."""
    n, K = 256, 3
    rng = np.random.default_rng(3)
    theta = (rng.integers(-1000, 1000, n) / 1024.0).astype(np.float32)
    b = (rng.integers(-1000, 1000, n) / 1024.0).astype(np.float32)
    reps = [theta.copy() for _ in range(K)]
    th, bb = theta.copy(), b.copy()
    OracleUnit(K, OracleConfig(outer_lr=0.5, momentum=0.5)).step(th, bb, reps)
    assert np.array_equal(bb, b * np.float32(0.5))
    # theta - nu*rho*(rho*b) = theta - 0.125*b
    assert np.array_equal(th, (theta.astype(np.float64) - 0.125 * b.astype(np.float64)).astype(np.float32))


def test_uniform_mean_invariant():
    """Eq. 2-3: equal norms give w_j = 1/K, so Delta_bar is the plain mean;
    with b = 0, nu = 1, rho = 0 and no clipping theta' = mean_j r_j."""
    rng = np.random.default_rng(4)
    n, K = 4096, 4
    theta = rng.normal(0, 0.02, n).astype(np.float32)
    d = (rng.integers(-512, 512, n) / 2.0 ** 19)  # dyadic, so theta + s*d is exact below
    theta = (np.round(theta * 2 ** 19) / 2 ** 19).astype(np.float32)
    reps = []
    for j in range(K):
        s = rng.choice([-1.0, 1.0], n)  # same |Delta| pattern, so G_j are bitwise equal
        reps.append((theta.astype(np.float64) + s * d).astype(np.float32))
    th, b = theta.copy(), np.zeros(n, np.float32)
    cfg = OracleConfig(outer_lr=1.0, momentum=0.0, clip_threshold=1e30, warmup_rounds=100)
    rec = OracleUnit(K, cfg).step(th, b, [r.copy() for r in reps])
    assert np.all(rec["weight"] == 0.25)
    mean = np.mean(np.stack([r.astype(np.float64) for r in reps]), axis=0)
    assert_f32_within_ulps(th, mean.astype(np.float32), ulps=0)


def test_gram_identity_of_synced_norm():
    """Eq. 3-4: Gbar^2 = ||sum_j w_j Delta_j||^2 = sum_jk w_j w_k <Delta_j, Delta_k>."""
    rng = np.random.default_rng(5)
    n, K = 3000, 6
    theta, mom, reps = make_inputs(rng, K, n, scales=rng.uniform(0.5, 2, K))
    deltas = [r.astype(np.float64) - theta.astype(np.float64) for r in reps]
    rec = OracleUnit(K, OracleConfig(warmup_rounds=100)).step(theta, mom, reps)
    w = rec["weight"]
    gram = np.array([[np.dot(a, b) for b in deltas] for a in deltas])
    assert math.isclose(rec["synced_norm"], math.sqrt(w @ gram @ w), rel_tol=1e-12)


# ------------------------------------------------------------------- EMA


def test_ema_closed_form_constant_norm():
    """Eq. 1 from mu_0 = sigma_0 = 0 with a constant norm G has the closed form
    mu_k = G(1 - a^k), sigma_k = G a^((k+1)/2) sqrt(1 - a^k), a = 1 - alpha."""
    n, K = 64, 2
    d = np.full(n, 2.0 ** -5, dtype=np.float32)  # G = 2^-5 * 8 = 0.25 exactly
    alpha = 0.02
    unit = OracleUnit(K, OracleConfig(outer_lr=0.0, momentum=0.0, ema_alpha=alpha, warmup_rounds=10 ** 6))
    theta = np.zeros(n, np.float32)
    for k in range(1, 41):
        reps = [d.copy(), (-d).copy()]
        rec = unit.step(theta, np.zeros(n, np.float32), reps)
        G = 0.25
        a = 1 - alpha
        mu_k = G * (1 - a ** k)
        sig_k = G * a ** ((k + 1) / 2) * math.sqrt(1 - a ** k)
        assert rec["norm"][0] == G
        for j in range(K):
            assert math.isclose(rec["mu"][j], mu_k, rel_tol=1e-13)
            assert math.isclose(rec["sigma"][j], sig_k, rel_tol=1e-12)
    # the values quoted for ten rounds: 0.18293 G and 0.38272 G
    a = 0.98
    assert math.isclose(1 - a ** 10, 0.18293, abs_tol=1e-5)
    assert math.isclose(a ** 5.5 * math.sqrt(1 - a ** 10), 0.38272, abs_tol=1e-5)


def test_anomalous_worker_is_masked_after_warmup_only():
    """Sec. 3.2: after ten clean warm-up rounds a worker whose norm jumps x50 is
    flagged by the z-test and its EMA state is left untouched.  From a zero
    state the clean z-score is (1 - 0.18293)/0.38272 = 2.135 and the x50
    worker's is (50 - 0.18293)/0.38272 = 130.2 (closed form of Eq. 1)."""
    rng = np.random.default_rng(6)
    n, K, W = 16384, 4, 10
    unit = OracleUnit(K, OracleConfig(outer_lr=0.7, momentum=0.9, clip_threshold=1.0, warmup_rounds=W))
    theta = rng.normal(0, 0.02, n).astype(np.float32)
    mom = np.zeros(n, np.float32)
    for t in range(W + 1):
        scales = np.ones(K)
        if t == W:
            scales[3] = 50.0
        reps = [(theta.astype(np.float64) + scales[j] * rng.normal(0, 1e-3, n)).astype(np.float32)
                for j in range(K)]
        mu0, sig0 = unit.mu.copy(), unit.sigma.copy()
        rec = unit.step(theta, mom, reps)
        if t < W:
            assert not rec["z_tested"] and not rec["anomalous"].any()
        else:
            assert rec["z_tested"]
            assert list(rec["anomalous"]) == [0, 0, 0, 1]
            z = (rec["norm"] - mu0) / sig0
            assert np.all(np.abs(z[:3] - 2.135) < 0.05) and abs(z[3] - 130.2) < 3
            assert rec["mu"][3] == mu0[3] and rec["sigma"][3] == sig0[3]
            assert rec["weight"][3] == 0.0


def test_scaled_worker_during_warmup_not_flagged():
    """Sec. 3.2: no worker is flagged during the warm-up period."""
    rng = np.random.default_rng(7)
    n, K = 512, 3
    unit = OracleUnit(K, OracleConfig(warmup_rounds=5))
    for t in range(5):
        theta, mom, reps = make_inputs(rng, K, n, scales=[1, 1, 100.0])
        rec = unit.step(theta, mom, reps)
        assert not rec["anomalous"].any()
    assert unit.round == 5


def test_rollback_when_every_worker_is_anomalous():
    """Sec. 3.2 / Algorithm 2: if all workers are flagged, the parameters return
    to theta_t; momentum and EMA state are untouched (reading of the rollback)."""
    rng = np.random.default_rng(8)
    n, K = 2048, 4
    for bf16 in (False, True):
        unit = OracleUnit(K, OracleConfig(warmup_rounds=3))
        for t in range(3):
            theta, mom, reps = make_inputs(rng, K, n)
            unit.step(theta, mom, reps)
        theta, _, reps = make_inputs(rng, K, n, scales=[100.0] * K)
        mom = rng.normal(0, 1e-3, n).astype(np.float32)
        if bf16:
            reps = [bf16_bits(r) for r in reps]
        th, b = theta.copy(), mom.copy()
        mu0, sig0 = unit.mu.copy(), unit.sigma.copy()
        rec = unit.step(th, b, reps)
        assert rec["rolled_back"] == 1 and rec["anomalous"].all()
        assert np.array_equal(th, theta) and np.array_equal(b, mom)
        expect = bf16_bits(theta) if bf16 else theta
        assert all(np.array_equal(r, expect) for r in reps)
        assert np.array_equal(unit.mu, mu0) and np.array_equal(unit.sigma, sig0)
        assert unit.round == 4


def test_nonfinite_worker_always_masked():
    """A NaN in a replica makes G non-finite: masked even during the warm-up and
    with anomaly elimination off; the others still synchronize (reading)."""
    rng = np.random.default_rng(9)
    n, K = 300, 3
    for flags in (AE | WA | GC, WA | GC, 0):
        theta, mom, reps = make_inputs(rng, K, n)
        reps[1][17] = np.nan
        rec = OracleUnit(K, OracleConfig(flags=flags)).step(theta, mom, reps)
        assert list(rec["anomalous"]) == [0, 1, 0]
        assert rec["weight"][1] == 0.0 and np.all(np.isfinite(theta)) and np.all(np.isfinite(mom))


# --------------------------------------------------------------- weights


def test_weights_two_workers_closed_form():
    """Eq. 2 with two workers: w_1 = 1 / (1 + exp(G_1 - G_2))."""
    rng = np.random.default_rng(10)
    n = 1024
    theta, mom, reps = make_inputs(rng, 2, n, delta_std=0.02, scales=[1.0, 1.7])
    rec = OracleUnit(2, OracleConfig(warmup_rounds=100)).step(theta, mom, reps)
    G = rec["norm"]
    assert math.isclose(rec["weight"][0], 1.0 / (1.0 + math.exp(G[0] - G[1])), rel_tol=1e-14)
    assert math.isclose(rec["weight"][1], 1.0 / (1.0 + math.exp(G[1] - G[0])), rel_tol=1e-14)


def test_weights_match_torch_softmax_over_unmasked():
    """Eq. 2 is a softmax of -G over the unmasked workers (masked: G = inf, w = 0)."""
    rng = np.random.default_rng(11)
    n, K, W = 2048, 6, 2
    unit = OracleUnit(K, OracleConfig(warmup_rounds=W))
    for t in range(W + 1):
        scales = rng.uniform(0.5, 2, K) * 40
        if t == W:
            scales[4] *= 60
        theta, mom, reps = make_inputs(rng, K, n, scales=scales)
        rec = unit.step(theta, mom, reps)
    assert rec["anomalous"][4] == 1
    G = torch.tensor(rec["norm"], dtype=torch.float64)
    G[torch.tensor(rec["anomalous"], dtype=torch.bool)] = math.inf
    ref = torch.softmax(-G, dim=0).numpy()
    np.testing.assert_allclose(rec["weight"], ref, rtol=1e-13, atol=0)


# ------------------------------------------------------------------ clip


def test_clip_bound_and_identity_below_threshold():
    """Eq. 4-5: ||Delta_hat|| = beta*Gbar <= phi, and beta = 1 when Gbar <= phi."""
    rng = np.random.default_rng(12)
    n, K = 5000, 4
    for phi in (1e-3, 5e-3, 1e3):
        theta = np.zeros(n, np.float32)
        _, _, reps = make_inputs(rng, K, n, theta_std=0.0)
        th, b = theta.copy(), np.zeros(n, np.float32)
        cfg = OracleConfig(outer_lr=1.0, momentum=0.0, clip_threshold=phi, warmup_rounds=100)
        rec = OracleUnit(K, cfg).step(th, b, reps)
        # theta_0 = 0, nu = 1, rho = 0  =>  theta_1 = Delta_hat (rounded to fp32)
        step_norm = float(np.linalg.norm(th.astype(np.float64)))
        if rec["synced_norm"] > phi:
            assert rec["clip_coef"] < 1.0
            assert step_norm <= phi * (1 + 1e-6)
            # ||beta * Delta_bar|| = phi * Gbar / (Gbar + eps)
            g = rec["synced_norm"]
            assert math.isclose(step_norm, phi * g / (g + 1e-6), rel_tol=1e-6)
        else:
            assert rec["clip_coef"] == 1.0
            assert math.isclose(step_norm, rec["synced_norm"], rel_tol=1e-6)


# ------------------------------------------------------------- Nesterov


@pytest.mark.parametrize("lr,rho", [(0.8, 0.85), (1.0, 0.8), (0.7, 0.9)])
def test_diloco_special_case_is_torch_sgd_nesterov(lr, rho):
    """'w/o ALL' (Sec. 4.5) is DiLoCo: OuterOpt = SGD with Nesterov momentum on the
    outer gradient theta_t - mean_j r_j (Sec. 4.1).  torch.optim.SGD(nesterov=True)
    in fp64, with theta and b rounded to fp32 after every round, must agree."""
    rng = np.random.default_rng(13)
    n, K = 4000, 4
    theta = rng.normal(0, 0.02, n).astype(np.float32)
    mom = np.zeros(n, np.float32)
    unit = OracleUnit(K, OracleConfig(outer_lr=lr, momentum=rho, flags=0))
    p = torch.nn.Parameter(torch.from_numpy(theta.astype(np.float64)))
    opt = torch.optim.SGD([p], lr=lr, momentum=rho, nesterov=True)
    for t in range(5):
        reps = [(theta.astype(np.float64) + rng.normal(0, 1e-3, n)).astype(np.float32) for _ in range(K)]
        mean = np.mean(np.stack([r.astype(np.float64) for r in reps]), axis=0)
        p.grad = torch.from_numpy(theta.astype(np.float64) - mean)
        opt.step()
        with torch.no_grad():
            p.copy_(p.float().double())
            buf = opt.state[p]["momentum_buffer"]
            buf.copy_(buf.float().double())
        unit.step(theta, mom, reps)
        assert_f32_within_ulps(theta, p.detach().numpy().astype(np.float32), ulps=1)
        # torch keeps the buffer as the *gradient* momentum; the oracle's b holds the same.
        assert_f32_within_ulps(mom, buf.numpy().astype(np.float32), ulps=1)


def test_first_nesterov_step_closed_form():
    """From b = 0: b_1 = -Delta_hat and theta_1 = theta_0 + nu(1 + rho) Delta_hat."""
    rng = np.random.default_rng(14)
    n, K = 1000, 3
    theta, mom, reps = make_inputs(rng, K, n)
    theta0 = theta.astype(np.float64)
    deltas = np.stack([r.astype(np.float64) - theta0 for r in reps])
    rec = OracleUnit(K, OracleConfig(outer_lr=0.8, momentum=0.85, warmup_rounds=100)).step(theta, mom, reps)
    dhat = rec["clip_coef"] * (rec["weight"] @ deltas)
    np.testing.assert_allclose(mom, (-dhat).astype(np.float32), rtol=2e-7, atol=1e-12)
    np.testing.assert_allclose(theta, (theta0 + 0.8 * 1.85 * dhat).astype(np.float32), rtol=2e-7, atol=1e-10)


# ------------------------------------------------------------ ablations


def test_ablation_switches():
    """Sec. 4.5: w/o WA gives uniform weights over the unmasked workers, w/o GC
    gives beta = 1, w/o AE flags nothing and keeps no EMA state."""
    rng = np.random.default_rng(15)
    n, K = 3000, 4
    theta, mom, reps = make_inputs(rng, K, n, delta_std=1.0, scales=[1, 2, 3, 100])
    rec = OracleUnit(K, OracleConfig(flags=AE | GC, warmup_rounds=0)).step(
        theta.copy(), mom.copy(), [r.copy() for r in reps])
    # no EMA history: sigma = mu = 0, so every worker with G > 0 is flagged -> rollback
    assert rec["rolled_back"] == 1
    rec = OracleUnit(K, OracleConfig(flags=GC)).step(theta.copy(), mom.copy(), [r.copy() for r in reps])
    assert not rec["anomalous"].any() and np.all(rec["weight"] == 0.25)
    rec_ae = OracleUnit(K, OracleConfig(flags=WA)).step(theta.copy(), mom.copy(), [r.copy() for r in reps])
    assert rec_ae["clip_coef"] == 1.0 and rec_ae["synced_norm"] > 10.0
    unit = OracleUnit(K, OracleConfig(flags=WA | GC))
    unit.step(theta.copy(), mom.copy(), [r.copy() for r in reps])
    assert np.all(unit.mu == 0) and np.all(unit.sigma == 0)


# ------------------------------------------------------------------ bf16


def test_bf16_rounding_matches_torch_cast():
    """The write-back to bf16 replicas is round-to-nearest-even; torch's cast is the
    reference (ties, subnormals, overflow, inf and nan included)."""
    rng = np.random.default_rng(16)
    vals = list(rng.normal(0, 1, 2000).astype(np.float32))
    base = rng.integers(0, 2 ** 16, 200).astype(np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)                 # exact midpoints
    near = (base | 0x7FFF).view(np.float32)
    vals += list(ties) + list(near)
    vals += [np.float32(x) for x in (0.0, -0.0, 1e-40, -3e-39, 3.3895314e38, 3.4028235e38,
                                     -3.4028235e38, np.inf, -np.inf)]
    vals = np.array([v for v in vals if np.isfinite(v) or np.isinf(v)], dtype=np.float32)
    ours = f32_to_bf16_bits(vals)
    ref = bf16_bits(vals)
    assert np.array_equal(ours, ref)
    nan_bits = f32_to_bf16_bits(np.array([np.nan], np.float32))
    assert (int(nan_bits[0]) & 0x7F80) == 0x7F80 and (int(nan_bits[0]) & 0x7F) != 0


# --------------------------------------------------- brute-force agreement


def _run_both(rng, K, n, rounds, flags, bf16, W=2):
    cfg = dict(outer_lr=0.8, momentum=0.85, clip_threshold=0.02, clip_eps=1e-6, ema_alpha=0.02,
               z_threshold=3.0, warmup_rounds=W, flags=flags)
    unit = OracleUnit(K, OracleConfig(**cfg))
    theta = rng.normal(0, 0.02, n).astype(np.float32)
    mom = np.zeros(n, np.float32)
    b_theta, b_mom = [float(x) for x in theta], [0.0] * n
    mu, sigma = [0.0] * K, [0.0] * K
    for t in range(rounds):
        scales = rng.uniform(0.5, 2, K)
        if t >= W and rng.random() < 0.5:
            scales[rng.integers(K)] *= 50
        noise = [rng.normal(0, 1e-3, n) * scales[j] for j in range(K)]
        reps32 = [(theta.astype(np.float64) + noise[j]).astype(np.float32) for j in range(K)]
        reps = [bf16_bits(r) for r in reps32] if bf16 else reps32
        rep_vals = [[float(x) for x in (bits_to_f32(r) if bf16 else r)] for r in reps]
        b_theta = [float(x) for x in theta]
        b_mom = [float(x) for x in mom]
        bt, bm, br, mu, sigma, brec = brute_sync(b_theta, b_mom, rep_vals, mu, sigma, t, cfg, bf16=bf16)
        rec = unit.step(theta, mom, reps)
        assert list(rec["anomalous"]) == [int(a) for a in brec["anomalous"]]
        assert rec["rolled_back"] == int(brec["rolled_back"])
        np.testing.assert_allclose(rec["norm"], brec["norm"], rtol=1e-13)
        np.testing.assert_allclose(rec["weight"], brec["weight"], rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(rec["mu"], mu, rtol=1e-13)
        np.testing.assert_allclose(rec["sigma"], sigma, rtol=1e-12)
        if not brec["rolled_back"]:
            assert math.isclose(rec["synced_norm"], brec["synced_norm"], rel_tol=1e-12)
            assert math.isclose(rec["clip_coef"], brec["clip_coef"], rel_tol=1e-12)
        assert_f32_within_ulps(theta, np.array(bt, np.float32), ulps=1)
        assert_f32_within_ulps(mom, np.array(bm, np.float32), ulps=1)
        for j in range(K):
            got = bits_to_f32(reps[j]) if bf16 else reps[j]
            # replicas are cast(theta'); a 1-ulp fp32 difference may move a bf16 tie
            assert_f32_within_ulps(got, np.array(br[j], np.float32), ulps=1 if not bf16 else 2 ** 16)
            assert np.array_equal(got, bits_to_f32(bf16_bits(theta)) if bf16 else theta)


@pytest.mark.parametrize("K", [1, 2, 3, 4])
@pytest.mark.parametrize("n", [1, 2, 3, 7])
@pytest.mark.parametrize("bf16", [False, True])
def test_brute_force_tiny(K, n, bf16):
    """Brute force on tiny K, n over several rounds, every switch combination."""
    rng = np.random.default_rng(1000 * K + 10 * n + bf16)
    for flags in range(8):
        _run_both(rng, K, n, rounds=5, flags=flags, bf16=bf16)


def test_brute_force_medium():
    rng = np.random.default_rng(77)
    _run_both(rng, 5, 257, rounds=8, flags=AE | WA | GC, bf16=True, W=3)
    _run_both(rng, 8, 129, rounds=8, flags=AE | WA | GC, bf16=False, W=3)


def test_literal_vs_stable_weights_only_differ_on_underflow():
    """Algorithm 2 tests gamma == 0 literally.  With norms near 800 every exp(-G)
    underflows in fp64, so the literal procedure rolls back while the shifted
    softmax (the oracle's reading) still averages; below that they agree."""
    rng = np.random.default_rng(17)
    n, K = 64, 3
    theta = np.zeros(n, np.float32)
    cfg = dict(outer_lr=0.8, momentum=0.85, clip_threshold=10.0, clip_eps=1e-6, ema_alpha=0.02,
               z_threshold=3.0, warmup_rounds=100, flags=AE | WA | GC)
    for G_target, diverge in ((600.0, False), (800.0, True)):
        reps = [np.full(n, G_target / 8.0 * (1 + 0.01 * j), np.float32) for j in range(K)]
        vals = [[float(x) for x in r] for r in reps]
        *_, brec = brute_sync([0.0] * n, [0.0] * n, vals, [0.0] * K, [0.0] * K, 0, cfg)
        rec = OracleUnit(K, OracleConfig(**{k: v for k, v in cfg.items()})).step(
            theta.copy(), np.zeros(n, np.float32), reps)
        assert rec["rolled_back"] == 0
        assert brec["rolled_back"] == diverge
        if not diverge:
            np.testing.assert_allclose(rec["weight"], brec["weight"], rtol=1e-10)


def test_oracle_is_deterministic():
    rng = np.random.default_rng(18)
    n, K = 10000, 4
    theta, mom, reps = make_inputs(rng, K, n)
    outs = []
    for _ in range(2):
        th, b, rs = theta.copy(), mom.copy(), [r.copy() for r in reps]
        rec = OracleUnit(K).step(th, b, rs)
        outs.append((th, b, rs, rec["norm"]))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    assert np.array_equal(outs[0][3], outs[1][3])
