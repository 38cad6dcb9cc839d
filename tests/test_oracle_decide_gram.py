"""Pins of the oracle's decision from a given Gram matrix (oracle_decide_gram).

That decision is the one of a step (Sec. 3.2, Eq. 1-4) with the norms and
Gbar read off the Gram matrix of the pseudo gradients: G_j^2 is its diagonal,
and ||sum_j w_j Delta_j||^2 = sum_jk w_j w_k Gram_jk by bilinearity.  The pins
compare it with the full step on the same inputs, whose Gbar comes from the
materialised weighted average instead (the Gram matrix here is a numpy
matrix product of the pseudo gradients), and with closed forms.
"""
import numpy as np
import pytest
import torch

from oracle import AE, GC, WA, OracleConfig, OracleUnit, f32_to_bf16_bits
from oracle.oracle import bf16_bits_to_f32


def upper(gram):
    """Row-major upper triangle (0,0), (0,1), ..., (K-1,K-1)."""
    K = gram.shape[0]
    return np.concatenate([gram[j, j:] for j in range(K)])


def deltas(theta, reps, bf16):
    wide = [bf16_bits_to_f32(r) if bf16 else r for r in reps]
    return np.stack([w.astype(np.float64) - theta.astype(np.float64) for w in wide])


def case(seed, K, n, bf16, flagged):
    """theta and K replicas; workers in `flagged` are x6."""
    rng = np.random.default_rng(seed)
    theta = rng.normal(0, 0.02, n).astype(np.float32)
    scale = np.where(np.isin(np.arange(K), flagged), 6.0, rng.uniform(0.8, 1.2, K))
    reps = [(theta + scale[j] * rng.normal(0, 1e-3, n)).astype(np.float32) for j in range(K)]
    if bf16:
        reps = [f32_to_bf16_bits(r) for r in reps]
    return theta, reps


@pytest.mark.parametrize("flags", [0, AE, WA | GC, AE | WA | GC])
@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("K", [1, 2, 5, 8, 16])
def test_matches_the_full_step(K, bf16, flags):
    """Same inputs, same EMA state (post warm-up, so the z-test is taken and
    the x6 workers fail it): the same mask, norms, weights, EMA update, Gbar
    and beta as the step that materialises Delta_bar (Eq. 3)."""
    n = 300
    flagged = [j for j in (1, 4) if j < K - 1]
    theta, reps = case(1000 * K + flags + 7 * bf16, K, n, bf16, flagged)
    D = deltas(theta, reps, bf16)
    gram = D @ D.T
    cfg = OracleConfig(flags=flags, clip_threshold=0.002, warmup_rounds=3)
    typical = 1e-3 * np.sqrt(n)
    state = (np.full(K, typical), np.full(K, 0.2 * typical), 5)
    a, b = OracleUnit(K, cfg), OracleUnit(K, cfg)
    a.set_state(*state)
    b.set_state(*state)
    ra = a.step(theta.copy(), np.zeros(n, np.float32), [r.copy() for r in reps])
    rb = b.decide_gram(upper(gram))
    np.testing.assert_array_equal(ra["anomalous"], rb["anomalous"])
    if flags & AE:
        assert ra["anomalous"].sum() == len(flagged)
    for key in ("rolled_back", "z_tested", "round"):
        assert ra[key] == rb[key], key
    for key in ("norm", "weight", "mu", "sigma"):
        np.testing.assert_allclose(rb[key], ra[key], rtol=1e-12, atol=0, err_msg=key)
    np.testing.assert_allclose(rb["synced_norm"], ra["synced_norm"], rtol=1e-10)
    np.testing.assert_allclose(rb["clip_coef"], ra["clip_coef"], rtol=1e-10)
    if flags & GC:
        assert ra["clip_coef"] < 1.0  # the clip is active in these cases


def test_rollback_matches_the_full_step():
    """Every worker fails the z-test: rollback, EMA state kept, round advanced."""
    K, n = 4, 200
    theta, reps = case(5, K, n, False, list(range(K)))
    D = deltas(theta, reps, False)
    cfg = OracleConfig(warmup_rounds=0)
    typical = 1e-3 * np.sqrt(n)
    a, b = OracleUnit(K, cfg), OracleUnit(K, cfg)
    for u in (a, b):
        u.set_state(np.full(K, typical), np.full(K, 0.2 * typical), 2)
    ra = a.step(theta.copy(), np.zeros(n, np.float32), [r.copy() for r in reps])
    rb = b.decide_gram(upper(D @ D.T))
    assert ra["rolled_back"] == rb["rolled_back"] == 1
    np.testing.assert_array_equal(rb["mu"], np.full(K, typical))
    assert rb["round"] == ra["round"] == 3


def test_orthogonal_pseudo_gradients_closed_form():
    """A diagonal Gram matrix (mutually orthogonal Delta_j): Gbar^2 = sum_j
    w_j^2 G_j^2 with w the softmax of -G (Eq. 2, via torch.softmax) and
    beta = min(phi/(Gbar + eps), 1) (Eq. 4)."""
    G = np.array([0.5, 1.0, 1.5, 3.0])
    cfg = OracleConfig(flags=WA | GC, clip_threshold=0.6, clip_eps=1e-6)
    rec = OracleUnit(4, cfg).decide_gram(upper(np.diag(G ** 2)))
    w = torch.softmax(-torch.tensor(G, dtype=torch.float64), 0).numpy()
    gbar = np.sqrt(np.sum(w ** 2 * G ** 2))
    np.testing.assert_allclose(rec["norm"], G, rtol=1e-15)
    np.testing.assert_allclose(rec["weight"], w, rtol=1e-14)
    np.testing.assert_allclose(rec["synced_norm"], gbar, rtol=1e-14)
    np.testing.assert_allclose(rec["clip_coef"], min(0.6 / (gbar + 1e-6), 1.0), rtol=1e-14)


@pytest.mark.parametrize("c", [[1.0, -1.0], [2.0, 0.5, -1.0], [1.0, 1.0, 1.0, 1.0]])
def test_rank_one_closed_form(c):
    """Delta_j = c_j v: Gram_jk = c_j c_k |v|^2 and, with uniform weights,
    Gbar = |mean_j c_j| |v|; opposite pseudo gradients cancel to Gbar = 0,
    which the clip leaves alone (beta = 1)."""
    c = np.asarray(c)
    v2 = 7.0
    cfg = OracleConfig(flags=GC, clip_threshold=1.0)
    rec = OracleUnit(len(c), cfg).decide_gram(upper(np.outer(c, c) * v2))
    gbar = abs(c.mean()) * np.sqrt(v2)
    assert abs(rec["synced_norm"] - gbar) <= 1e-14 * max(1.0, gbar)
    np.testing.assert_allclose(rec["norm"], np.abs(c) * np.sqrt(v2), rtol=1e-15)
    np.testing.assert_allclose(rec["clip_coef"], min(1.0 / (gbar + cfg.clip_eps), 1.0), rtol=1e-14)


def test_squared_norm_rounded_below_zero_reads_as_zero():
    """A Gram matrix that rounding left slightly indefinite: the quadratic
    form is a squared norm, so a negative value is taken as 0 (Gbar = 0,
    beta = 1), not as a NaN."""
    g = [1.0, -(1.0 + 2.0 ** -52), 1.0]
    rec = OracleUnit(2, OracleConfig(flags=GC)).decide_gram(np.array(g))
    assert rec["synced_norm"] == 0.0 and rec["clip_coef"] == 1.0


def test_flagged_worker_with_nonfinite_entries_is_left_out():
    """Worker 2's pseudo gradient is non-finite (its Gram row is NaN): it is
    flagged even in the warm-up, and Gbar and beta are those of workers 0
    and 1 alone."""
    full = np.array([[4.0, 1.0, np.nan], [1.0, 9.0, np.nan], [np.nan, np.nan, np.nan]])
    cfg = OracleConfig(flags=AE | WA | GC, clip_threshold=0.5, warmup_rounds=10)
    rec = OracleUnit(3, cfg).decide_gram(upper(full))
    sub = OracleUnit(2, cfg).decide_gram(upper(full[:2, :2]))
    assert list(rec["anomalous"]) == [0, 0, 1]
    np.testing.assert_array_equal(rec["weight"][:2], sub["weight"])
    assert rec["weight"][2] == 0.0
    assert np.isfinite(rec["synced_norm"]) and rec["synced_norm"] == sub["synced_norm"]
    assert rec["clip_coef"] == sub["clip_coef"]


def test_rejects_a_wrong_length():
    with pytest.raises(ValueError):
        OracleUnit(3).decide_gram(np.zeros(5))
