"""Units past 2^31 elements: 64-bit indexing in every kernel.

One unit of 2^31 + 9 elements (theta alone is 8 GiB, so element indices and
byte offsets pass 2^31 and 2^32) with bf16 replicas: one warm-up round from
the zero EMA state through edit_outer_step_layer, at K = 2 (the VALU Gram
pass) and at K = 9 (the matrix-core Gram pass); at K = 2 also the same round
through two sync-group workers (the collectives stood in for on the
device); all against the oracle's full step.  The decision (G, w, Gbar,
beta) is compared in full; theta, b and the replicas at the first and last
65,536 elements (the ragged tail included) and at 2^20 seeded random
indices, to the usual tolerances.  Device memory: about 100 GB.
"""
import numpy as np
import pytest
import torch

from oracle import OracleConfig, OracleUnit
from parity import assert_replica_close, assert_tensor_close, host_bits
from paper_2412_07210_amd import EditOuter, OuterConfig, SyncGroupWorker, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
N = 2 ** 31 + 9


def _sample_idx(n):
    rng = np.random.default_rng(2 ** 31)
    edge = np.concatenate([np.arange(65_536), np.arange(n - 65_536, n)])
    return np.unique(np.concatenate([edge, rng.integers(0, n, 2 ** 20)]))


def _close(lib, ref, rtol, what):
    lib, ref = np.float64(lib), np.float64(ref)
    assert lib == ref or abs(lib - ref) <= rtol * abs(ref), f"{what}: library {lib} oracle {ref}"


# The oracle's single-threaded pass over 2^31 elements takes minutes, more
# than the per-test limit the GPU suite otherwise runs under.
@pytest.mark.timeout(900)
@pytest.mark.parametrize("K", [2, 9])
def test_unit_past_2_to_the_31_elements(K):
    if torch.cuda.get_device_properties(DEV).total_memory < 120 * 2 ** 30:
        pytest.skip("needs about 100 GB of device memory")
    group = K == 2
    wl = synth.small("llama1b-k8-bf16", [N], num_workers=K, name="max2p31")
    hyper = wl.hyper()
    warm = hyper.pop("warmup_rounds")
    cfg = OuterConfig(num_workers=K, layer_numel=[N], replica_dtype="bf16", ema_warmup_rounds=warm, **hyper)
    theta = wl.init_theta(0, DEV)
    reps = [torch.empty(N, dtype=torch.bfloat16, device=DEV) for _ in range(K)]
    wl.fill_replicas(theta, reps, 0, 0)
    theta_h = theta.cpu().numpy()
    reps_h = [host_bits(r) for r in reps]
    idx = _sample_idx(N)
    print(f"  n = {N:,}: inputs made", flush=True)

    # single-GPU step (all K replicas in this GPU's memory)
    lib = EditOuter(cfg, DEV)
    th1, b1, reps1 = theta.clone(), torch.zeros_like(theta), [r.clone() for r in reps]
    lib.step_layer(0, th1, b1, reps1)
    torch.cuda.synchronize(DEV)
    st = lib.state_get(0)
    lib.close()
    print("  single-GPU step done", flush=True)

    if group:
        gst, th2, b2, reps2 = _group_round(cfg, theta, reps, K)
    del theta, reps

    # the oracle's full step on host copies
    oracle = OracleUnit(K, OracleConfig(**wl.hyper()))
    mom_h = np.zeros(N, np.float32)
    rec = oracle.step(theta_h, mom_h, reps_h)
    print("  oracle done", flush=True)

    tol = 1e-12 + N * 2.0 ** -53
    checks = [("single-GPU", st, tol)] + ([("group rank 0", gst[0], 1e-5), ("group rank 1", gst[1], 1e-5)]
                                          if group else [])
    for what, s, gbar_tol in checks:
        assert np.array_equal(np.asarray(s.anomalous[:K], np.uint8), rec["anomalous"]), what
        assert s.round == 1 and not s.rolled_back, what
        for j in range(K):
            _close(s.norm[j], rec["norm"][j], tol, f"{what} G_{j}")
            _close(s.weight[j], rec["weight"][j], tol * (1 + max(rec["norm"])), f"{what} w_{j}")
        _close(s.synced_norm, rec["synced_norm"], max(gbar_tol, 1e-9), f"{what} Gbar")
        _close(s.clip_coef, rec["clip_coef"], max(gbar_tol, 1e-9), f"{what} beta")
    ti = torch.from_numpy(idx).to(DEV)
    outs = [("single-GPU", th1, b1, reps1[K - 1])] + ([("group rank 1", th2[1], b2[1], reps2[1])] if group else [])
    for what, th, b, rp in outs:
        assert_tensor_close(th[ti].cpu().numpy(), theta_h[idx], what + ": theta")
        assert_tensor_close(b[ti].cpu().numpy(), mom_h[idx], what + ": momentum")
        assert_replica_close(host_bits(rp[ti]), reps_h[K - 1][idx], True, what + ": replica")
    if group:  # every rank holds the same result
        for r in range(K):
            assert torch.equal(th2[r], th2[0]) and torch.equal(reps2[r].view(torch.int16), reps2[0].view(torch.int16))


def _group_round(cfg, theta, reps, K):
    """The same round as K sync-group workers on this device."""
    ranks = [SyncGroupWorker(cfg, r, DEV) for r in range(K)]
    th2 = [theta.clone() for _ in range(K)]
    b2 = [torch.zeros_like(theta) for _ in range(K)]
    reps2 = [r.clone() for r in reps]
    delta = [torch.empty_like(theta) for _ in range(K)]
    pairs = [w.norm(0, th2[r], reps2[r], delta[r]) for r, w in enumerate(ranks)]
    gathered = torch.stack(pairs).reshape(-1)
    wts = [w.weights(0, gathered, delta[r]) for r, w in enumerate(ranks)]
    dbar = delta[0].mul_(wts[0].to(torch.float32))
    dbar.add_(delta[1] * wts[1].to(torch.float32))
    del delta
    for r, w in enumerate(ranks):
        w.apply(0, dbar, th2[r], b2[r], reps2[r])
    torch.cuda.synchronize(DEV)
    gst = [w.state_get(0) for w in ranks]
    for w in ranks:
        w.close()
    print("  sync-group round done", flush=True)
    return gst, th2, b2, reps2
