"""One worker's share of a sync group whose K replicas sit on K GPUs,
simulated on one GPU.

K SyncGroupWorker handles (ranks 0..K-1) share the device, each with its own
copy of theta and b and its own replica, as K GPUs would hold them.  The two
collectives between the calls are stood in for on the device: the
all-gather stacks the ranks' {G, flag} pairs in rank order, and the
all-reduce sums w_j * delta_j in fp32 in rank order (a pre-multiplied sum, up
to the summation order a collective would use).  Every rank must end with
the same theta, b and replica bit for bit, and they must match the oracle's
full step on all K replicas (Sec. 3.2, Algorithm 2): theta and b to the usual
tolerance, the replica as the cast of theta, the mask exactly, and Gbar and
beta to 1e-5 (here Delta_bar is summed from fp32 pseudo gradients).  Each
G_j and each rank's EMA pair are fp64 sums on both sides in different orders:
they must agree to 1e-12 + n 2^-53 relative (the rounding bound of the
oracle's sequential sum), the weights to that times (1 + max G), since
exp(-G) turns an absolute error of G into a relative one of w.
"""
import numpy as np
import pytest
import torch

from oracle import OracleConfig, OracleUnit
from parity import NEAR_TIE, NearTie, assert_replica_close, assert_tensor_close, host_bits
from paper_2412_07210_amd import EditOuterError, OuterConfig, SyncGroupWorker, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _close(lib, ref, rtol, what):
    lib = np.asarray(lib, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    ok = (lib == ref) | (np.abs(lib - ref) <= rtol * np.abs(ref)) | (np.isnan(lib) & np.isnan(ref))
    assert ok.all(), f"{what}: library {lib} oracle {ref}"


class Group:
    """K ranks on one device, lock-step with the oracle over one module."""

    def __init__(self, wl, n, ema=None):
        self.wl, self.n, self.K = wl, n, wl.num_workers
        hyper = wl.hyper()
        warm = hyper.pop("warmup_rounds")
        cfg = OuterConfig(num_workers=self.K, layer_numel=[n], replica_dtype=wl.replica_dtype,
                          ema_warmup_rounds=warm, **hyper)
        self.ranks = [SyncGroupWorker(cfg, r, DEV) for r in range(self.K)]
        self.oracle = OracleUnit(self.K, OracleConfig(**wl.hyper()))
        self.theta_h = wl.init_theta(0, DEV)[:n].cpu().numpy().copy()
        self.mom_h = np.zeros(n, np.float32)
        self.ema = ema or {}

    def close(self):
        for w in self.ranks:
            w.close()

    def round(self, t, std=None, poison=None):
        K, n, wl = self.K, self.n, self.wl
        what = f"{wl.name} K={K} n={n} round {t}"
        if t in self.ema:
            mu, sigma, r0 = self.ema[t]
            self.oracle.set_state(mu, sigma, r0)
            for r, w in enumerate(self.ranks):
                w.state_set(0, mu[r], sigma[r], r0)
        theta = torch.from_numpy(self.theta_h).to(DEV)
        reps = [torch.empty(n, dtype=wl.torch_dtype, device=DEV) for _ in range(K)]
        if n:
            wl.fill_replicas(theta, reps, 0, t, std=std)
        if poison is not None and n:
            reps[poison][n // 2] = float("nan")
        reps_h = [host_bits(r) for r in reps]
        # each rank's own copies, as on its own GPU
        th = [theta.clone() for _ in range(K)]
        mo = [torch.from_numpy(self.mom_h).to(DEV) for _ in range(K)]
        delta = [torch.empty(n, dtype=torch.float32, device=DEV) for _ in range(K)]
        pairs = [w.norm(0, th[r], reps[r], delta[r]) for r, w in enumerate(self.ranks)]
        gathered = torch.stack(pairs).reshape(-1)                  # the all-gather
        wts = [w.weights(0, gathered, delta[r]) for r, w in enumerate(self.ranks)]
        dbar = torch.zeros(n, dtype=torch.float32, device=DEV)      # the all-reduce
        for r in range(K):
            dbar += wts[r].to(torch.float32) * delta[r]
        for r, w in enumerate(self.ranks):
            w.apply(0, dbar, th[r], mo[r], reps[r])
        rec = self.oracle.step(self.theta_h, self.mom_h, reps_h)
        torch.cuda.synchronize(DEV)

        states = [w.state_get(0) for w in self.ranks]
        tol = 1e-12 + n * 2.0 ** -53
        gmax = float(np.max(rec["norm"][np.isfinite(rec["norm"])], initial=0.0))
        for r, st in enumerate(states):
            who = f"{what} rank {r}"
            mask_l = np.asarray(st.anomalous[:K], dtype=np.uint8)
            near = np.asarray(rec["margin"][:K]) < NEAR_TIE
            if np.any(mask_l[near] != rec["anomalous"][near]):
                raise NearTie(f"{who}: z-test within {NEAR_TIE} of a tie")
            assert np.array_equal(mask_l, rec["anomalous"]), f"{who}: mask {mask_l} vs {rec['anomalous']}"
            assert st.round == rec["round"] and int(st.rolled_back) == rec["rolled_back"], who
            assert int(st.z_tested) == rec["z_tested"], who
            _close(st.norm, rec["norm"], tol, who + ": G")
            _close(st.weight, rec["weight"], tol * (1.0 + gmax), who + ": w")
            _close(st.ema_mean[r], rec["mu"][r], tol, who + ": mu")
            _close(st.ema_std[r], rec["sigma"][r], tol, who + ": sigma")
            if not rec["rolled_back"]:
                _close(st.synced_norm, rec["synced_norm"], 1e-5, who + ": Gbar")
                _close(st.clip_coef, rec["clip_coef"], 1e-5, who + ": beta")
        bf16 = wl.replica_dtype == "bf16"
        for r in range(1, K):  # every rank computed the same thing
            assert torch.equal(th[r], th[0]) and torch.equal(mo[r], mo[0]), f"{what}: rank {r} differs"
        assert_tensor_close(th[0].cpu().numpy(), self.theta_h, what + ": theta")
        assert_tensor_close(mo[0].cpu().numpy(), self.mom_h, what + ": momentum")
        expect = th[0].to(wl.torch_dtype)
        for r in range(K):
            got = reps[r].view(torch.int16) if bf16 else reps[r]
            assert torch.equal(got, expect.view(torch.int16) if bf16 else expect), \
                f"{what}: replica of rank {r} is not the cast of theta"
        if n:
            assert_replica_close(host_bits(reps[0]), reps_h[0], bf16, what + ": replica")
        return rec, states


def _preset(wl, n, K):
    """A post-warm-up EMA state under which clean workers pass the z-test and
    x30 workers fail it (same on both sides)."""
    G = wl.delta_std * np.sqrt(max(n, 1))
    return (np.full(K, 1.25 * G), np.full(K, 0.45 * G), wl.warmup_rounds)


@pytest.mark.parametrize("K,dtype", [(1, "bf16"), (2, "f32"), (4, "bf16"), (8, "bf16"), (8, "f32"),
                                     (13, "bf16"), (16, "bf16")])
@pytest.mark.parametrize("n", [0, 1, 9, 4099, 1_000_003])
def test_group_matches_the_full_step(K, dtype, n):
    """Two warm-up rounds from the zero EMA state, then, from a preset
    post-warm-up state, two rounds in which three workers are x30 (for K < 4
    the last worker is x50) and must be masked by their own z-tests."""
    mode = "three_x30_after_warmup" if K >= 4 else "last_x50_from_round_10"
    wl = synth.small("aedit1b-k16-bf16", [max(n, 1)], num_workers=K, replica_dtype=dtype,
                     anomaly_mode=mode, name=f"grp{K}{dtype}")
    W = wl.warmup_rounds
    g = Group(wl, n, ema={W: _preset(wl, n, K)})
    try:
        recs = [g.round(t)[0] for t in [0, 1, W, W + 1]]
    except NearTie as e:
        pytest.skip(str(e))
    finally:
        g.close()
    if n >= 4099 and K >= 4:  # enough elements for the x30 norms to stand out
        assert recs[2]["anomalous"].sum() == 3 and not recs[2]["rolled_back"]


def test_group_rollback_and_clip():
    """phi small enough to clip in a warm-up round; after the warm-up, from a
    settled EMA state, every worker x100 fails its own z-test, so the round
    rolls back on every rank."""
    wl = synth.small("linear1m-k4", [70_001], num_workers=4, replica_dtype="bf16", clip_threshold=1e-3)
    W = wl.warmup_rounds
    g = Group(wl, 70_001, ema={W: _preset(wl, 70_001, 4)})
    try:
        r0, _ = g.round(0)
        r1, states = g.round(W, std=wl.worker_std(W) * 100.0)
    finally:
        g.close()
    assert r0["clip_coef"] < 1.0 and not r0["rolled_back"]
    assert r1["rolled_back"] and all(st.rolled_back for st in states)


def test_group_nan_worker_is_left_out():
    """Rank 2's replica holds a NaN: its norm is NaN, it is flagged by every
    rank (even in the warm-up), its export is cleared before the sum, and
    theta stays finite."""
    wl = synth.small("llama1b-k8-bf16", [50_000], num_workers=5, name="grpnan")
    g = Group(wl, 50_000)
    try:
        rec, states = g.round(0, poison=2)
    finally:
        g.close()
    assert list(rec["anomalous"]) == [0, 0, 1, 0, 0]
    assert all(st.weight[2] == 0.0 and np.isnan(st.norm[2]) for st in states)
    assert np.isfinite(g.theta_h).all()


def test_group_full_size_1b_unit():
    """One 51,384,320-element unit of the 1B K = 8 bf16 workload on all eight
    ranks, in the post-warm-up state with the round-19 x20 worker."""
    wl = synth.get("llama1b-k8-bf16")
    n, K = wl.unit_numel(0), wl.num_workers
    g = Group(wl.with_units([0]), n, ema={19: _preset(wl, n, K)})
    try:
        rec, _ = g.round(19)
    except NearTie as e:
        pytest.skip(str(e))
    finally:
        g.close()
    assert rec["anomalous"].sum() >= 1 and not rec["rolled_back"]


def test_group_rejects_bad_arguments():
    cfg = OuterConfig(num_workers=2, layer_numel=[1024], replica_dtype="f32")
    w = SyncGroupWorker(cfg, 1, DEV)
    try:
        th = torch.zeros(1024, device=DEV)
        rep = torch.zeros(1024, device=DEV)
        big = torch.zeros(2048 + 4, device=DEV)
        with pytest.raises(EditOuterError, match="overlap"):  # delta inside theta's range
            w.norm(0, big[:1024], rep, big[512:1536])
        with pytest.raises(EditOuterError, match="aligned"):
            w.norm(0, th, rep, big[1:1025])
        with pytest.raises(ValueError):
            w.weights(0, torch.zeros(3, dtype=torch.float64, device=DEV), th)
        with pytest.raises(EditOuterError, match="state"):
            w.state_get(0)
        w.state_set(0, 2.0, 0.5, 7)
        st = w.state_get(0)
        assert st.round == 7 and st.ema_mean[1] == 2.0 and st.ema_std[1] == 0.5 and st.ema_mean[0] == 0.0
    finally:
        w.close()
