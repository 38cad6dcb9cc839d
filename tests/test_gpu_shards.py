"""A module sharded over several units decides on norms of the whole module.

The paper takes every pseudo-gradient norm over an entire module even when the
module's parameters are sharded over a model-shard group (Sec. 3.1-3.2); the
shards exchange partial sums first.  Here each shard is a unit of one handle:
edit_outer_gram_layer per shard, the Gram vectors added on the device (the
stand-in for the group's all-reduce), then edit_outer_apply_layer per shard
with the sum.  The concatenated result must match the oracle stepping the
unsplit module (mask exact, tensors and scalars to the usual tolerances), and
every shard must hold the same decision and EMA state bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import OracleConfig, OracleUnit
from parity import (NearTie, assert_replica_close, assert_tensor_close, compare_decision,
                    host_bits)
from paper_2412_07210_amd import EditOuter, EditOuterError, OuterConfig, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _lib(wl, numel, flags=None):
    hyper = wl.hyper()
    kw = {} if flags is None else {"flags": flags}
    return EditOuter(OuterConfig(num_workers=wl.num_workers, layer_numel=numel,
                                 replica_dtype=wl.replica_dtype,
                                 ema_warmup_rounds=hyper.pop("warmup_rounds"), **hyper, **kw), DEV)


def _state_tuple(st, K):
    return (st.round, st.rolled_back, st.z_tested, tuple(st.anomalous[:K]),
            tuple(st.ema_mean[:K]), tuple(st.ema_std[:K]), tuple(st.norm[:K]),
            tuple(st.weight[:K]), st.synced_norm, st.clip_coef)


def _preset_ema(wl, n):
    """A post-warm-up EMA state (same on both sides) under which clean
    workers pass the z-test and x30 workers fail it."""
    G = wl.delta_std * np.sqrt(n)
    K = wl.num_workers
    return (np.full(K, 1.25 * G), np.full(K, 0.45 * G), wl.warmup_rounds)


def _sharded_rounds(wl, shards, rounds, ema=None, verbose=True, scale=None):
    """Lock-step: oracle on the whole module, library on its shards.  `ema`
    maps a round to the EMA state both sides take before that round, `scale`
    a round to a factor on every worker's pseudo gradient."""
    K, bf16 = wl.num_workers, wl.replica_dtype == "bf16"
    n = wl.unit_numel(0)
    assert sum(shards) == n
    cuts = np.cumsum([0] + list(shards))
    lib = _lib(wl, shards)
    oracle = OracleUnit(K, OracleConfig(**wl.hyper()))
    ema = ema or {}
    theta_h = wl.init_theta(0, DEV).cpu().numpy().copy()
    mom_h = np.zeros(n, np.float32)
    try:
        for t in rounds:
            what = f"{wl.name} n={n} shards={list(shards)} round {t}"
            if t in ema:
                oracle.set_state(*ema[t])
                for s in range(len(shards)):
                    lib.state_set(s, *ema[t])
            theta = torch.from_numpy(theta_h).to(DEV)
            reps = [torch.empty(n, dtype=wl.torch_dtype, device=DEV) for _ in range(K)]
            wl.fill_replicas(theta, reps, 0, t, std=wl.worker_std(t) * (scale or {}).get(t, 1.0))
            reps_h = [host_bits(r) for r in reps]
            # each shard in buffers of its own (16-byte aligned, as a device would hold them)
            th_s = [theta[a:b].clone() for a, b in zip(cuts[:-1], cuts[1:])]
            mo_s = [torch.from_numpy(mom_h[a:b].copy()).to(DEV) for a, b in zip(cuts[:-1], cuts[1:])]
            rp_s = [[r[a:b].clone() for r in reps] for a, b in zip(cuts[:-1], cuts[1:])]
            grams = [lib.gram_layer(s, th_s[s], rp_s[s]) for s in range(len(shards))]
            total = grams[0].clone()
            for g in grams[1:]:
                total += g
            for s in range(len(shards)):
                lib.apply_layer(s, total, th_s[s], mo_s[s], rp_s[s])
            rec = oracle.step(theta_h, mom_h, reps_h)
            torch.cuda.synchronize(DEV)
            states = [lib.state_get(s) for s in range(len(shards))]
            compare_decision(states[0], rec, K, what)
            for s in range(1, len(shards)):
                assert _state_tuple(states[s], K) == _state_tuple(states[0], K), \
                    f"{what}: shard {s} decided differently from shard 0"
            th = torch.cat(th_s)
            assert_tensor_close(th.cpu().numpy(), theta_h, what + ": theta")
            assert_tensor_close(torch.cat(mo_s).cpu().numpy(), mom_h, what + ": momentum")
            # the oracle gives every worker the same value, so replica 0 against
            # the oracle and every replica against the cast of theta cover all
            expect = th.to(wl.torch_dtype)
            for j in range(K):
                r = torch.cat([rp_s[s][j] for s in range(len(shards))])
                assert torch.equal(r.view(torch.int16) if bf16 else r,
                                   expect.view(torch.int16) if bf16 else expect), \
                    f"{what}: replica {j} is not the cast of theta"
                assert np.array_equal(reps_h[j], reps_h[0]), f"{what}: oracle replicas differ"
                if j == 0:
                    assert_replica_close(host_bits(r), reps_h[0], bf16, what + ": replica 0")
            if verbose:
                print(f"  {what}: mask {list(rec['anomalous'])} beta {rec['clip_coef']:.4f} "
                      f"rolled_back {rec['rolled_back']}", flush=True)
            yield rec
    finally:
        lib.close()


@pytest.mark.parametrize("K,dtype", [(4, "f32"), (8, "bf16"), (11, "bf16"), (16, "bf16"), (24, "bf16"),
                                     (32, "f32")])
@pytest.mark.parametrize("shards", [(40000, 33333, 26670), (100003, 0), (8, 99995)])
def test_sharded_module_matches_unsplit_oracle(K, dtype, shards):
    """Three-way ragged split, an empty shard, and an 8-element shard.  Two
    warm-up rounds from the zero EMA state, then (from a preset post-warm-up
    state) two rounds in which three workers are x30 and must be masked."""
    wl = synth.small("aedit1b-k16-bf16", [sum(shards)], num_workers=K, replica_dtype=dtype)
    rounds = [0, 1, wl.warmup_rounds, wl.warmup_rounds + 1]
    try:
        recs = list(_sharded_rounds(wl, shards, rounds,
                                    ema={wl.warmup_rounds: _preset_ema(wl, sum(shards))}))
    except NearTie as e:
        pytest.skip(str(e))
    assert not recs[0]["anomalous"].any() and not recs[1]["anomalous"].any()
    assert recs[2]["anomalous"].sum() == 3 and not recs[2]["rolled_back"]


def test_sharded_module_rollback_and_clip():
    """phi small enough to clip in a warm-up round; after the warm-up, from a
    settled EMA state, every worker x100: all fail the z-test on the module
    norm and the module rolls back (twice, the state being unchanged)."""
    wl = synth.small("linear1m-k4", [65536 + 4099], num_workers=4, replica_dtype="bf16",
                     clip_threshold=1e-3)
    W = wl.warmup_rounds
    try:
        recs = list(_sharded_rounds(wl, (65536, 4099), [0, W, W + 1],
                                    ema={W: _preset_ema(wl, 65536 + 4099)}, scale={W: 100.0, W + 1: 100.0}))
    except NearTie as e:
        pytest.skip(str(e))
    assert recs[0]["clip_coef"] < 1.0 and not recs[0]["rolled_back"]
    assert recs[1]["rolled_back"] and recs[2]["rolled_back"]


@pytest.mark.parametrize("K,dtype,n", [(8, "bf16", 3_000_017), (4, "f32", 1_000_005),
                                       (16, "bf16", 2_000_003), (11, "f32", 65_537),
                                       (21, "f32", 300_001), (32, "bf16", 1_000_003)])
def test_gram_then_apply_is_step_layer_bitwise(K, dtype, n):
    """For an unsplit unit the two-call path is the one-call path, bit for bit:
    a warm-up round, then two rounds with three x30 workers."""
    wl = synth.small("aedit1b-k16-bf16", [n], num_workers=K, replica_dtype=dtype)
    a, b = _lib(wl, [n]), _lib(wl, [n])
    th0 = wl.init_theta(0, DEV)
    tha, thb = th0.clone(), th0.clone()
    moa, mob = torch.zeros_like(th0), torch.zeros_like(th0)
    try:
        for t in [0, wl.warmup_rounds, wl.warmup_rounds + 1]:
            if t == wl.warmup_rounds:
                for h in (a, b):
                    h.state_set(0, *_preset_ema(wl, n))
            ra = [torch.empty(n, dtype=wl.torch_dtype, device=DEV) for _ in range(K)]
            wl.fill_replicas(tha, ra, 0, t)
            rb = [r.clone() for r in ra]
            a.step_layer(0, tha, moa, ra)
            gram = b.gram_layer(0, thb, rb)
            b.apply_layer(0, gram, thb, mob, rb)
            torch.cuda.synchronize(DEV)
            assert torch.equal(tha, thb) and torch.equal(moa, mob), f"round {t}: theta/b differ"
            for j in range(K):
                assert torch.equal(ra[j].view(torch.int16) if dtype == "bf16" else ra[j],
                                   rb[j].view(torch.int16) if dtype == "bf16" else rb[j])
            sa, sb = a.state_get(0), b.state_get(0)
            assert _state_tuple(sa, K) == _state_tuple(sb, K)
            assert sa.anomalous[:K].sum() == (3 if t >= wl.warmup_rounds else 0)
            # the diagonal of the exported Gram holds G_j^2
            diag = gram.cpu().numpy()[[j * K - j * (j - 1) // 2 for j in range(K)]]
            np.testing.assert_allclose(np.sqrt(diag), np.asarray(sb.norm[:K]), rtol=1e-15)
    finally:
        a.close()
        b.close()


def test_full_size_7b_layer_as_two_shards():
    """A 202,383,360-element module (the size of a whole 7B decoder layer) as
    two contiguous halves of 101,191,680 (each the shape of the 7B half-shard
    workload), one round from a preset post-warm-up EMA state: the decision
    covers both halves, and clipping is active."""
    n_half = synth.get("llama7b-half-k8-bf16").unit_numel(0)
    wl = synth.small("llama7b-half-k8-bf16", [2 * n_half])
    try:
        recs = list(_sharded_rounds(wl, (n_half, n_half), [wl.warmup_rounds],
                                    ema={wl.warmup_rounds: _preset_ema(wl, 2 * n_half)}))
    except NearTie as e:
        pytest.skip(str(e))
    assert recs[0]["clip_coef"] < 1.0 and not recs[0]["anomalous"].any()


def test_gram_and_apply_reject_bad_arguments():
    wl = synth.small("linear1m-k4", [1024], num_workers=2, replica_dtype="f32")
    lib = _lib(wl, [1024])
    try:
        th = torch.zeros(1024, device=DEV)
        mo = torch.zeros(1024, device=DEV)
        reps = [torch.zeros(1024, device=DEV) for _ in range(2)]
        with pytest.raises(ValueError):
            lib.gram_layer(0, th, reps, gram=torch.zeros(2, dtype=torch.float64, device=DEV))
        with pytest.raises(ValueError):
            lib.apply_layer(0, torch.zeros(3, dtype=torch.float32, device=DEV), th, mo, reps)
        # a Gram vector inside theta's range is refused by the library itself
        big = torch.zeros(1024 + 8, dtype=torch.float64, device=DEV)
        th64 = big[:512].view(torch.float32)
        with pytest.raises(EditOuterError, match="overlap"):
            lib.gram_layer(0, th64, reps, gram=big[510:513])
    finally:
        lib.close()
