"""Seeded fuzz of the round path (GPU; a tool, not collected by pytest).

    python tests/fuzz_round.py [CASES [FIRST]]      # FUZZ_SECONDS caps the run time

Case i draws, from seed 5000 + i: K (1 to 16), one to seven units whose
sizes range from 0 to 4,194,305 elements (so rounds mix single-block units,
stepped whole in small launches, with larger ones), the replica type, the
penalty switches or the one-pass mode, and hyper-parameters with edge values.
Two handles then step the same inputs for four rounds, one through
edit_outer_step_round in a shuffled unit order and one through
edit_outer_step_layer, and the oracle steps a third copy.  Checked every
round: the two handles agree bit for bit (theta, b, replicas, records); every
replica is the cast of theta; the decision and theta, b match the oracle
within the parity bars of tests/parity.py.  Some rounds put a NaN, an Inf or
1e30 into one replica element, and some cases restore a perturbed EMA state
after the first round.  In the one-pass mode a non-finite replica reaches
theta by design (there is no norm before the average), so such a unit is
only held to the bitwise agreement of the two handles from then on.
"""
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))
from oracle import OracleConfig, OracleUnit  # noqa: E402
from parity import NearTie, assert_tensor_close, compare_decision, host_bits  # noqa: E402
from paper_2412_07210_amd import ONE_PASS, EditOuter, OuterConfig, synth  # noqa: E402

DEV = torch.device("cuda:0")


def bits(t):
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t).cpu().numpy().tobytes()


def case(i):
    rng = np.random.default_rng(5000 + i)
    K = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 9, 12, 13, 16]))
    L = int(rng.integers(1, 8))
    sizes = [int(x) for x in rng.choice([0, 1, 5, 8, 9, 33, 257, 4099, 65_537, 300_001, 1_000_003, 4_194_305], size=L,
                                         p=[.08, .08, .08, .08, .08, .08, .1, .1, .1, .1, .08, .04])]
    dtype = str(rng.choice(["f32", "bf16"]))
    flags = int(rng.integers(0, 10))
    if flags >= 8:
        flags = ONE_PASS
    hyper = dict(outer_lr=float(rng.choice([0.1, 0.8, 1.4])), momentum=float(rng.choice([0.0, 0.85, 0.99])),
                 clip_threshold=float(rng.choice([0.0, 1e-3, 0.05, 10.0])), clip_eps=float(rng.choice([1e-6, 1e-3])),
                 ema_alpha=float(rng.choice([0.02, 0.3, 1.0])), z_threshold=float(rng.choice([0.0, 1.0, 3.0])),
                 warmup_rounds=int(rng.choice([0, 1, 2, 10])))
    wl = synth.small("llama1b-k8-bf16", sizes, num_workers=K, replica_dtype=dtype, name=f"fuzz{i}", **hyper)
    h = wl.hyper()
    warm = h.pop("warmup_rounds")
    cfg = OuterConfig(K, wl.layer_numel, dtype, ema_warmup_rounds=warm, flags=flags, **h)
    A, B = EditOuter(cfg, DEV), EditOuter(cfg, DEV)
    oc = OracleConfig(**wl.hyper(), flags=flags & 7)
    orc = [OracleUnit(K, oc) for _ in range(L)]
    th_h = [wl.init_theta(u, DEV).cpu().numpy().copy() for u in range(L)]
    mo_h = [np.zeros(sizes[u], np.float32) for u in range(L)]
    order = [int(x) for x in rng.permutation(L)]
    poisoned, reset = [], [0] * L
    try:
        for t in range(4):
            std = wl.worker_std(t)
            for j in range(K):
                x = rng.random()
                std[j] *= 30.0 if x < 0.15 else (1000.0 if x < 0.2 else 1.0)
            ua, ub, reps_h = [], [], []
            for u in range(L):
                th = torch.from_numpy(th_h[u]).to(DEV)
                reps = [torch.empty(sizes[u], dtype=wl.torch_dtype, device=DEV) for _ in range(K)]
                if sizes[u]:
                    wl.fill_replicas(th, reps, u, t, std=std)
                reps_h.append([host_bits(r) for r in reps])
                mo = torch.from_numpy(mo_h[u]).to(DEV)
                ua.append((th, mo, reps))
                ub.append((th.clone(), mo.clone(), [r.clone() for r in reps]))
            if rng.random() < 0.15:
                u = int(rng.integers(0, L))
                if sizes[u]:
                    j, k = int(rng.integers(0, K)), int(rng.integers(0, sizes[u]))
                    val = float(rng.choice([np.nan, np.inf, -np.inf, 1e30]))
                    for rep in (ua[u][2][j], ub[u][2][j]):
                        rep[k] = val
                    reps_h[u][j] = host_bits(ua[u][2][j])
                    poisoned.append((t, u, j, k, val))
            A.step_round([ua[u] for u in order], layers=order)
            for u in order:
                B.step_layer(u, *ub[u])
            recs = [orc[u].step(th_h[u], mo_h[u], reps_h[u]) for u in range(L)]
            torch.cuda.synchronize()
            for u in range(L):
                what = f"case {i} unit {u} round {t} poisoned {poisoned}"
                sa, sb = A.state_get(u), B.state_get(u)
                assert bits(ua[u][0]) == bits(ub[u][0]) and bits(ua[u][1]) == bits(ub[u][1]), what + ": round != layer"
                assert all(bits(x) == bits(y) for x, y in zip(ua[u][2], ub[u][2])), what + ": replicas"
                # one-pass mode: a non-finite replica reaches theta by design (no norm
                # before the average), so that unit leaves the oracle comparison
                tainted = flags == ONE_PASS and any(p[1] == u for p in poisoned)
                cast = bits(ua[u][0].to(wl.torch_dtype))
                if not tainted:
                    assert all(bits(x) == cast for x in ua[u][2]), what + ": replica != cast(theta)"
                for f in ("norm", "weight", "ema_mean", "ema_std", "anomalous", "synced_norm", "clip_coef",
                          "round", "rolled_back", "z_tested"):
                    assert np.asarray(getattr(sa, f)).tobytes() == np.asarray(getattr(sb, f)).tobytes(), what + " " + f
                assert sa.round == t + 1 + reset[u], what
                if flags != ONE_PASS:
                    compare_decision(sa, recs[u], K, what)
                if not tainted:
                    assert_tensor_close(ua[u][0].cpu().numpy(), th_h[u], what + ": theta")
                    assert_tensor_close(ua[u][1].cpu().numpy(), mo_h[u], what + ": b")
            if t == 0 and rng.random() < 0.3:
                for u in range(L):
                    mu = orc[u].mu * rng.uniform(0.5, 2.0, K)
                    sg = orc[u].sigma * rng.uniform(0.5, 2.0, K)
                    if not (np.isfinite(mu).all() and np.isfinite(sg).all()):
                        continue
                    r = int(rng.integers(0, 20))
                    for side in (A, B):
                        side.state_set(u, mu, sg, r)
                    orc[u].set_state(mu, sg, r)
                    reset[u] = r - 1
    except NearTie as e:
        return f"near tie: {e}"
    except AssertionError as e:
        return f"FAIL K={K} L={L} sizes={sizes} {dtype} flags={flags} {hyper}: {e}"
    finally:
        A.close()
        B.close()
    return f"ok K={K} L={L} {dtype} flags={flags}"


def main() -> int:
    n = int(sys.argv[1]) if len(sys.argv) > 1 else 300
    first = int(sys.argv[2]) if len(sys.argv) > 2 else 0
    budget = float(os.environ.get("FUZZ_SECONDS", "760"))
    t0 = time.time()
    done = failed = skipped = 0
    for i in range(first, first + n):
        if time.time() - t0 > budget:
            print(f"time budget reached before case {i}", flush=True)
            break
        r = case(i)
        done += 1
        skipped += r.startswith("near")
        failed += r.startswith("FAIL")
        if i % 20 == 0 or not r.startswith("ok"):
            print(f"[{time.time() - t0:.0f}s] case {i}: {r}", flush=True)
    print(f"done: {done} cases, {failed} failed, {skipped} near ties, {time.time() - t0:.0f}s", flush=True)
    return 1 if failed else 0


if __name__ == "__main__":
    sys.exit(main())
