"""Every worker count the library accepts, K = 1..32, against the oracle (GPU).

The kernels are instantiated once per K (VALU Gram accumulators up to
K = 8, matrix-core tiles above: G = ceil(K/4) worker groups, the last one
partly empty unless 4 divides K).  Each K steps two units through
edit_outer_step_round for three rounds after the warm-up (Sec. 3.2,
Algorithm 2): a 131,075-element unit (several Gram-pass blocks, a last
group of vectors cut short by the unit's end, and a ragged tail) and a
2,051-element unit of at most 256 vectors, stepped whole in a small launch.
Replicas alternate between bf16 and fp32 with K; the last round scales the
last worker x40, which the z-test must flag on the larger unit while every
other worker passes.  The one-pass mean step runs for every K on the same
units, with the replica type the other way round.
"""
import numpy as np
import pytest

from parity import NearTie, ParityRun, steady_ema
from paper_2412_07210_amd import ONE_PASS, synth
from paper_2412_07210_amd.outer import MAX_K

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
SIZES = [131_075, 2_051]


@pytest.mark.parametrize("K", range(1, MAX_K + 1))
def test_every_worker_count(K):
    dtype = "bf16" if K % 2 else "f32"
    wl = synth.small("llama1b-k8-bf16", SIZES, num_workers=K, replica_dtype=dtype, clip_threshold=0.05,
                     name=f"everyk{K}{dtype}")
    W = wl.warmup_rounds
    run = ParityRun(wl, range(len(SIZES)), DEV,
                    ema_state={u: steady_ema(wl, n, W) for u, n in enumerate(SIZES)})
    try:
        for t in range(W, W + 3):
            last = t == W + 2
            std = wl.worker_std(t) * (np.where(np.arange(K) == K - 1, 40.0, 1.0) if last else 1.0)
            recs = run.round(t, std=std, via_round=True, verbose=False)
            big = recs[0]
            assert big["z_tested"], f"K={K} round {t}: not z-tested"
            bad = [K - 1] if last else []
            flagged = sorted(np.flatnonzero(big["anomalous"][:K]).tolist())
            if K > 1 or not last:
                assert flagged == bad, f"K={K} round {t}: flagged {flagged}, expected {bad}"
    except NearTie as e:
        pytest.skip(str(e))
    finally:
        run.close()


@pytest.mark.parametrize("K", range(1, MAX_K + 1))
def test_every_worker_count_one_pass(K):
    """The one-pass mean step (EDIT_ONE_PASS: no penalty component, the
    DiLoCo outer step) for every K on the same two units, two rounds."""
    dtype = "f32" if K % 2 else "bf16"
    wl = synth.small("llama1b-k8-bf16", SIZES, num_workers=K, replica_dtype=dtype, name=f"everyk1p{K}{dtype}")
    run = ParityRun(wl, range(len(SIZES)), DEV, flags=ONE_PASS)
    try:
        for t in range(2):
            run.round(t, via_round=True, verbose=False)
    finally:
        run.close()
