"""GPU parity of the one-pass mean step (flag EDIT_ONE_PASS) against the oracle.

With anomaly elimination, weighted averaging and clipping all off (the
"w/o ALL" ablation of Sec. 4.5, the DiLoCo outer step) every weight is 1/K,
and the library runs the average, Nesterov and the write-back in one pass.
The oracle steps with all three components off; for finite inputs both
compute the same thing, so the usual tolerances apply, and the reported
norms G_j and ||Delta_bar|| are compared too.
"""
import numpy as np
import pytest
import torch

from parity import NearTie, ParityRun
from paper_2412_07210_amd import AE, ONE_PASS, EditOuter, EditOuterError, OuterConfig, synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _run(run, rounds, **kw):
    try:
        return [run.round(t, verbose=False, **kw) for t in rounds]
    except NearTie as e:  # no z-test in this mode, so this does not happen
        pytest.skip(str(e))
    finally:
        run.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K", [1, 2, 3, 5, 8, 9, 13, 16])
def test_one_pass_ragged_sizes(K, dtype):
    """Unit sizes around the 16-byte vector and the block, K = 1..16."""
    sizes = [0, 1, 7, 8, 9, 255, 2049, 100_003, 1_000_005]
    wl = synth.small("llama1b-k8-bf16", sizes, num_workers=K, replica_dtype=dtype, name=f"onepass{K}{dtype}")
    recs = _run(ParityRun(wl, range(len(sizes)), DEV, flags=ONE_PASS), range(3))
    for r in recs[-1]:
        assert r["state"].round == 3
        assert not r["state"].anomalous.any() and r["state"].clip_coef == 1.0
        np.testing.assert_array_equal(r["state"].weight[:K], np.full(K, 1.0 / K))


def test_one_pass_full_size_1b_units():
    """Two 51,384,320-element units of the 1B K=8 bf16 workload, in the launch
    configuration of a handle holding all 24 units."""
    wl = synth.get("llama1b-k8-bf16")
    _run(ParityRun(wl, [0, 23], DEV, flags=ONE_PASS), [10, 19])


def test_one_pass_full_size_k16():
    """A 51,380,224-element unit and a 2,048-element unit at K = 16."""
    wl = synth.get("aedit1b-k16-bf16")
    _run(ParityRun(wl, [0, 1], DEV, flags=ONE_PASS), [0])


def _fresh(wl, u, t):
    th = wl.init_theta(u, DEV)
    reps = [torch.empty(th.numel(), dtype=wl.torch_dtype, device=DEV) for _ in range(wl.num_workers)]
    wl.fill_replicas(th, reps, u, t)
    return th, torch.zeros_like(th), reps


@pytest.mark.parametrize("K,dtype", [(8, "bf16"), (4, "f32"), (16, "bf16")])
def test_one_pass_round_matches_unit_by_unit(K, dtype):
    """A round (fused passes back to back, one batched record launch at the
    end) gives the same bits and records as unit-by-unit calls."""
    sizes = [1_000_000, 2048, 7, 3_000_017, 0, 65_536 + 3]
    wl = synth.small("llama1b-k8-bf16", sizes, num_workers=K, replica_dtype=dtype, name=f"oproun{K}{dtype}")
    order = [2, 0, 5, 1, 4, 3]
    results = []
    for mode in ("layer", "round"):
        h = EditOuter(OuterConfig(K, wl.layer_numel, dtype, flags=ONE_PASS), DEV)
        units = [_fresh(wl, u, 0) for u in range(wl.num_units)]
        for t in range(3):
            for u in range(wl.num_units):
                wl.fill_replicas(units[u][0], units[u][2], u, t)
            if mode == "layer":
                for u in order:
                    h.step_layer(u, *units[u])
            else:
                h.step_round([units[u] for u in order], layers=order)
            torch.cuda.synchronize()
        results.append((units, [h.state_get(u) for u in range(wl.num_units)]))
        h.close()
    (ua, sa), (ub, sb) = results
    for a, b in zip(ua, ub):
        assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
        assert all(torch.equal(x, y) for x, y in zip(a[2], b[2]))
    for x, y in zip(sa, sb):
        assert np.array_equal(x.norm, y.norm) and x.synced_norm == y.synced_norm
        assert x.round == y.round == 3


def test_one_pass_nonfinite_is_reported_not_masked():
    """There is no norm before the average in this mode: a NaN in a replica
    reaches theta at that element, and the worker's reported G_j is NaN."""
    wl = synth.small("llama1b-k8-bf16", [10_000], num_workers=5, name="opnan")
    h = EditOuter(OuterConfig(5, wl.layer_numel, "bf16", flags=ONE_PASS), DEV)
    try:
        th, b, reps = _fresh(wl, 0, 0)
        reps[2][13] = float("nan")
        h.step_layer(0, th, b, reps)
        torch.cuda.synchronize()
        st = h.state_get(0)
        assert np.isnan(st.norm[2]) and np.isfinite(np.delete(st.norm[:5], 2)).all()
        assert not st.anomalous.any()
        theta = th.cpu().numpy()
        assert np.isnan(theta[13]) and np.isfinite(np.delete(theta, 13)).all()
    finally:
        h.close()


def test_one_pass_flag_rules():
    """EDIT_ONE_PASS needs the three components clear, and the Gram entry
    points are refused in this mode."""
    with pytest.raises(EditOuterError, match="ONE_PASS"):
        EditOuter(OuterConfig(4, [1024], "bf16", flags=ONE_PASS | AE), DEV)
    h = EditOuter(OuterConfig(4, [1024], "bf16", flags=ONE_PASS), DEV)
    try:
        th = torch.zeros(1024, device=DEV)
        reps = [torch.zeros(1024, dtype=torch.bfloat16, device=DEV) for _ in range(4)]
        with pytest.raises(EditOuterError, match="ONE_PASS"):
            h.gram_layer(0, th, reps)
    finally:
        h.close()
