"""theta and momentum in host memory: edit_outer_step_round_host.

The paper keeps the outer optimizer's state off the accelerator to save its
memory (Sec. 3.2).  Here theta_t and b live in pinned host memory; each unit
is copied to a device staging slot, stepped by the resident kernels, and
copied back, overlapped over a ring of three slots.  The results must be the
resident round's bit for bit, and match the oracle.
"""
import ctypes

import numpy as np
import pytest
import torch

from oracle import OracleConfig, OracleUnit
from parity import assert_tensor_close, compare_decision, host_bits
from paper_2412_07210_amd import ONE_PASS, EditOuter, OuterConfig, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _inputs(wl, u, t):
    th = wl.init_theta(u, DEV)
    reps = [torch.empty(th.numel(), dtype=wl.torch_dtype, device=DEV) for _ in range(wl.num_workers)]
    wl.fill_replicas(th, reps, u, t)
    return th, torch.zeros_like(th), reps


@pytest.mark.parametrize("one_pass", [False, True])
@pytest.mark.parametrize("K,dtype", [(8, "bf16"), (4, "f32"), (16, "bf16"), (32, "bf16")])
def test_host_round_matches_resident_round(K, dtype, one_pass):
    """Six units of mixed sizes (more than the three staging slots) in a
    non-index order, three rounds: theta, b, replicas and records equal the
    resident round's bit for bit."""
    sizes = [1_000_000, 2048, 7, 3_000_017, 0, 65_536 + 3]
    wl = synth.small("llama1b-k8-bf16", sizes, num_workers=K, replica_dtype=dtype, name=f"host{K}{dtype}")
    order = [2, 0, 5, 1, 4, 3]
    flags = {"flags": ONE_PASS} if one_pass else {}
    dev_h = EditOuter(OuterConfig(K, wl.layer_numel, dtype, **flags), DEV)
    host_h = EditOuter(OuterConfig(K, wl.layer_numel, dtype, **flags), DEV)
    dev_units = [_inputs(wl, u, 0) for u in range(wl.num_units)]
    host_units = []
    for th, b, reps in dev_units:
        th_h = torch.empty(th.numel(), dtype=torch.float32, pin_memory=True)
        b_h = torch.empty(th.numel(), dtype=torch.float32, pin_memory=True)
        th_h.copy_(th)
        b_h.copy_(b)
        host_units.append((th_h, b_h, [r.clone() for r in reps]))
    try:
        dev_plan = dev_h.prepare_round([dev_units[u] for u in order], layers=order)
        host_plan = host_h.prepare_round([host_units[u] for u in order], layers=order, host=True)
        for t in range(3):
            if t:
                for u in range(wl.num_units):
                    wl.fill_replicas(dev_units[u][0], dev_units[u][2], u, t)
                    for a, b in zip(dev_units[u][2], host_units[u][2]):
                        b.copy_(a)
            torch.cuda.synchronize()
            dev_plan.run()
            host_plan.run()
            torch.cuda.synchronize()
            for u in range(wl.num_units):
                (td, bd, rd), (th_, bh, rh) = dev_units[u], host_units[u]
                assert torch.equal(td.cpu(), th_), f"round {t} unit {u}: theta differs"
                assert torch.equal(bd.cpu(), bh), f"round {t} unit {u}: momentum differs"
                assert all(torch.equal(x, y) for x, y in zip(rd, rh)), f"round {t} unit {u}: replicas"
                sa, sb = dev_h.state_get(u), host_h.state_get(u)
                assert np.array_equal(sa.norm, sb.norm) and sa.synced_norm == sb.synced_norm
                assert np.array_equal(sa.anomalous, sb.anomalous) and sa.round == sb.round == t + 1
    finally:
        dev_h.close()
        host_h.close()


def test_host_round_matches_oracle():
    """Two units, three rounds against the oracle: two warm-up rounds, then,
    from a preset post-warm-up EMA state on both sides, a round in which
    worker 1 is x40 and must be masked while the others pass.  Each round
    both sides start from the oracle's theta and b (byte-identical inputs)."""
    wl = synth.small("llama1b-k8-bf16", [300_001, 4099], num_workers=5, replica_dtype="bf16",
                     clip_threshold=0.2, name="hostpar")
    K, W = wl.num_workers, wl.warmup_rounds
    lib = EditOuter(OuterConfig(K, wl.layer_numel, "bf16", ema_warmup_rounds=W, clip_threshold=0.2), DEV)
    oracles = [OracleUnit(K, OracleConfig(**wl.hyper())) for _ in range(2)]
    th_h = [wl.init_theta(u, DEV).cpu().pin_memory() for u in range(2)]
    b_h = [torch.zeros(wl.unit_numel(u), dtype=torch.float32).pin_memory() for u in range(2)]
    o_th = [t.numpy().copy() for t in th_h]
    o_b = [np.zeros(wl.unit_numel(u), np.float32) for u in range(2)]
    reps = [[torch.empty(wl.unit_numel(u), dtype=torch.bfloat16, device=DEV) for _ in range(K)]
            for u in range(2)]
    try:
        plan = lib.prepare_round([(th_h[u], b_h[u], reps[u]) for u in range(2)], host=True)
        for t in (0, 1, W):
            std = wl.worker_std(t) * (np.where(np.arange(K) == 1, 40.0, 1.0) if t == W else 1.0)
            reps_h = []
            for u in range(2):
                if t == W:
                    G0 = wl.delta_std * np.sqrt(wl.unit_numel(u))
                    ema = (np.full(K, 1.25 * G0), np.full(K, 0.45 * G0), W)
                    oracles[u].set_state(*ema)
                    lib.state_set(u, *ema)
                th_h[u].copy_(torch.from_numpy(o_th[u]))
                b_h[u].copy_(torch.from_numpy(o_b[u]))
                wl.fill_replicas(th_h[u].to(DEV), reps[u], u, t, std=std)
                reps_h.append([host_bits(r) for r in reps[u]])
            torch.cuda.synchronize()
            plan.run()
            recs = [oracles[u].step(o_th[u], o_b[u], reps_h[u]) for u in range(2)]
            torch.cuda.synchronize()
            for u in range(2):
                what = f"host round {t} unit {u}"
                compare_decision(lib.state_get(u), recs[u], K, what)
                assert_tensor_close(th_h[u].numpy(), o_th[u], what + ": theta")
                assert_tensor_close(b_h[u].numpy(), o_b[u], what + ": momentum")
            if t == W:
                assert [list(r["anomalous"]) for r in recs] == [[0, 1, 0, 0, 0]] * 2
    finally:
        lib.close()


def test_host_round_rejects_pageable_memory():
    """The copies are asynchronous, so theta and b must be page-locked; the
    library checks this itself (here called without the binding's checks)."""
    wl = synth.small("llama1b-k8-bf16", [4096], num_workers=2, replica_dtype="f32", name="hostbad")
    h = EditOuter(OuterConfig(2, wl.layer_numel, "f32"), DEV)
    try:
        th = np.zeros(4096, np.float32)
        b = np.zeros(4096, np.float32)
        reps = [torch.zeros(4096, device=DEV) for _ in range(2)]
        lib = h._lib
        layers = (ctypes.c_int32 * 1)(0)
        tp = (ctypes.c_void_p * 1)(th.ctypes.data)
        bp = (ctypes.c_void_p * 1)(b.ctypes.data)
        rp = (ctypes.c_void_p * 2)(*[r.data_ptr() for r in reps])
        rc = lib.edit_outer_step_round_host(h._h, 1, layers, tp, bp, rp, None)
        assert rc == -1 and b"pinned" in lib.edit_outer_last_error()
        with pytest.raises(ValueError, match="pinned"):
            h.prepare_round([(torch.zeros(4096), torch.zeros(4096), reps)], host=True)
    finally:
        h.close()
