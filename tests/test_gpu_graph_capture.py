"""The no-allocation step captured in a HIP graph and replayed (GPU).

edit_outer_step_layer_noalloc allocates nothing and synchronises nothing, so
a caller can capture it (here with torch.cuda.graph on a side stream) and
replay it.  One handle replays the captured step on fixed tensors; a second
handle with the same units and EMA state steps the same inputs eagerly with
edit_outer_step_layer.  Between replays the program does its own eager work
(new replicas, the eager step) and synchronises, and after every replay
theta, b, every replica and the decision record (Sec. 3.2, Eq. 1-5) must
equal the eager step's bit for bit: the same kernels reduce the same partial
sums in the same order.  The replays start from a settled EMA state after
the warm-up; the third has a x40 worker, so the z-test and the masked
average run inside the graph.
"""
import ctypes

import numpy as np
import pytest
import torch

from parity import steady_ema
from paper_2412_07210_amd import EditOuter, OuterConfig, synth
from paper_2412_07210_amd.outer import EDIT_OK

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _noalloc(h, layer, theta, mom, reps):
    """edit_outer_step_layer_noalloc through the C ABI, on the current stream."""
    ptrs = (ctypes.c_void_p * len(reps))(*[r.data_ptr() for r in reps])
    stream = torch.cuda.current_stream(DEV).cuda_stream
    rc = h._lib.edit_outer_step_layer_noalloc(h._h, layer, theta.data_ptr(), mom.data_ptr(), ptrs, stream)
    return rc, h._lib.edit_outer_last_error().decode()


def _fields(st):
    return (st.round, st.rolled_back, st.z_tested, st.anomalous.tolist(), st.norm.tolist(),
            st.ema_mean.tolist(), st.ema_std.tolist(), st.weight.tolist(), st.synced_norm, st.clip_coef)


@pytest.mark.parametrize("K,dtype,n", [(8, "bf16", 1_000_003), (16, "bf16", 700_001), (5, "f32", 300_007)])
def test_captured_noalloc_step_replays_like_eager_steps(K, dtype, n):
    wl = synth.small("llama1b-k8-bf16", [n], num_workers=K, replica_dtype=dtype, name=f"graph{K}{dtype}")
    W = wl.warmup_rounds
    cfg = OuterConfig(K, wl.layer_numel, dtype, ema_warmup_rounds=W)
    print(f"graph case K={K} {dtype} n={n}", flush=True)
    a, b = EditOuter(cfg, DEV), EditOuter(cfg, DEV)  # a: captured step, b: eager steps
    try:
        for h in (a, b):
            h.state_set(0, *steady_ema(wl, n, W))
        th0 = wl.init_theta(0, DEV)
        tha, thb = th0.clone(), th0.clone()
        ba, bb = torch.zeros_like(th0), torch.zeros_like(th0)
        ra = [torch.empty(n, dtype=wl.torch_dtype, device=DEV) for _ in range(K)]
        rb = [torch.empty_like(r) for r in ra]
        torch.cuda.synchronize(DEV)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=torch.cuda.Stream(DEV)):
            rc, msg = _noalloc(a, 0, tha, ba, ra)
        assert rc == EDIT_OK, msg
        for t in range(W, W + 4):
            std = wl.worker_std(t) * (np.where(np.arange(K) == K - 1, 40.0, 1.0) if t == W + 2 else 1.0)
            wl.fill_replicas(tha, ra, 0, t, std=std)
            for x, y in zip(ra, rb):
                y.copy_(x)
            torch.cuda.synchronize(DEV)
            graph.replay()
            b.step_layer(0, thb, bb, rb)
            torch.cuda.synchronize(DEV)
            what = f"replay {t - W} (round {t})"
            assert torch.equal(tha, thb), what + ": theta"
            assert torch.equal(ba, bb), what + ": momentum"
            assert all(torch.equal(x, y) for x, y in zip(ra, rb)), what + ": replicas"
            sa, sb = a.state_get(0), b.state_get(0)
            assert _fields(sa) == _fields(sb), what + ": record"
            assert sb.round == t + 1 and sb.z_tested, what
            if t == W + 2:
                assert sa.anomalous[K - 1] == 1 and not sa.anomalous[:K - 1].any(), what + ": mask"
        del graph
    finally:
        a.close()
        b.close()
