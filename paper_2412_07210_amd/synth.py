"""Seeded synthetic workloads for the outer synchronization step.

This module only *makes inputs*: initial parameters and, for every outer
round, each worker's replica after its inner steps, modelled as
``cast(theta_t + s_j * N(0, 1))``.  It holds none of the outer step's own
arithmetic, so both the HIP path and the CPU oracle may consume its output.

The paper trains Llama models on FineWeb-Edu and an in-house corpus; neither
the data nor the weights are available, so seeded Gaussian layers with the
shapes of Llama decoder layers stand in for them (paper Sec. 4.1 and the
model table of the appendix list the model family and scales).
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, replace
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

# A segment of a flat unit: (name, number of elements, kind); kind is
# "matrix" (initialised N(0, 0.02)) or "norm" (RMSNorm gain, initialised 1).
Segment = Tuple[str, int, str]


def llama_layer_segments(hidden: int, ffn: int) -> List[Segment]:
    """One Llama decoder layer flattened in module order (SwiGLU FFN)."""
    return [
        ("attn.q", hidden * hidden, "matrix"),
        ("attn.k", hidden * hidden, "matrix"),
        ("attn.v", hidden * hidden, "matrix"),
        ("attn.o", hidden * hidden, "matrix"),
        ("mlp.gate", ffn * hidden, "matrix"),
        ("mlp.up", ffn * hidden, "matrix"),
        ("mlp.down", hidden * ffn, "matrix"),
        ("attn_norm", hidden, "norm"),
        ("ffn_norm", hidden, "norm"),
    ]


def _take_prefix(segments: Sequence[Segment], count: int) -> List[Segment]:
    out, left = [], count
    for name, n, kind in segments:
        if left <= 0:
            break
        take = min(n, left)
        out.append((name, take, kind))
        left -= take
    return out


def _seed(*parts) -> int:
    text = "/".join(str(p) for p in parts).encode()
    return int.from_bytes(hashlib.blake2b(text, digest_size=8).digest(), "little") & (2**63 - 1)


@dataclass(frozen=True)
class Workload:
    """Shapes, hyper-parameters and per-round noise recipe of one workload."""
    name: str
    description: str
    num_workers: int
    replica_dtype: str                      # "f32" or "bf16"
    units: Tuple[Tuple[Segment, ...], ...]  # per sync unit, its segments
    delta_std: float                        # base std of a worker's pseudo gradient
    scale_mode: str = "fixed"               # fixed | uniform_0.5_2 | aedit_steps
    # none | last_x50_from_round_10 | one_x20_every_10_rounds | three_x30_after_warmup
    anomaly_mode: str = "none"
    rounds: int = 10
    outer_lr: float = 0.8
    momentum: float = 0.85
    clip_threshold: float = 10.0
    clip_eps: float = 1e-6
    ema_alpha: float = 0.02
    z_threshold: float = 3.0
    warmup_rounds: int = 10
    theta_std: float = 0.02

    # -- shapes -------------------------------------------------------------
    @property
    def num_units(self) -> int:
        return len(self.units)

    def unit_numel(self, u: int) -> int:
        return sum(n for _, n, _ in self.units[u])

    @property
    def layer_numel(self) -> List[int]:
        return [self.unit_numel(u) for u in range(self.num_units)]

    @property
    def total_numel(self) -> int:
        return sum(self.layer_numel)

    @property
    def replica_bytes(self) -> int:
        return 4 if self.replica_dtype == "f32" else 2

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.replica_dtype == "f32" else torch.bfloat16

    def hyper(self) -> Dict[str, float]:
        return dict(outer_lr=self.outer_lr, momentum=self.momentum,
                    clip_threshold=self.clip_threshold, clip_eps=self.clip_eps,
                    ema_alpha=self.ema_alpha, z_threshold=self.z_threshold,
                    warmup_rounds=self.warmup_rounds)

    def with_units(self, units: Sequence[int]) -> "Workload":
        """The same workload restricted to a subset of its units."""
        return replace(self, units=tuple(self.units[u] for u in units))

    # -- per-round recipe ---------------------------------------------------
    def anomalies(self, round_: int, seed: int = 0) -> Dict[int, float]:
        """Workers whose pseudo gradient is scaled up this round: {worker: factor}."""
        K = self.num_workers
        if self.anomaly_mode == "last_x50_from_round_10":
            # Ten clean rounds seed the EMA state; then the last worker is x50.
            return {K - 1: 50.0} if round_ >= 10 else {}
        if self.anomaly_mode == "one_x20_every_10_rounds":
            # One seeded worker x20 in rounds 19, 29, ..., after the warm-up.
            if round_ >= 19 and round_ % 10 == 9:
                rng = np.random.default_rng(_seed(seed, self.name, round_, "anomaly"))
                return {int(rng.integers(K)): 20.0}
            return {}
        if self.anomaly_mode == "three_x30_after_warmup":
            # After the clean warm-up, three seeded workers are x30 every round.
            if round_ >= self.warmup_rounds:
                rng = np.random.default_rng(_seed(seed, self.name, round_, "anomaly"))
                return {int(j): 30.0 for j in rng.choice(K, size=3, replace=False)}
            return {}
        return {}

    def worker_std(self, round_: int, seed: int = 0) -> np.ndarray:
        """Per-worker std of this round's pseudo gradient (anomalies included)."""
        K = self.num_workers
        rng = np.random.default_rng(_seed(seed, self.name, round_, "scale"))
        if self.scale_mode == "fixed":
            std = np.full(K, self.delta_std)
        elif self.scale_mode == "uniform_0.5_2":
            std = self.delta_std * rng.uniform(0.5, 2.0, size=K)
        elif self.scale_mode == "aedit_steps":
            # A-EDiT: each worker runs as many local steps as fit its time
            # budget; the pseudo gradient's std grows like sqrt(steps).
            steps = rng.integers(8, 33, size=K)
            std = self.delta_std * np.sqrt(steps / 16.0)
        else:
            raise ValueError(self.scale_mode)
        for j, f in self.anomalies(round_, seed).items():
            std[j] *= f
        return std.astype(np.float64)

    # -- tensors --------------------------------------------------------------
    def init_theta(self, u: int, device, seed: int = 0) -> torch.Tensor:
        """theta_0 of unit u: matrices N(0, theta_std), RMSNorm gains 1."""
        n = self.unit_numel(u)
        out = torch.empty(n, dtype=torch.float32, device=device)
        gen = torch.Generator(device=out.device)
        off = 0
        for s, (name, m, kind) in enumerate(self.units[u]):
            view = out[off:off + m]
            if kind == "norm":
                view.fill_(1.0)
            else:
                gen.manual_seed(_seed(seed, self.name, "theta", u, s))
                view.normal_(0.0, self.theta_std, generator=gen)
            off += m
        return out

    def fill_replicas(self, theta: torch.Tensor, replicas: Sequence[torch.Tensor], u: int,
                      round_: int, seed: int = 0, std: Optional[np.ndarray] = None) -> None:
        """replicas[j] <- cast(theta + std_j * N(0, 1)), seeded per (round, unit, worker)."""
        if std is None:
            std = self.worker_std(round_, seed)
        gen = torch.Generator(device=theta.device)
        noise = torch.empty_like(theta)
        for j, r in enumerate(replicas):
            gen.manual_seed(_seed(seed, self.name, "delta", round_, u, j))
            noise.normal_(0.0, 1.0, generator=gen)
            noise.mul_(float(std[j])).add_(theta)
            r.copy_(noise)


def _repeat(seg: Sequence[Segment], times: int) -> Tuple[Tuple[Segment, ...], ...]:
    return tuple(tuple(seg) for _ in range(times))


def _aedit_units() -> Tuple[Tuple[Segment, ...], ...]:
    layer = llama_layer_segments(2048, 5632)
    units = []
    for _ in range(24):
        units.append(tuple(layer[:7]))   # the seven matrices of one layer
        units.append((layer[7],))        # attention RMSNorm gain (2048)
        units.append((layer[8],))        # FFN RMSNorm gain (2048)
    return tuple(units)


_HALF_7B = _take_prefix(llama_layer_segments(4096, 11008), 202_383_360 // 2)

WORKLOADS: Dict[str, Workload] = {
    "linear1m-k4": Workload(
        name="linear1m-k4",
        description="linear layer 1024x1024 fp32, K=4, worker 3 x50 after 10 clean rounds",
        num_workers=4, replica_dtype="f32",
        units=((("linear", 1024 * 1024, "matrix"),),),
        delta_std=1e-3, scale_mode="fixed", anomaly_mode="last_x50_from_round_10", rounds=11,
        outer_lr=0.7, momentum=0.9, clip_threshold=1.0),
    "llama350m-k8-f32": Workload(
        name="llama350m-k8-f32",
        description="Llama-style 350M: 24 layers, hidden 1024, FFN 2816, fp32 replicas, K=8",
        num_workers=8, replica_dtype="f32",
        units=_repeat(llama_layer_segments(1024, 2816), 24),
        delta_std=1e-3, scale_mode="uniform_0.5_2", rounds=30),
    "llama1b-k8-bf16": Workload(
        name="llama1b-k8-bf16",
        description="Llama-style 1B: 24 layers, hidden 2048, FFN 5632, bf16 replicas, K=8",
        num_workers=8, replica_dtype="bf16",
        units=_repeat(llama_layer_segments(2048, 5632), 24),
        delta_std=1e-3, scale_mode="uniform_0.5_2", anomaly_mode="one_x20_every_10_rounds", rounds=100),
    # The paper's own 1B model (its model-settings table): 32 layers, hidden
    # 1536, intermediate 4096, i.e. 28,314,624 parameters per layer.
    "paper1b-k8-bf16": Workload(
        name="paper1b-k8-bf16",
        description="the paper's Llama 1B: 32 layers, hidden 1536, FFN 4096, bf16 replicas, K=8",
        num_workers=8, replica_dtype="bf16",
        units=_repeat(llama_layer_segments(1536, 4096), 32),
        delta_std=1e-3, scale_mode="uniform_0.5_2", anomaly_mode="one_x20_every_10_rounds", rounds=100),
    "llama7b-half-k8-bf16": Workload(
        name="llama7b-half-k8-bf16",
        description="Llama-style 7B half shard: 32 layers x 101,191,680, bf16, K=8, clip active",
        num_workers=8, replica_dtype="bf16",
        units=_repeat(_HALF_7B, 32),
        delta_std=5e-4, scale_mode="fixed", rounds=20,
        clip_threshold=0.889),
    "aedit1b-k16-bf16": Workload(
        name="aedit1b-k16-bf16",
        description="A-EDiT round on 1B shapes: 72 units (matrices + two RMSNorm gains per layer), K=16",
        num_workers=16, replica_dtype="bf16",
        units=_aedit_units(),
        delta_std=1e-3, scale_mode="aedit_steps", anomaly_mode="three_x30_after_warmup", rounds=20),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]


def small(recipe: str, numel: Sequence[int], **overrides) -> Workload:
    """A workload with the recipe of `recipe` but custom (small) unit sizes."""
    base = WORKLOADS[recipe]
    units = tuple(((f"flat{i}", int(n), "matrix"),) for i, n in enumerate(numel))
    return replace(base, units=units, **overrides)
