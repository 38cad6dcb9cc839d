"""Python binding of libedit_outer.so (argument marshalling only).

Every step of the outer synchronization runs in the HIP kernels of the
library; this module checks tensors, passes device pointers and HIP stream
handles through the C ABI of include/edit_outer.h, and converts results.
PyTorch provides the device memory and the streams.  There is no fallback:
if the library is missing or fails to load, EditOuterError is raised.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(PKG, "libedit_outer.so")

MAX_K = 32
AE, WA, GC = 1, 2, 4
ONE_PASS = 8  # single-pass mean step; only with AE, WA and GC clear
F32, BF16 = 0, 1

EDIT_OK, EDIT_EINVAL, EDIT_ENOMEM, EDIT_EHIP, EDIT_ESTATE, EDIT_ENODEV = 0, -1, -2, -3, -4, -5

# Every function the header declares; the CPU tests check the library exports them.
EXPORTS = (
    "edit_outer_init", "edit_outer_min_warmup", "edit_outer_step_layer", "edit_outer_step_layer_noalloc",
    "edit_outer_step_round",
    "edit_outer_step_round_host", "edit_outer_gram_layer", "edit_outer_apply_layer",
    "edit_outer_state_get", "edit_outer_state_set",
    "edit_outer_destroy", "edit_outer_strerror", "edit_outer_last_error",
    "edit_outer_set_profiling", "edit_outer_kernel_times", "edit_outer_update_probe", "edit_outer_copy_probe",
    "edit_group_init", "edit_group_norm", "edit_group_weights", "edit_group_apply",
    "edit_group_state_get", "edit_group_state_set", "edit_group_destroy",
)


class EditOuterError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


class _Config(ctypes.Structure):
    _fields_ = [
        ("num_workers", ctypes.c_int32),
        ("num_layers", ctypes.c_int32),
        ("layer_numel", ctypes.POINTER(ctypes.c_int64)),
        ("replica_dtype", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
        ("outer_lr", ctypes.c_double),
        ("momentum", ctypes.c_double),
        ("clip_threshold", ctypes.c_double),
        ("clip_eps", ctypes.c_double),
        ("ema_alpha", ctypes.c_double),
        ("z_threshold", ctypes.c_double),
        ("ema_warmup_rounds", ctypes.c_int64),
    ]


class _LayerState(ctypes.Structure):
    _fields_ = [
        ("round", ctypes.c_int64),
        ("num_workers", ctypes.c_int32),
        ("rolled_back", ctypes.c_int32),
        ("z_tested", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("ema_mean", ctypes.c_double * MAX_K),
        ("ema_std", ctypes.c_double * MAX_K),
        ("norm", ctypes.c_double * MAX_K),
        ("weight", ctypes.c_double * MAX_K),
        ("anomalous", ctypes.c_uint8 * MAX_K),
        ("synced_norm", ctypes.c_double),
        ("clip_coef", ctypes.c_double),
    ]


_lib = None


def load_library() -> ctypes.CDLL:
    """Load the in-tree library (built by `python -m paper_2412_07210_amd.build`)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIBRARY):
        raise EditOuterError(EDIT_ENODEV, f"{LIBRARY} is not built; run "
                             "`python -m paper_2412_07210_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIBRARY)
    st = ctypes.c_int
    vp = ctypes.c_void_p
    lib.edit_outer_init.argtypes = [ctypes.POINTER(_Config), ctypes.POINTER(vp)]
    lib.edit_outer_init.restype = st
    lib.edit_outer_min_warmup.argtypes = [ctypes.c_double, ctypes.c_double]
    lib.edit_outer_min_warmup.restype = ctypes.c_int64
    lib.edit_outer_step_layer.argtypes = [vp, ctypes.c_int32, vp, vp, ctypes.POINTER(vp), vp]
    lib.edit_outer_step_layer.restype = st
    lib.edit_outer_step_layer_noalloc.argtypes = [vp, ctypes.c_int32, vp, vp, ctypes.POINTER(vp), vp]
    lib.edit_outer_step_layer_noalloc.restype = st
    lib.edit_outer_step_round.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                          ctypes.POINTER(vp), ctypes.POINTER(vp),
                                          ctypes.POINTER(vp), vp]
    lib.edit_outer_step_round.restype = st
    lib.edit_outer_step_round_host.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                               ctypes.POINTER(vp), ctypes.POINTER(vp),
                                               ctypes.POINTER(vp), vp]
    lib.edit_outer_step_round_host.restype = st
    lib.edit_outer_gram_layer.argtypes = [vp, ctypes.c_int32, vp, ctypes.POINTER(vp), vp, vp]
    lib.edit_outer_gram_layer.restype = st
    lib.edit_outer_apply_layer.argtypes = [vp, ctypes.c_int32, vp, vp, vp, ctypes.POINTER(vp), vp]
    lib.edit_outer_apply_layer.restype = st
    lib.edit_outer_state_get.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(_LayerState)]
    lib.edit_outer_state_get.restype = st
    lib.edit_outer_state_set.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(_LayerState)]
    lib.edit_outer_state_set.restype = st
    lib.edit_outer_destroy.argtypes = [vp]
    lib.edit_outer_destroy.restype = None
    lib.edit_outer_strerror.argtypes = [st]
    lib.edit_outer_strerror.restype = ctypes.c_char_p
    lib.edit_outer_last_error.argtypes = []
    lib.edit_outer_last_error.restype = ctypes.c_char_p
    lib.edit_outer_set_profiling.argtypes = [vp, ctypes.c_int32]
    lib.edit_outer_set_profiling.restype = st
    lib.edit_outer_kernel_times.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(ctypes.c_float)]
    lib.edit_outer_kernel_times.restype = st
    lib.edit_outer_update_probe.argtypes = [vp, ctypes.c_int32, vp, vp, ctypes.POINTER(vp), vp]
    lib.edit_outer_update_probe.restype = st
    lib.edit_outer_copy_probe.argtypes = [vp, vp, ctypes.c_int64, vp]
    lib.edit_outer_copy_probe.restype = st
    lib.edit_group_init.argtypes = [ctypes.POINTER(_Config), ctypes.c_int32, ctypes.POINTER(vp)]
    lib.edit_group_init.restype = st
    lib.edit_group_norm.argtypes = [vp, ctypes.c_int32, vp, vp, vp, vp, vp]
    lib.edit_group_norm.restype = st
    lib.edit_group_weights.argtypes = [vp, ctypes.c_int32, vp, vp, vp, vp]
    lib.edit_group_weights.restype = st
    lib.edit_group_apply.argtypes = [vp, ctypes.c_int32, vp, vp, vp, vp, vp]
    lib.edit_group_apply.restype = st
    lib.edit_group_state_get.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(_LayerState)]
    lib.edit_group_state_get.restype = st
    lib.edit_group_state_set.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(_LayerState)]
    lib.edit_group_state_set.restype = st
    lib.edit_group_destroy.argtypes = [vp]
    lib.edit_group_destroy.restype = None
    _lib = lib
    return lib


def _check(status: int, what: str) -> None:
    if status != EDIT_OK:
        lib = load_library()
        msg = lib.edit_outer_last_error().decode(errors="replace")
        name = lib.edit_outer_strerror(status).decode()
        raise EditOuterError(status, f"{what}: {name}: {msg}")


def min_warmup(ema_alpha: float = 0.02, z_threshold: float = 3.0) -> int:
    """Shortest EMA warm-up (rounds) the library accepts with anomaly
    elimination on (edit_outer_min_warmup; -1 if none does)."""
    return int(load_library().edit_outer_min_warmup(float(ema_alpha), float(z_threshold)))


def _stream_handle(stream: Optional[torch.cuda.Stream], device: torch.device) -> int:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return int(s.cuda_stream)


@dataclass
class OuterConfig:
    """Configuration of one handle; names follow the paper's notation."""
    num_workers: int                       # K
    layer_numel: Sequence[int]             # elements of each sync unit
    replica_dtype: str = "bf16"            # "bf16" or "f32"
    outer_lr: float = 0.8                  # nu
    momentum: float = 0.85                 # rho
    clip_threshold: float = 10.0           # phi (Eq. 4)
    clip_eps: float = 1e-6                 # eps (Eq. 4)
    ema_alpha: float = 0.02                # alpha (Eq. 1)
    z_threshold: float = 3.0               # delta
    ema_warmup_rounds: int = 10
    flags: int = AE | WA | GC

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.replica_dtype == "bf16" else torch.float32


def _c_config(cfg: OuterConfig, numel: List[int]):
    """The C configuration (and the element-count array it points to, which
    must stay alive until the init call returns)."""
    arr = (ctypes.c_int64 * len(numel))(*numel)
    c = _Config(int(cfg.num_workers), len(numel), arr,
                BF16 if cfg.replica_dtype == "bf16" else F32, int(cfg.flags),
                float(cfg.outer_lr), float(cfg.momentum), float(cfg.clip_threshold),
                float(cfg.clip_eps), float(cfg.ema_alpha), float(cfg.z_threshold),
                int(cfg.ema_warmup_rounds))
    return c, arr


def _layer_state(st: "_LayerState", K: int) -> "LayerState":
    return LayerState(
        round=int(st.round), rolled_back=bool(st.rolled_back), z_tested=bool(st.z_tested),
        ema_mean=np.array(st.ema_mean[:K]), ema_std=np.array(st.ema_std[:K]),
        norm=np.array(st.norm[:K]), weight=np.array(st.weight[:K]),
        anomalous=np.array(st.anomalous[:K], dtype=np.uint8),
        synced_norm=float(st.synced_norm), clip_coef=float(st.clip_coef))


@dataclass
class LayerState:
    round: int
    rolled_back: bool
    z_tested: bool
    ema_mean: np.ndarray
    ema_std: np.ndarray
    norm: np.ndarray
    weight: np.ndarray
    anomalous: np.ndarray
    synced_norm: float
    clip_coef: float


class EditOuter:
    """A handle of the C library: EMA state and scratch for L sync units."""

    def __init__(self, cfg: OuterConfig, device: Optional[torch.device] = None):
        self.cfg = cfg
        device = torch.device("cuda") if device is None else torch.device(device)
        if device.type != "cuda":
            raise ValueError("the handle needs a GPU device")
        if device.index is None:
            device = torch.device("cuda", torch.cuda.current_device())
        self.device = device
        if cfg.replica_dtype not in ("bf16", "f32"):
            raise ValueError("replica_dtype must be 'bf16' or 'f32'")
        lib = load_library()
        self._numel = [int(n) for n in cfg.layer_numel]
        c, arr = _c_config(cfg, self._numel)
        h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(lib.edit_outer_init(ctypes.byref(c), ctypes.byref(h)), "edit_outer_init")
        self._h = h
        self._lib = lib

    # -- lifetime ------------------------------------------------------------
    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            with torch.cuda.device(self.device):
                self._lib.edit_outer_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- the step --------------------------------------------------------------
    def _check_tensor(self, t: torch.Tensor, n: int, dtype: torch.dtype, what: str) -> None:
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{what} must be a torch.Tensor")
        if t.device != self.device:
            raise ValueError(f"{what} is on {t.device}, the handle on {self.device}")
        if t.dtype != dtype:
            raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{what} must be contiguous")
        if t.numel() != n:
            raise ValueError(f"{what} has {t.numel()} elements, unit has {n}")

    def step_layer(self, layer: int, theta: torch.Tensor, momentum: torch.Tensor,
                   replicas: Sequence[torch.Tensor], stream: Optional[torch.cuda.Stream] = None) -> None:
        """Enqueue one outer step of unit `layer` (in place on all tensors)."""
        if not 0 <= layer < len(self._numel):
            raise IndexError(f"layer {layer} out of range")
        n = self._numel[layer]
        K = self.cfg.num_workers
        if len(replicas) != K:
            raise ValueError(f"expected {K} replicas, got {len(replicas)}")
        self._check_tensor(theta, n, torch.float32, "theta")
        self._check_tensor(momentum, n, torch.float32, "momentum")
        for j, r in enumerate(replicas):
            self._check_tensor(r, n, self.cfg.torch_dtype, f"replicas[{j}]")
        ptrs = (ctypes.c_void_p * K)(*[r.data_ptr() for r in replicas])
        if torch.cuda.current_device() != self.device.index:
            with torch.cuda.device(self.device):
                status = self._lib.edit_outer_step_layer(self._h, int(layer), theta.data_ptr(),
                                                         momentum.data_ptr(), ptrs,
                                                         _stream_handle(stream, self.device))
        else:
            status = self._lib.edit_outer_step_layer(self._h, int(layer), theta.data_ptr(),
                                                     momentum.data_ptr(), ptrs,
                                                     _stream_handle(stream, self.device))
        _check(status, "edit_outer_step_layer")

    @property
    def num_pairs(self) -> int:
        """Length of a Gram vector: K(K+1)/2."""
        K = self.cfg.num_workers
        return K * (K + 1) // 2

    def _call(self, fn, *args) -> int:
        if torch.cuda.current_device() != self.device.index:
            with torch.cuda.device(self.device):
                return fn(self._h, *args)
        return fn(self._h, *args)

    def _unit_tensors(self, layer: int, theta, momentum, replicas):
        if not 0 <= layer < len(self._numel):
            raise IndexError(f"layer {layer} out of range")
        n = self._numel[layer]
        K = self.cfg.num_workers
        if len(replicas) != K:
            raise ValueError(f"expected {K} replicas, got {len(replicas)}")
        self._check_tensor(theta, n, torch.float32, "theta")
        if momentum is not None:
            self._check_tensor(momentum, n, torch.float32, "momentum")
        for j, r in enumerate(replicas):
            self._check_tensor(r, n, self.cfg.torch_dtype, f"replicas[{j}]")
        return (ctypes.c_void_p * K)(*[r.data_ptr() for r in replicas])

    def gram_layer(self, layer: int, theta: torch.Tensor, replicas: Sequence[torch.Tensor],
                   gram: Optional[torch.Tensor] = None,
                   stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        """Enqueue pass 1 of unit `layer` and return its Gram vector (fp64,
        K(K+1)/2 upper-triangle sums, row by row) on the device.  For a module
        sharded over several units, add the shards' vectors and hand the sum
        to apply_layer of every shard."""
        ptrs = self._unit_tensors(layer, theta, None, replicas)
        if gram is None:
            gram = torch.empty(self.num_pairs, dtype=torch.float64, device=self.device)
        self._check_tensor(gram, self.num_pairs, torch.float64, "gram")
        _check(self._call(self._lib.edit_outer_gram_layer, int(layer), theta.data_ptr(), ptrs,
                          gram.data_ptr(), _stream_handle(stream, self.device)),
               "edit_outer_gram_layer")
        return gram

    def apply_layer(self, layer: int, gram: torch.Tensor, theta: torch.Tensor,
                    momentum: torch.Tensor, replicas: Sequence[torch.Tensor],
                    stream: Optional[torch.cuda.Stream] = None) -> None:
        """Enqueue the decision from `gram` and the update pass of unit `layer`."""
        ptrs = self._unit_tensors(layer, theta, momentum, replicas)
        self._check_tensor(gram, self.num_pairs, torch.float64, "gram")
        _check(self._call(self._lib.edit_outer_apply_layer, int(layer), gram.data_ptr(),
                          theta.data_ptr(), momentum.data_ptr(), ptrs,
                          _stream_handle(stream, self.device)),
               "edit_outer_apply_layer")

    def prepare_round(self, units: Sequence[tuple], layers: Optional[Sequence[int]] = None,
                      host: bool = False) -> "RoundPlan":
        """Validate a round's tensors once; RoundPlan.run() then enqueues it
        with a single edit_outer_step_round call (no per-tensor Python work).
        host=True: theta and momentum of every unit are pinned CPU tensors,
        stepped through edit_outer_step_round_host; synchronise the stream
        before reading them."""
        return RoundPlan(self, units, layers, host)

    def step_round(self, units: Sequence[tuple], streams: Optional[List[torch.cuda.Stream]] = None,
                   layers: Optional[Sequence[int]] = None) -> None:
        """Step every unit in forward order.

        units[i] = (theta, momentum, replicas) of unit layers[i] (default i).
        Without `streams` this is one edit_outer_step_round call on the
        current stream.  With streams, unit i goes to streams[i % S] through
        edit_outer_step_layer; the streams start after the current stream's
        pending work and the current stream waits for all of them.
        """
        layers = list(range(len(units))) if layers is None else list(layers)
        if not streams:
            RoundPlan(self, units, layers).run()
            return
        if len(layers) != len(units):
            raise ValueError("layers and units differ in length")
        cur = torch.cuda.current_stream(self.device)
        start = torch.cuda.Event()
        start.record(cur)
        for s in streams:
            s.wait_event(start)
        for i, (l, (th, b, reps)) in enumerate(zip(layers, units)):
            self.step_layer(l, th, b, reps, stream=streams[i % len(streams)])
        for s in streams:
            ev = torch.cuda.Event()
            ev.record(s)
            cur.wait_event(ev)

    # -- state ----------------------------------------------------------------
    def state_get(self, layer: int) -> LayerState:
        st = _LayerState()
        with torch.cuda.device(self.device):
            _check(self._lib.edit_outer_state_get(self._h, int(layer), ctypes.byref(st)),
                   "edit_outer_state_get")
        return _layer_state(st, self.cfg.num_workers)

    def state_set(self, layer: int, ema_mean: Sequence[float], ema_std: Sequence[float],
                  round_: int) -> None:
        st = _LayerState()
        st.round = int(round_)
        st.num_workers = self.cfg.num_workers
        for j in range(self.cfg.num_workers):
            st.ema_mean[j] = float(ema_mean[j])
            st.ema_std[j] = float(ema_std[j])
        with torch.cuda.device(self.device):
            _check(self._lib.edit_outer_state_set(self._h, int(layer), ctypes.byref(st)),
                   "edit_outer_state_set")

    # -- measurement ------------------------------------------------------------
    def set_profiling(self, every: int) -> None:
        """Record kernel events on units l with l % every == 0 (0: off)."""
        _check(self._lib.edit_outer_set_profiling(self._h, int(every)), "set_profiling")

    def update_probe(self, layer: int, theta: torch.Tensor, momentum: torch.Tensor,
                     replicas: Sequence[torch.Tensor], stream: Optional[torch.cuda.Stream] = None) -> None:
        """Enqueue unit `layer`'s update-pass traffic with no arithmetic (the
        tensors are read and written back unchanged)."""
        ptrs = self._unit_tensors(layer, theta, momentum, replicas)
        _check(self._call(self._lib.edit_outer_update_probe, int(layer), theta.data_ptr(), momentum.data_ptr(),
                          ptrs, _stream_handle(stream, self.device)), "edit_outer_update_probe")

    def kernel_times(self, layer: int) -> tuple:
        """(pass-1 ms incl. the decision, pass-2 ms) of the unit's last profiled step."""
        ms = (ctypes.c_float * 2)()
        with torch.cuda.device(self.device):
            _check(self._lib.edit_outer_kernel_times(self._h, int(layer), ms), "kernel_times")
        return float(ms[0]), float(ms[1])


class RoundPlan:
    """A validated round: the units' tensors checked once, their device
    pointers marshalled once.  The plan keeps the tensors alive; their storage
    must not be reallocated while the plan is used."""

    def __init__(self, handle: EditOuter, units: Sequence[tuple],
                 layers: Optional[Sequence[int]] = None, host: bool = False):
        layers = list(range(len(units))) if layers is None else list(layers)
        self._host = host
        if len(layers) != len(units) or not units:
            raise ValueError("need one layer index per unit and at least one unit")
        K = handle.cfg.num_workers
        c = len(units)
        self._handle = handle
        self._units = list(units)
        self._count = c
        self._layers = (ctypes.c_int32 * c)(*layers)
        self._theta = (ctypes.c_void_p * c)()
        self._mom = (ctypes.c_void_p * c)()
        self._reps = (ctypes.c_void_p * (c * K))()
        for i, (l, (t, b, reps)) in enumerate(zip(layers, units)):
            if not 0 <= l < len(handle._numel):
                raise IndexError(f"layer {l} out of range")
            n = handle._numel[l]
            if len(reps) != K:
                raise ValueError(f"expected {K} replicas, got {len(reps)}")
            if host:  # theta and momentum in page-locked host memory
                for x, what in ((t, "theta"), (b, "momentum")):
                    if not isinstance(x, torch.Tensor) or x.device.type != "cpu":
                        raise ValueError(f"{what} must be a CPU tensor for a host round")
                    if x.dtype != torch.float32 or not x.is_contiguous() or x.numel() != n:
                        raise ValueError(f"{what} must be contiguous float32 with {n} elements")
                    if n and not x.is_pinned():
                        raise ValueError(f"{what} must be pinned (torch.empty(..., pin_memory=True))")
            else:
                handle._check_tensor(t, n, torch.float32, "theta")
                handle._check_tensor(b, n, torch.float32, "momentum")
            for j, r in enumerate(reps):
                handle._check_tensor(r, n, handle.cfg.torch_dtype, f"replicas[{j}]")
                self._reps[i * K + j] = r.data_ptr()
            self._theta[i], self._mom[i] = t.data_ptr(), b.data_ptr()

    def run(self, stream: Optional[torch.cuda.Stream] = None) -> None:
        h = self._handle
        s = _stream_handle(stream, h.device)
        name = "edit_outer_step_round_host" if self._host else "edit_outer_step_round"
        fn = getattr(h._lib, name)
        _check(h._call(fn, self._count, self._layers, self._theta, self._mom, self._reps, s), name)


class SyncGroupWorker:
    """One worker (rank) of a sync group whose K replicas sit on K GPUs: its
    share of the Sync() procedure on its own GPU (edit_group_* of the C ABI).
    The all-gather of the norm pairs and the all-reduce of w_j * Delta_j
    between the three calls are the caller's collectives."""

    def __init__(self, cfg: OuterConfig, rank: int, device: Optional[torch.device] = None):
        self.cfg = cfg
        self.rank = int(rank)
        device = torch.device("cuda") if device is None else torch.device(device)
        if device.type != "cuda":
            raise ValueError("the handle needs a GPU device")
        if device.index is None:
            device = torch.device("cuda", torch.cuda.current_device())
        self.device = device
        if cfg.replica_dtype not in ("bf16", "f32"):
            raise ValueError("replica_dtype must be 'bf16' or 'f32'")
        lib = load_library()
        self._numel = [int(n) for n in cfg.layer_numel]
        c, arr = _c_config(cfg, self._numel)
        h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(lib.edit_group_init(ctypes.byref(c), self.rank, ctypes.byref(h)), "edit_group_init")
        self._h = h
        self._lib = lib

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            with torch.cuda.device(self.device):
                self._lib.edit_group_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _arg(self, t: torch.Tensor, n: int, dtype: torch.dtype, what: str) -> int:
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{what} must be a torch.Tensor")
        if t.device != self.device or t.dtype != dtype or not t.is_contiguous() or t.numel() != n:
            raise ValueError(f"{what} must be a contiguous {dtype} tensor of {n} elements on {self.device}")
        return t.data_ptr()

    def _n(self, layer: int) -> int:
        if not 0 <= layer < len(self._numel):
            raise IndexError(f"layer {layer} out of range")
        return self._numel[layer]

    def _call(self, fn, what: str, *args) -> None:
        with torch.cuda.device(self.device):
            _check(fn(self._h, *args), what)

    def norm(self, layer: int, theta: torch.Tensor, replica: torch.Tensor, delta: torch.Tensor,
             norm_out: Optional[torch.Tensor] = None,
             stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        """Enqueue the norm pass; returns norm_out = [G_rank, flag] (fp64,
        device), this rank's part of the all-gather.  delta receives Delta_rank (fp32)."""
        n = self._n(layer)
        if norm_out is None:
            norm_out = torch.empty(2, dtype=torch.float64, device=self.device)
        self._call(self._lib.edit_group_norm, "edit_group_norm", int(layer),
                   self._arg(theta, n, torch.float32, "theta"),
                   self._arg(replica, n, self.cfg.torch_dtype, "replica"),
                   self._arg(delta, n, torch.float32, "delta"),
                   self._arg(norm_out, 2, torch.float64, "norm_out"), _stream_handle(stream, self.device))
        return norm_out

    def weights(self, layer: int, gathered: torch.Tensor, delta: torch.Tensor,
                weight_out: Optional[torch.Tensor] = None,
                stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        """Enqueue the group decision from the gathered [K, 2] pairs; returns
        weight_out = [w_rank] (fp64, device).  delta is cleared if this rank is flagged."""
        n = self._n(layer)
        K = self.cfg.num_workers
        if weight_out is None:
            weight_out = torch.empty(1, dtype=torch.float64, device=self.device)
        self._call(self._lib.edit_group_weights, "edit_group_weights", int(layer),
                   self._arg(gathered, 2 * K, torch.float64, "gathered"),
                   self._arg(weight_out, 1, torch.float64, "weight_out"),
                   self._arg(delta, n, torch.float32, "delta"), _stream_handle(stream, self.device))
        return weight_out

    def apply(self, layer: int, dbar: torch.Tensor, theta: torch.Tensor, momentum: torch.Tensor,
              replica: torch.Tensor, stream: Optional[torch.cuda.Stream] = None) -> None:
        """Enqueue the clip and the update from the all-reduced dbar (in place
        on theta, momentum and the replica)."""
        n = self._n(layer)
        self._call(self._lib.edit_group_apply, "edit_group_apply", int(layer),
                   self._arg(dbar, n, torch.float32, "dbar"),
                   self._arg(theta, n, torch.float32, "theta"),
                   self._arg(momentum, n, torch.float32, "momentum"),
                   self._arg(replica, n, self.cfg.torch_dtype, "replica"), _stream_handle(stream, self.device))

    def state_get(self, layer: int) -> LayerState:
        st = _LayerState()
        self._call(self._lib.edit_group_state_get, "edit_group_state_get", int(layer), ctypes.byref(st))
        return _layer_state(st, self.cfg.num_workers)

    def state_set(self, layer: int, ema_mean: float, ema_std: float, round_: int) -> None:
        """This worker's EMA pair and the round counter of unit `layer`."""
        st = _LayerState()
        st.round = int(round_)
        st.num_workers = self.cfg.num_workers
        st.ema_mean[self.rank] = float(ema_mean)
        st.ema_std[self.rank] = float(ema_std)
        self._call(self._lib.edit_group_state_set, "edit_group_state_set", int(layer), ctypes.byref(st))


def copy_probe(dst: torch.Tensor, src: torch.Tensor, stream: Optional[torch.cuda.Stream] = None) -> None:
    """Plain device copy kernel of the library (bandwidth / counter calibration)."""
    if dst.device != src.device or dst.device.type != "cuda":
        raise ValueError("dst and src must be on the same GPU")
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("dst and src sizes differ")
    lib = load_library()
    _check(lib.edit_outer_copy_probe(dst.data_ptr(), src.data_ptr(), nbytes,
                                     _stream_handle(stream, dst.device)), "edit_outer_copy_probe")
