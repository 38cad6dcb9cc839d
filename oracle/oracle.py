"""ctypes front end of the C oracle (test infrastructure only).

Inputs are numpy arrays in host memory: theta and momentum float32, the
replicas float32 or uint16 (bfloat16 bit patterns).  The step runs in place,
exactly like the C function it wraps.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field
from typing import List, Sequence

import numpy as np

from .build import LIBRARY, build_oracle

MAX_K = 64
AE, WA, GC = 1, 2, 4


class _Cfg(ctypes.Structure):
    _fields_ = [
        ("outer_lr", ctypes.c_double),
        ("momentum", ctypes.c_double),
        ("clip_threshold", ctypes.c_double),
        ("clip_eps", ctypes.c_double),
        ("ema_alpha", ctypes.c_double),
        ("z_threshold", ctypes.c_double),
        ("warmup_rounds", ctypes.c_int64),
        ("flags", ctypes.c_uint32),
    ]


class _Ema(ctypes.Structure):
    _fields_ = [
        ("mu", ctypes.c_double * MAX_K),
        ("sigma", ctypes.c_double * MAX_K),
        ("round", ctypes.c_int64),
    ]


class _Record(ctypes.Structure):
    _fields_ = [
        ("norm", ctypes.c_double * MAX_K),
        ("anomalous", ctypes.c_uint8 * MAX_K),
        ("weight", ctypes.c_double * MAX_K),
        ("margin", ctypes.c_double * MAX_K),
        ("synced_norm", ctypes.c_double),
        ("clip_coef", ctypes.c_double),
        ("rolled_back", ctypes.c_int32),
        ("z_tested", ctypes.c_int32),
    ]


_lib_handle = None


def library_path() -> str:
    return LIBRARY


def _lib():
    global _lib_handle
    if _lib_handle is None:
        # EDIT_ORACLE_LIBRARY points the tests at a deliberately broken build
        # (tests/test_oracle_mutants.py checks that the pins reject it)
        path = os.environ.get("EDIT_ORACLE_LIBRARY", LIBRARY)
        if path == LIBRARY and not os.path.exists(LIBRARY):
            build_oracle()
        lib = ctypes.CDLL(path)
        lib.oracle_step.restype = ctypes.c_int
        lib.oracle_step.argtypes = [
            ctypes.POINTER(_Cfg), ctypes.c_int, ctypes.c_int64, ctypes.c_int,
            ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p),
            ctypes.POINTER(_Ema), ctypes.POINTER(_Record),
        ]
        lib.oracle_decide_gram.restype = ctypes.c_int
        lib.oracle_decide_gram.argtypes = [
            ctypes.POINTER(_Cfg), ctypes.c_int, ctypes.c_void_p, ctypes.POINTER(_Ema),
            ctypes.POINTER(_Record),
        ]
        lib.oracle_f32_to_bf16.restype = ctypes.c_uint16
        lib.oracle_f32_to_bf16.argtypes = [ctypes.c_float]
        lib.oracle_bf16_to_f32.restype = ctypes.c_float
        lib.oracle_bf16_to_f32.argtypes = [ctypes.c_uint16]
        _lib_handle = lib
    return _lib_handle


@dataclass
class OracleConfig:
    """Hyper-parameters of one outer step (names follow the paper)."""
    outer_lr: float = 0.8          # nu
    momentum: float = 0.85         # rho
    clip_threshold: float = 10.0   # phi, Eq. 4
    clip_eps: float = 1e-6         # epsilon, Eq. 4
    ema_alpha: float = 0.02        # alpha, Eq. 1
    z_threshold: float = 3.0       # delta of the z-test
    warmup_rounds: int = 10        # rounds with no anomaly flagging
    flags: int = AE | WA | GC

    def _c(self) -> _Cfg:
        return _Cfg(self.outer_lr, self.momentum, self.clip_threshold, self.clip_eps,
                    self.ema_alpha, self.z_threshold, int(self.warmup_rounds), int(self.flags))


@dataclass
class OracleUnit:
    """One module's EMA state plus the step that advances it."""
    num_workers: int
    config: OracleConfig = field(default_factory=OracleConfig)

    def __post_init__(self):
        if not 1 <= self.num_workers <= MAX_K:
            raise ValueError("num_workers out of range")
        self._ema = _Ema()

    # -- state ------------------------------------------------------------
    @property
    def round(self) -> int:
        return int(self._ema.round)

    @property
    def mu(self) -> np.ndarray:
        return np.array(self._ema.mu[: self.num_workers], dtype=np.float64)

    @property
    def sigma(self) -> np.ndarray:
        return np.array(self._ema.sigma[: self.num_workers], dtype=np.float64)

    def set_state(self, mu: Sequence[float], sigma: Sequence[float], round_: int) -> None:
        for j in range(self.num_workers):
            self._ema.mu[j] = float(mu[j])
            self._ema.sigma[j] = float(sigma[j])
        self._ema.round = int(round_)

    # -- the step -----------------------------------------------------------
    def step(self, theta: np.ndarray, momentum: np.ndarray, replicas: List[np.ndarray]) -> dict:
        K = self.num_workers
        if len(replicas) != K:
            raise ValueError("expected %d replicas" % K)
        n = theta.size
        for a, dt in [(theta, np.float32), (momentum, np.float32)]:
            if a.dtype != dt or not a.flags.c_contiguous or a.size != n:
                raise ValueError("theta/momentum must be contiguous float32 of equal size")
        rdt = replicas[0].dtype
        if rdt not in (np.float32, np.uint16):
            raise ValueError("replicas must be float32 or uint16 (bf16 bits)")
        for r in replicas:
            if r.dtype != rdt or not r.flags.c_contiguous or r.size != n:
                raise ValueError("replicas must be contiguous, same dtype and size")
        ptrs = (ctypes.c_void_p * K)(*[r.ctypes.data for r in replicas])
        rec = _Record()
        rc = _lib().oracle_step(ctypes.byref(self.config._c()), K, n, int(rdt == np.uint16),
                                theta.ctypes.data, momentum.ctypes.data, ptrs,
                                ctypes.byref(self._ema), ctypes.byref(rec))
        if rc != 0:
            raise RuntimeError("oracle_step failed with %d" % rc)
        return self._record(rec)

    def decide_gram(self, gram: np.ndarray) -> dict:
        """The decision of one step from a given Gram matrix of the pseudo
        gradients (upper triangle row by row, fp64), advancing the EMA state
        as step() does; no elementwise update."""
        K = self.num_workers
        g = np.ascontiguousarray(gram, dtype=np.float64)
        if g.shape != (K * (K + 1) // 2,):
            raise ValueError("expected the %d upper-triangle entries" % (K * (K + 1) // 2))
        rec = _Record()
        rc = _lib().oracle_decide_gram(ctypes.byref(self.config._c()), K, g.ctypes.data,
                                       ctypes.byref(self._ema), ctypes.byref(rec))
        if rc != 0:
            raise RuntimeError("oracle_decide_gram failed with %d" % rc)
        return self._record(rec)

    def _record(self, rec: "_Record") -> dict:
        K = self.num_workers
        return {
            "norm": np.array(rec.norm[:K]),
            "anomalous": np.array(rec.anomalous[:K], dtype=np.uint8),
            "weight": np.array(rec.weight[:K]),
            "margin": np.array(rec.margin[:K]),
            "synced_norm": float(rec.synced_norm),
            "clip_coef": float(rec.clip_coef),
            "rolled_back": int(rec.rolled_back),
            "z_tested": int(rec.z_tested),
            "mu": self.mu,
            "sigma": self.sigma,
            "round": self.round,
        }


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Oracle's round-to-nearest-even fp32 -> bf16 (elementwise, slow)."""
    lib = _lib()
    flat = np.asarray(x, dtype=np.float32).ravel()
    return np.array([lib.oracle_f32_to_bf16(float(v)) for v in flat], dtype=np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    lib = _lib()
    flat = np.asarray(h, dtype=np.uint16).ravel()
    out = np.array([lib.oracle_bf16_to_f32(int(v)) for v in flat], dtype=np.float32)
    return out
