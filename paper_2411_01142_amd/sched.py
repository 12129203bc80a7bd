"""Python binding of the library's cost model and load-aware scheduler
simulator (Sec. 3.2): argument marshalling only; every step runs in the
library's C++ (``csrc/scheduler.cpp``)."""
from __future__ import annotations

import ctypes
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

from . import NeoError, _check, load_library

POLICIES = {"neo": 0, "gpu_only": 1}
MODES = {0: "gpu_only", 1: "two_batch"}


class _Grid(ctypes.Structure):
    _fields_ = [("n_b", ctypes.c_int32), ("n_s", ctypes.c_int32),
                ("b", ctypes.POINTER(ctypes.c_double)), ("s", ctypes.POINTER(ctypes.c_double)),
                ("t", ctypes.POINTER(ctypes.c_double))]


class _Curve(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("x", ctypes.POINTER(ctypes.c_double)),
                ("t", ctypes.POINTER(ctypes.c_double))]


class _Config(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("gpu_blocks", ctypes.c_int64), ("cpu_blocks", ctypes.c_int64),
                ("max_batch_tokens", ctypes.c_int64), ("swap_in_reserve_blocks", ctypes.c_int64),
                ("t_ga", _Grid), ("t_ca", _Grid), ("t_l", _Curve), ("policy", ctypes.c_int32)]


class _Iter(ctypes.Structure):
    _fields_ = [("done", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("n_prefill", ctypes.c_int32), ("n_prefill_to_cpu", ctypes.c_int32),
                ("n_gpu_decode", ctypes.c_int32), ("n_cpu_decode0", ctypes.c_int32),
                ("n_cpu_decode1", ctypes.c_int32), ("n_swap_out", ctypes.c_int32),
                ("n_swap_in", ctypes.c_int32), ("n_tokens", ctypes.c_int64),
                ("t_iter", ctypes.c_double), ("t_two_batch", ctypes.c_double),
                ("t_gpu_only", ctypes.c_double), ("t_l0", ctypes.c_double),
                ("t_l1", ctypes.c_double), ("t_ga0", ctypes.c_double), ("t_ca0", ctypes.c_double),
                ("t_ca1", ctypes.c_double), ("now", ctypes.c_double)]


class _Stats(ctypes.Structure):
    _fields_ = [("now", ctypes.c_double)] + [(n, ctypes.c_int64) for n in (
        "tokens", "iterations", "two_batch_iterations", "finished", "swapped_out", "swapped_in",
        "preempted", "gpu_blocks_held", "cpu_blocks_held", "waiting", "gpu_running",
        "cpu_running")]


def _setup(lib):
    if getattr(lib, "_neo_sched_ready", False):
        return lib
    P = ctypes.c_void_p
    D = ctypes.c_double
    lib.neo_cost_eval_grid.argtypes = [ctypes.POINTER(_Grid), D, D, ctypes.POINTER(D)]
    lib.neo_cost_eval_grid.restype = ctypes.c_int
    lib.neo_cost_eval_curve.argtypes = [ctypes.POINTER(_Curve), D, ctypes.POINTER(D)]
    lib.neo_cost_eval_curve.restype = ctypes.c_int
    lib.neo_sched_create.argtypes = [ctypes.POINTER(_Config), ctypes.POINTER(P)]
    lib.neo_sched_create.restype = ctypes.c_int
    lib.neo_sched_add_request.argtypes = [P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, D]
    lib.neo_sched_add_request.restype = ctypes.c_int
    lib.neo_sched_step.argtypes = [P, ctypes.POINTER(_Iter), ctypes.POINTER(ctypes.c_int64),
                                   ctypes.c_int64]
    lib.neo_sched_step.restype = ctypes.c_int
    lib.neo_sched_get_stats.argtypes = [P, ctypes.POINTER(_Stats)]
    lib.neo_sched_get_stats.restype = ctypes.c_int
    lib.neo_sched_destroy.argtypes = [P]
    lib.neo_sched_destroy.restype = None
    lib._neo_sched_ready = True
    return lib


def _dbl(a):
    a = np.ascontiguousarray(a, dtype=np.float64)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


@dataclass
class CostGrid:
    """Per-layer seconds on a (requests, total context tokens) grid."""
    b: Sequence[float]
    s: Sequence[float]
    t: Sequence[Sequence[float]]  # [len(b)][len(s)]

    def _c(self, keep: list) -> _Grid:
        b, pb = _dbl(self.b)
        s, ps = _dbl(self.s)
        t, pt = _dbl(self.t)
        if t.shape != (len(b), len(s)):
            raise ValueError("t must be [len(b)][len(s)]")
        keep += [b, s, t]
        return _Grid(len(b), len(s), pb, ps, pt)

    def __call__(self, b: float, s: float) -> float:
        keep: list = []
        g = self._c(keep)
        out = ctypes.c_double()
        lib = _setup(load_library())
        _check(lib.neo_cost_eval_grid(ctypes.byref(g), float(b), float(s), ctypes.byref(out)))
        return out.value


@dataclass
class CostCurve:
    """Per-layer seconds over a token count."""
    x: Sequence[float]
    t: Sequence[float]

    def _c(self, keep: list) -> _Curve:
        x, px = _dbl(self.x)
        t, pt = _dbl(self.t)
        if t.shape != x.shape:
            raise ValueError("x and t must have the same length")
        keep += [x, t]
        return _Curve(len(x), px, pt)

    def __call__(self, x: float) -> float:
        keep: list = []
        c = self._c(keep)
        out = ctypes.c_double()
        lib = _setup(load_library())
        _check(lib.neo_cost_eval_curve(ctypes.byref(c), float(x), ctypes.byref(out)))
        return out.value


@dataclass
class SchedConfig:
    num_layers: int
    block_size: int
    gpu_blocks: int
    cpu_blocks: int
    max_batch_tokens: int
    t_ga: CostGrid
    t_ca: CostGrid
    t_l: CostCurve
    swap_in_reserve_blocks: int = 0
    policy: str = "neo"


@dataclass
class Iteration:
    mode: str
    prefill: List[int]
    gpu_decode: List[int]
    cpu_decode0: List[int]
    cpu_decode1: List[int]
    swap_out: List[int]
    swap_in: List[int]
    n_prefill_to_cpu: int
    n_tokens: int
    t_iter: float
    t_two_batch: float
    t_gpu_only: float
    t_l0: float
    t_l1: float
    t_ga0: float
    t_ca0: float
    t_ca1: float
    now: float


class Scheduler:
    """The library's scheduler simulator (one handle)."""

    def __init__(self, cfg: SchedConfig):
        self._lib = _setup(load_library())
        keep: list = []
        c = _Config(cfg.num_layers, cfg.block_size, cfg.gpu_blocks, cfg.cpu_blocks,
                    cfg.max_batch_tokens, cfg.swap_in_reserve_blocks, cfg.t_ga._c(keep),
                    cfg.t_ca._c(keep), cfg.t_l._c(keep), POLICIES[cfg.policy])
        h = ctypes.c_void_p()
        _check(self._lib.neo_sched_create(ctypes.byref(c), ctypes.byref(h)))
        self._h = h
        self._n = 0

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.neo_sched_destroy(h)
            self._h = None

    def add(self, rid: int, prompt_len: int, output_len: int, arrival: float = 0.0):
        _check(self._lib.neo_sched_add_request(self._h, int(rid), int(prompt_len),
                                               int(output_len), float(arrival)))
        self._n += 1

    def step(self) -> Optional[Iteration]:
        """One iteration; None when every request has finished."""
        it = _Iter()
        cap = max(1, 3 * self._n)
        ids = (ctypes.c_int64 * cap)()
        _check(self._lib.neo_sched_step(self._h, ctypes.byref(it), ids, cap))
        if it.done:
            return None
        counts = [it.n_prefill, it.n_gpu_decode, it.n_cpu_decode0, it.n_cpu_decode1,
                  it.n_swap_out, it.n_swap_in]
        lists, k = [], 0
        for c in counts:
            lists.append([int(ids[k + j]) for j in range(c)])
            k += c
        return Iteration(MODES[it.mode], *lists, it.n_prefill_to_cpu, it.n_tokens, it.t_iter,
                         it.t_two_batch, it.t_gpu_only, it.t_l0, it.t_l1, it.t_ga0, it.t_ca0,
                         it.t_ca1, it.now)

    def stats(self) -> dict:
        st = _Stats()
        _check(self._lib.neo_sched_get_stats(self._h, ctypes.byref(st)))
        return {name: getattr(st, name) for name, _ in _Stats._fields_}

    def run(self, max_iterations: int = 10 ** 7) -> List[Iteration]:
        out = []
        for _ in range(max_iterations):
            it = self.step()
            if it is None:
                return out
            out.append(it)
        raise NeoError(1, "simulation did not finish")
