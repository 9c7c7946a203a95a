"""Seeded synthetic inputs shared by the tests, the bench and the oracle's callers.

This package generates inputs only (replay rows and the workload descriptions);
it contains none of the update's arithmetic, imports neither the oracle nor the
HIP package, and is imported by neither of them.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .workloads import WORKLOADS, Workload, workload  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile synth.c into libsynth.so next to it (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        fp = ctypes.POINTER(ctypes.c_float)
        lib.synth_rows.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_double, ctypes.c_int64, ctypes.c_int64, fp, fp, fp, fp, fp]
        lib.synth_rows.restype = None
        lib.synth_rows_at.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_double, ctypes.POINTER(ctypes.c_int64), ctypes.c_int64,
                                      fp, fp, fp, fp, fp]
        lib.synth_rows_at.restype = None
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def _alloc(n, O, A):
    return (np.empty((n, O), np.float32), np.empty((n, A), np.float32), np.empty(n, np.float32),
            np.empty(n, np.float32), np.empty((n, O), np.float32))


def rows(obs_dim: int, act_dim: int, row0: int, n: int, seed: int = 0, zero_mod: int = 0,
         p_done: float = 0.01):
    """Rows row0..row0+n-1 as (obs, act, rew, done, next_obs) float32 arrays."""
    out = _alloc(n, obs_dim, act_dim)
    if n:
        _load().synth_rows(seed, obs_dim, act_dim, zero_mod, p_done, row0, n, *map(_ptr, out))
    return out


def rows_at(obs_dim: int, act_dim: int, idx, seed: int = 0, zero_mod: int = 0, p_done: float = 0.01):
    """The rows listed in idx (int64, any order) as (obs, act, rew, done, next_obs)."""
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64))
    out = _alloc(idx.size, obs_dim, act_dim)
    if idx.size:
        _load().synth_rows_at(seed, obs_dim, act_dim, zero_mod, p_done,
                              idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), idx.size,
                              *map(_ptr, out))
    return out


def workload_rows(w: Workload, row0: int, n: int, seed: int = 0):
    return rows(w.obs_dim, w.act_dim, row0, n, seed, w.zero_mod, w.p_done)


def workload_rows_at(w: Workload, idx, seed: int = 0):
    return rows_at(w.obs_dim, w.act_dim, idx, seed, w.zero_mod, w.p_done)
