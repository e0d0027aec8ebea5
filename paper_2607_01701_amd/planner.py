"""Binding of the native cascade planner (t2v_list_schedule, t2v_plan_cascades): argument
marshalling only. The planner runs in the host-only library, so no GPU is needed.

A problem is a DAG of cascades (predecessor lists), the set K of parallel degrees, per-cascade
latency L[c][j] and memory Mem[c][j] at degree K[j], a per-GPU memory cap W and N GPUs
(paper Section IV-A, Eqs. (1)-(7); Alg. 1).
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import _lib

_dp = ctypes.POINTER(ctypes.c_double)


def _csr(preds):
    ptr = np.zeros(len(preds) + 1, dtype=np.int32)
    idx = []
    for c, ps in enumerate(preds):
        idx.extend(int(p) for p in ps)
        ptr[c + 1] = len(idx)
    return ptr, np.asarray(idx if idx else [0], dtype=np.int32)


def list_schedule(preds, degree, latency, n_gpus: int, L=None):
    """Critical-path list schedule for fixed degrees; returns (starts [n], makespan)."""
    L = L or _lib.host_lib()
    n = len(preds)
    ptr, idx = _csr(preds)
    deg = np.ascontiguousarray(degree, dtype=np.int32)
    lat = np.ascontiguousarray(latency, dtype=np.float64)
    if deg.shape != (n,) or lat.shape != (n,):
        raise ValueError("degree and latency need one entry per cascade")
    start = np.zeros(max(n, 1), dtype=np.float64)
    T = ctypes.c_double(0.0)
    st = L.t2v_list_schedule(n, ptr.ctypes.data_as(_lib._i32p), idx.ctypes.data_as(_lib._i32p),
                             deg.ctypes.data_as(_lib._i32p), lat.ctypes.data_as(_dp), int(n_gpus),
                             start.ctypes.data_as(_dp), ctypes.byref(T))
    _lib._check(L, st)
    return start[:n], T.value


def plan(preds, degrees, latency, mem, mem_cap: float, n_gpus: int, population: int = 64, generations: int = 200,
         mutation: float = 0.05, elite: int = 4, seed: int = 0, L=None):
    """Genetic-algorithm plan (Alg. 1); returns (degree per cascade, starts, makespan)."""
    L = L or _lib.host_lib()
    n = len(preds)
    ptr, idx = _csr(preds)
    K = np.ascontiguousarray(degrees, dtype=np.int32)
    lat = np.ascontiguousarray(latency, dtype=np.float64).reshape(n, K.shape[0]) if n else np.zeros((0, K.shape[0]))
    mm = np.ascontiguousarray(mem, dtype=np.float64).reshape(n, K.shape[0]) if n else np.zeros((0, K.shape[0]))
    lat = np.ascontiguousarray(lat)
    mm = np.ascontiguousarray(mm)
    deg_out = np.zeros(max(n, 1), dtype=np.int32)
    start = np.zeros(max(n, 1), dtype=np.float64)
    T = ctypes.c_double(0.0)
    st = L.t2v_plan_cascades(n, ptr.ctypes.data_as(_lib._i32p), idx.ctypes.data_as(_lib._i32p), int(K.shape[0]),
                             K.ctypes.data_as(_lib._i32p), lat.ctypes.data_as(_dp), mm.ctypes.data_as(_dp),
                             float(mem_cap), int(n_gpus), int(population), int(generations), float(mutation),
                             int(elite), int(seed) & ((1 << 64) - 1), deg_out.ctypes.data_as(_lib._i32p),
                             start.ctypes.data_as(_dp), ctypes.byref(T))
    _lib._check(L, st)
    return deg_out[:n], start[:n], T.value
