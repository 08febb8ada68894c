"""Seeded synthetic inputs for the RaaS decode path.

Test and benchmark infrastructure: it draws Q/K/V for the workloads in
``synth.workloads`` and holds none of the method's arithmetic. The same
arrays feed the HIP path and the CPU oracle. Values are returned as float32
arrays whose entries are exactly representable in the workload's dtype
(bf16 workloads are rounded to bf16, nearest-even, before being widened).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .workloads import WORKLOADS, Workload, get_workload  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "raas_synth.c")
_LIB_PATH = os.path.join(_HERE, "libraas_synth.so")
_lib = None


class _SynthWorkload(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_layers", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("prefill_len", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("ms_period", ctypes.c_int32),
        ("ms_phase_random", ctypes.c_int32),
        ("ms_wmin", ctypes.c_int32),
        ("ms_wmax", ctypes.c_int32),
        ("outlier_p", ctypes.c_double),
        ("seed", ctypes.c_uint64),
    ]


def build(force: bool = False) -> str:
    """Compile the generator with gcc (OpenMP across units)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        fp = ctypes.POINTER(ctypes.c_float)
        wp = ctypes.POINTER(_SynthWorkload)
        lib.synth_prefill.argtypes = [wp, ctypes.c_int, fp, fp]
        lib.synth_prefill.restype = None
        lib.synth_prefill_units.argtypes = [wp, ctypes.c_int, ctypes.POINTER(ctypes.c_int), ctypes.c_int, fp, fp]
        lib.synth_prefill_units.restype = None
        lib.synth_steps.argtypes = [wp, ctypes.c_int, ctypes.c_int, ctypes.c_int, fp, fp, fp]
        lib.synth_steps.restype = None
        lib.synth_steps_units.argtypes = [wp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          ctypes.POINTER(ctypes.c_int), ctypes.c_int, fp, fp, fp]
        lib.synth_steps_units.restype = None
        lib.synth_active_milestones.argtypes = [
            wp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
            ctypes.POINTER(ctypes.c_int), ctypes.c_int,
        ]
        lib.synth_active_milestones.restype = ctypes.c_int
        u32p = ctypes.POINTER(ctypes.c_uint32)
        lib.synth_philox4x32_10.argtypes = [u32p, u32p, u32p]
        lib.synth_philox4x32_10.restype = None
        _lib = lib
    return _lib


def _cstruct(w: Workload, seed: int) -> _SynthWorkload:
    return _SynthWorkload(
        w.batch, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, w.prefill_len,
        1 if w.dtype == "bf16" else 0, w.ms_period, 1 if w.ms_phase_random else 0,
        w.ms_wmin, w.ms_wmax, float(w.outlier_p), int(seed) & 0xFFFFFFFFFFFFFFFF,
    )


def _fptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def prefill(w: Workload, seed: int, layer: int = 0, prefill_len: int | None = None):
    """K, V of the prefill tokens: float32 [batch][n_kv_heads][P][head_dim]."""
    lib = _load()
    cw = _cstruct(w, seed)
    if prefill_len is not None:
        cw.prefill_len = int(prefill_len)
    shape = (w.batch, w.n_kv_heads, cw.prefill_len, w.head_dim)
    K = np.empty(shape, np.float32)
    V = np.empty(shape, np.float32)
    lib.synth_prefill(ctypes.byref(cw), int(layer), _fptr(K), _fptr(V))
    return K, V


def prefill_units(w: Workload, seed: int, layer: int, prefill_len: int, units):
    """prefill() restricted to chosen units (unit = sequence * n_kv_heads +
    KV head), with the same values: K, V float32 [len(units)][P][head_dim]."""
    lib = _load()
    cw = _cstruct(w, seed)
    cw.prefill_len = int(prefill_len)
    u = np.ascontiguousarray(np.asarray(units, dtype=np.int32))
    K = np.empty((len(u), cw.prefill_len, w.head_dim), np.float32)
    V = np.empty((len(u), cw.prefill_len, w.head_dim), np.float32)
    if len(u) and cw.prefill_len:
        lib.synth_prefill_units(ctypes.byref(cw), int(layer), u.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), len(u),
                                _fptr(K), _fptr(V))
    return K, V


def steps(w: Workload, seed: int, layer: int, t0: int, n: int):
    """Decode inputs of steps t0..t0+n-1.

    Returns q [n][batch][n_q_heads][d], k and v [n][batch][n_kv_heads][d]
    (float32)."""
    lib = _load()
    cw = _cstruct(w, seed)
    q = np.empty((n, w.batch, w.n_q_heads, w.head_dim), np.float32)
    k = np.empty((n, w.batch, w.n_kv_heads, w.head_dim), np.float32)
    v = np.empty((n, w.batch, w.n_kv_heads, w.head_dim), np.float32)
    if n > 0:
        lib.synth_steps(ctypes.byref(cw), int(layer), int(t0), int(n), _fptr(q), _fptr(k), _fptr(v))
    return q, k, v


def steps_units(w: Workload, seed: int, layer: int, t0: int, n: int, units):
    """steps() restricted to chosen units (unit = sequence * n_kv_heads + KV
    head), with the same values: q [n][len(units)][G][d], k and v
    [n][len(units)][d] (float32)."""
    lib = _load()
    cw = _cstruct(w, seed)
    u = np.ascontiguousarray(np.asarray(units, dtype=np.int32))
    nu = len(u)
    q = np.empty((n, nu, w.group, w.head_dim), np.float32)
    k = np.empty((n, nu, w.head_dim), np.float32)
    v = np.empty((n, nu, w.head_dim), np.float32)
    if n > 0 and nu > 0:
        lib.synth_steps_units(ctypes.byref(cw), int(layer), int(t0), int(n),
                              u.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), nu, _fptr(q), _fptr(k), _fptr(v))
    return q, k, v


def active_milestones(w: Workload, seed: int, layer: int, seq: int, kv_head: int, t: int):
    """Decode steps of the milestones whose window covers step t."""
    lib = _load()
    cw = _cstruct(w, seed)
    buf = (ctypes.c_int * 256)()
    n = lib.synth_active_milestones(ctypes.byref(cw), layer, seq, kv_head, t, buf, 256)
    return [buf[i] for i in range(min(n, 256))]


def philox4x32_10(ctr, key):
    lib = _load()
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    lib.synth_philox4x32_10(c, k, o)
    return [int(o[i]) for i in range(4)]
