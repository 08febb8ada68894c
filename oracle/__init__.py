"""CPU oracle for page-based RaaS decode -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product path (the HIP library and
its binding) never calls it.

``raas_oracle.c`` is a plain fp64 implementation of one decode step of
page-based RaaS (Algorithm 1; Sections 3.2 and 3.3 of arXiv 2502.11147);
this module compiles it with gcc and wraps it with ctypes. ``history.py`` is
an independent pure-Python statement of the eviction rule used to pin the C
code.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "raas_oracle.c")
LIB_PATH = os.path.join(_HERE, "libraas_oracle.so")

OK, E_INVALID, E_BUDGET, E_STATE, E_INTERNAL = 0, -1, -2, -3, -10
FREE, PINNED, EVICTABLE = 0, 1, 2
PIN_HEAD, ERROR = 0, 1
AGG_MAX, AGG_SOFTMAX_SUM = 0, 1  # head aggregation of the page score

_libs: dict[str, ctypes.CDLL] = {}


def build(src: str = SRC, out: str = LIB_PATH, force: bool = False, extra=()) -> str:
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp",
                               *extra, "-o", tmp, src, "-lm"])
        os.replace(tmp, out)
    return out


def load(path: str | None = None) -> ctypes.CDLL:
    path = path or LIB_PATH
    if path not in _libs:
        if path == LIB_PATH:
            build()  # (re)compiles when missing or older than the source
        lib = ctypes.CDLL(path)
        vp, ip, dp = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double)
        lib.orc_new.argtypes = [ctypes.c_int] * 4 + [ctypes.c_double, ctypes.c_int]
        lib.orc_new.restype = vp
        lib.orc_free.argtypes = [vp]
        lib.orc_free.restype = None
        lib.orc_prefill.argtypes = [vp, dp, dp, ctypes.c_int]
        lib.orc_prefill.restype = ctypes.c_int
        lib.orc_decode.argtypes = [vp, dp, dp, dp, dp, dp]
        lib.orc_decode.restype = ctypes.c_int
        lib.orc_state.argtypes = [vp, ip, ip, ip, ip, ip]
        lib.orc_state.restype = None
        lib.orc_last_scores.argtypes = [vp, dp, dp]
        lib.orc_last_scores.restype = None
        lib.orc_pages.argtypes = [vp, dp, dp, dp, dp]
        lib.orc_pages.restype = None
        fp = ctypes.POINTER(ctypes.c_float)
        lib.orc_decode_batch.argtypes = [ctypes.POINTER(vp), ctypes.c_int, fp, fp, fp, dp]
        lib.orc_decode_batch.restype = ctypes.c_int
        lib.orc_decode_group.argtypes = [ctypes.POINTER(vp), ctypes.c_int, dp, dp, dp, dp]
        lib.orc_decode_group.restype = ctypes.c_int
        lib.orc_set_prompt_selection.argtypes = [vp, ctypes.c_int, ctypes.c_int]
        lib.orc_set_prompt_selection.restype = ctypes.c_int
        lib.orc_last_attended.argtypes = [vp, ip]
        lib.orc_last_attended.restype = None
        lib.orc_set_variant.argtypes = [vp, ctypes.c_int, ctypes.c_int]
        lib.orc_set_variant.restype = ctypes.c_int
        lib.orc_adopt_retention.argtypes = [vp, ip, ip, ctypes.c_int]
        lib.orc_adopt_retention.restype = ctypes.c_int
        lib.orc_state_batch.argtypes = [ctypes.POINTER(vp), ctypes.c_int, ip, ip, ip]
        lib.orc_state_batch.restype = None
        lib.orc_scores_batch.argtypes = [ctypes.POINTER(vp), ctypes.c_int, dp, dp]
        lib.orc_scores_batch.restype = None
        lib.orc_set_threads.argtypes = [ctypes.c_int]
        lib.orc_set_threads.restype = None
        lib.orc_threads.argtypes = []
        lib.orc_threads.restype = ctypes.c_int
        _libs[path] = lib
    return _libs[path]


def _dptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a, shape=None):
    if a is None:
        return None
    x = np.ascontiguousarray(a, dtype=np.float64)
    if shape is not None:
        x = x.reshape(shape)
    return x


class OracleError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__("%s returned %d" % (what, code))
        self.code = code


class Kvm:
    """The KV manager of one unit (sequence, layer, KV head) with G query heads."""

    def __init__(self, G: int, d: int, page_size: int, slots: int, r: float = 0.5,
                 policy: int = PIN_HEAD, lib: str | None = None, aggregation: int = AGG_MAX,
                 rank_pinned: bool = False, prompt_slots: int | None = None, prompt_topk: int | None = None):
        self.lib = load(lib)
        self.G, self.d, self.ps, self.S = G, d, page_size, slots
        self._h = self.lib.orc_new(G, d, page_size, slots, float(r), policy)
        if not self._h:
            raise ValueError("invalid oracle configuration")
        if aggregation != AGG_MAX or rank_pinned:
            if self.lib.orc_set_variant(self._h, int(aggregation), int(bool(rank_pinned))) != OK:
                raise ValueError("invalid oracle variant")
        if prompt_topk is not None:
            if self.lib.orc_set_prompt_selection(self._h, int(prompt_slots), int(prompt_topk)) != OK:
                raise ValueError("invalid prompt selection")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            self.lib.orc_free(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    def prefill(self, K, V) -> int:
        K = _f64(K)
        V = _f64(V)
        P = 0 if K is None else K.shape[0]
        return self.lib.orc_prefill(self._h, _dptr(K), _dptr(V), P)

    def decode(self, q, k, v, want_out: bool = True):
        """One decode step; returns the [G][d] fp64 attention output (or None)."""
        q = _f64(q, (self.G, self.d))
        k = _f64(k, (self.d,))
        v = _f64(v, (self.d,))
        out = np.empty((self.G, self.d), np.float64) if want_out else None
        rc = self.lib.orc_decode(self._h, _dptr(q), _dptr(k), _dptr(v), _dptr(out), None)
        if rc != OK:
            raise OracleError(rc, "orc_decode")
        return out

    def decode_with_scores(self, scores):
        """Retention-only step: the per-slot page scores are given, not computed."""
        s = _f64(scores, (self.S,))
        rc = self.lib.orc_decode(self._h, None, None, None, None, _dptr(s))
        if rc != OK:
            raise OracleError(rc, "orc_decode")

    def state(self) -> dict:
        S = self.S
        pt = np.empty(S, np.int32)
        ts = np.empty(S, np.int32)
        st = np.empty(S, np.int32)
        fl = np.empty(S, np.int32)
        un = np.empty(6, np.int32)
        ip = ctypes.POINTER(ctypes.c_int)
        self.lib.orc_state(self._h, *(a.ctypes.data_as(ip) for a in (pt, ts, st, fl, un)))
        return dict(page_table=pt, ts=ts, state=st, fill=fl, tail=int(un[0]), next_lid=int(un[1]),
                    clock=int(un[2]), evicted=int(un[3]), n_evictable=int(un[4]),
                    k_refreshed=int(un[5]))

    def adopt_retention(self, page_table, ts, evicted: int):
        """Lockstep test hook: take another implementation's retention
        decision of the last step (orc_adopt_retention). Raises when it
        differs in more than the step's own decisions."""
        pt = np.ascontiguousarray(page_table, np.int32)
        t = np.ascontiguousarray(ts, np.int32)
        ip = ctypes.POINTER(ctypes.c_int)
        rc = self.lib.orc_adopt_retention(self._h, pt.ctypes.data_as(ip), t.ctypes.data_as(ip), int(evicted))
        if rc != OK:
            raise OracleError(rc, "orc_adopt_retention")

    def last_attended(self):
        """slots the last step attended to (with outputs requested), as bools"""
        a = np.empty(self.S, np.int32)
        self.lib.orc_last_attended(self._h, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int)))
        return a.astype(bool)

    def last_scores(self):
        sc = np.empty(self.S, np.float64)
        th = ctypes.c_double()
        self.lib.orc_last_scores(self._h, _dptr(sc), ctypes.byref(th))
        return sc, th.value

    def pages(self):
        S, ps, d = self.S, self.ps, self.d
        K = np.empty((S, ps, d))
        V = np.empty((S, ps, d))
        kmin = np.empty((S, d))
        kmax = np.empty((S, d))
        self.lib.orc_pages(self._h, _dptr(K), _dptr(V), _dptr(kmin), _dptr(kmax))
        return K, V, kmin, kmax


def decode_batch(units: list[Kvm], q, k, v, want_out: bool = True):
    """One decode step for many units (OpenMP across units).

    q: float32 [n][G][d]; k, v: float32 [n][d]. Returns fp64 [n][G][d] or None."""
    n = len(units)
    lib = units[0].lib
    arr = (ctypes.c_void_p * n)(*[u.handle for u in units])
    q = np.ascontiguousarray(q, np.float32)
    k = np.ascontiguousarray(k, np.float32)
    v = np.ascontiguousarray(v, np.float32)
    out = np.empty((n, units[0].G, units[0].d), np.float64) if want_out else None
    fp = ctypes.POINTER(ctypes.c_float)
    rc = lib.orc_decode_batch(arr, n, q.ctypes.data_as(fp), k.ctypes.data_as(fp),
                              v.ctypes.data_as(fp), _dptr(out))
    if rc != OK:
        raise OracleError(rc, "orc_decode_batch")
    return out


def state_batch(units: list[Kvm]):
    """Page tables and timestamps [n][S] and evicted ids [n] of n alike units."""
    n, S = len(units), units[0].S
    arr = (ctypes.c_void_p * n)(*[u.handle for u in units])
    pt = np.empty((n, S), np.int32)
    ts = np.empty((n, S), np.int32)
    ev = np.empty(n, np.int32)
    ip = ctypes.POINTER(ctypes.c_int)
    units[0].lib.orc_state_batch(arr, n, pt.ctypes.data_as(ip), ts.ctypes.data_as(ip), ev.ctypes.data_as(ip))
    return pt, ts, ev


def scores_batch(units: list[Kvm]):
    """Last step's page scores [n][S] (NaN where not ranked) and thresholds [n]."""
    n, S = len(units), units[0].S
    arr = (ctypes.c_void_p * n)(*[u.handle for u in units])
    sc = np.empty((n, S), np.float64)
    th = np.empty(n, np.float64)
    units[0].lib.orc_scores_batch(arr, n, _dptr(sc), _dptr(th))
    return sc, th


def decode_group(units: list[Kvm], q, k, v, want_out: bool = True):
    """One decode step of a sequence whose KV heads (units, alike) share one
    page table (orc_decode_group). q: [n][G][d]; k, v: [n][d] (fp64).
    Returns fp64 [n][G][d] or None."""
    n = len(units)
    G, d = units[0].G, units[0].d
    arr = (ctypes.c_void_p * n)(*[u.handle for u in units])
    q = _f64(q, (n, G, d))
    k = _f64(k, (n, d))
    v = _f64(v, (n, d))
    out = np.empty((n, G, d), np.float64) if want_out else None
    rc = units[0].lib.orc_decode_group(arr, n, _dptr(q), _dptr(k), _dptr(v), _dptr(out))
    if rc != OK:
        raise OracleError(rc, "orc_decode_group")
    return out


def threads() -> int:
    return int(load().orc_threads())


def set_threads(n: int):
    """OpenMP threads of the batched oracle calls."""
    load().orc_set_threads(int(n))
