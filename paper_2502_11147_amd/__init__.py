"""MI355X decode path of page-based RaaS (arXiv 2502.11147) -- Python binding.

A thin ctypes binding of ``libraas.so`` (the C ABI in ``include/raas.h``):
argument marshalling only. Every step of the path runs in the library's HIP
kernels on the GPU; PyTorch supplies device memory and the stream. There is
no fallback: without the built library, or without a GPU, calls fail.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libraas.so")

OK, E_INVALID, E_BUDGET, E_STATE, E_HIP, E_OOM = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
PREFILL_PIN_HEAD, PREFILL_ERROR = 0, 1
SCORE_MAX, SCORE_SOFTMAX_SUM = 0, 1
SCOPE_KV_HEAD, SCOPE_SEQUENCE = 0, 1
FREE, PINNED, EVICTABLE = 0, 1, 2
KERNELS = ("step", "epilogue", "prompt_select")  # raas_profile kernel indices

# C entry points declared in include/raas.h
EXPORTS = (
    "raas_create_pool", "raas_prefill", "raas_decode_step", "raas_destroy", "raas_last_error",
    "raas_abi_version", "raas_pool_bytes", "raas_export_state", "raas_set_attention_splits",
    "raas_profile", "raas_profile_read", "raas_prefill_ragged", "raas_decode_step_masked",
    "raas_decode_step_static", "raas_layer_checkpoint_bytes", "raas_save_layer", "raas_load_layer",
)


class RaasError(RuntimeError):
    def __init__(self, code: int, what: str, msg: str):
        super().__init__("%s failed (%d): %s" % (what, code, msg))
        self.code = code


class Config(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_layers", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("budget_tokens", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("r", ctypes.c_double),
        ("prefill_policy", ctypes.c_int32),
        ("score_aggregation", ctypes.c_int32),
        ("rank_pinned", ctypes.c_int32),
        ("decision_scope", ctypes.c_int32),
        ("prompt_tokens", ctypes.c_int32),
        ("prompt_topk", ctypes.c_int32),
        ("deterministic", ctypes.c_int32),
    ]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libraas.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("%s is not built: run __graft_entry__.build() (hipcc, gfx950)" % path)
    lib = ctypes.CDLL(path)
    vp, i32, ip = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)
    lib.raas_create_pool.argtypes = [ctypes.POINTER(Config), vp, ctypes.POINTER(vp)]
    lib.raas_create_pool.restype = i32
    lib.raas_prefill.argtypes = [vp, i32, vp, vp, i32, vp]
    lib.raas_prefill.restype = i32
    lib.raas_decode_step.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.raas_decode_step.restype = i32
    lib.raas_prefill_ragged.argtypes = [vp, i32, vp, vp, ip, ip, i32, vp]
    lib.raas_prefill_ragged.restype = i32
    lib.raas_decode_step_masked.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.raas_decode_step_masked.restype = i32
    lib.raas_decode_step_static.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.raas_decode_step_static.restype = i32
    lib.raas_destroy.argtypes = [vp]
    lib.raas_destroy.restype = None
    lib.raas_last_error.argtypes = []
    lib.raas_last_error.restype = ctypes.c_char_p
    lib.raas_abi_version.argtypes = []
    lib.raas_abi_version.restype = i32
    lib.raas_pool_bytes.argtypes = [vp]
    lib.raas_pool_bytes.restype = ctypes.c_size_t
    lib.raas_export_state.argtypes = [vp, i32, ip, ctypes.c_size_t, vp]
    lib.raas_export_state.restype = i32
    lib.raas_layer_checkpoint_bytes.argtypes = [vp]
    lib.raas_layer_checkpoint_bytes.restype = ctypes.c_size_t
    lib.raas_save_layer.argtypes = [vp, i32, vp, ctypes.c_size_t, vp]
    lib.raas_save_layer.restype = i32
    lib.raas_load_layer.argtypes = [vp, i32, vp, ctypes.c_size_t, vp]
    lib.raas_load_layer.restype = i32
    lib.raas_set_attention_splits.argtypes = [vp, i32]
    lib.raas_set_attention_splits.restype = i32
    lib.raas_profile.argtypes = [vp, i32]
    lib.raas_profile.restype = i32
    lib.raas_profile_read.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    lib.raas_profile_read.restype = i32
    _lib = lib
    return lib


def last_error() -> str:
    return load_library().raas_last_error().decode()


def _check(rc: int, what: str):
    if rc != OK:
        raise RaasError(rc, what, last_error())


def _torch():
    import torch

    return torch


def _stream_handle(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class Pool:
    """A fixed HBM page pool for every layer, with RaaS retention (raas_create_pool)."""

    def __init__(self, batch: int, n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 page_size: int, budget_tokens: int, dtype: str = "bf16", r: float = 0.5,
                 prefill_policy: int = PREFILL_PIN_HEAD, score_aggregation: int = SCORE_MAX,
                 rank_pinned: bool = False, decision_scope: int = SCOPE_KV_HEAD, prompt_tokens: int = 0,
                 prompt_topk: int = 0, deterministic: bool = False, stream=None):
        self.lib = load_library()
        self.cfg = Config(batch, n_layers, n_q_heads, n_kv_heads, head_dim, page_size, budget_tokens,
                          BF16 if dtype == "bf16" else F32, r, prefill_policy, score_aggregation,
                          int(rank_pinned), decision_scope, prompt_tokens, prompt_topk, int(deterministic))
        self.dtype = dtype
        self.batch, self.n_layers = batch, n_layers
        self.n_q_heads, self.n_kv_heads, self.head_dim = n_q_heads, n_kv_heads, head_dim
        self.page_size, self.budget = page_size, budget_tokens
        self.slots = (budget_tokens + prompt_tokens) // page_size
        self.units = batch * n_kv_heads
        self._h = ctypes.c_void_p()
        _check(self.lib.raas_create_pool(ctypes.byref(self.cfg), _stream_handle(stream), ctypes.byref(self._h)),
               "raas_create_pool")

    @classmethod
    def for_workload(cls, w, **kw):
        return cls(w.batch, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, w.page_size, w.budget,
                   w.dtype, w.r, **kw)

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            self.lib.raas_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    def _tensor(self, t, shape, name):
        torch = _torch()
        want = torch.bfloat16 if self.dtype == "bf16" else torch.float32
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise TypeError("%s must be a CUDA (HIP) tensor" % name)
        if t.dtype != want or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
            raise ValueError("%s must be a contiguous %s tensor of shape %s (got %s %s)"
                             % (name, want, tuple(shape), t.dtype, tuple(t.shape)))
        return ctypes.c_void_p(t.data_ptr())

    @staticmethod
    def _i32(t, shape, name):
        if t is None:
            return None
        torch = _torch()
        if not t.is_cuda or t.dtype != torch.int32 or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
            raise ValueError("%s must be a contiguous int32 CUDA tensor of shape %s" % (name, tuple(shape)))
        return ctypes.c_void_p(t.data_ptr())

    def prefill(self, layer: int, k, v, stream=None):
        """k, v: [batch][n_kv_heads][P][head_dim] device tensors (raas_prefill)."""
        P = 0 if k is None else int(k.shape[2])
        shape = (self.batch, self.n_kv_heads, P, self.head_dim)
        kp = self._tensor(k, shape, "k") if P > 0 else None
        vp = self._tensor(v, shape, "v") if P > 0 else None
        _check(self.lib.raas_prefill(self._h, layer, kp, vp, P, _stream_handle(stream)), "raas_prefill")

    def prefill_ragged(self, layer: int, k, v, lens, mask=None, stream=None):
        """Per-sequence prompt lengths (raas_prefill_ragged). k, v: [batch]
        [n_kv_heads][max_len][head_dim] device tensors; lens, mask: host
        sequences of batch ints (mask: the sequences to (re)initialise)."""
        B = self.batch
        lens = [int(x) for x in lens]
        if len(lens) != B:
            raise ValueError("lens must have %d entries" % B)
        max_len = 0 if k is None else int(k.shape[2])
        shape = (B, self.n_kv_heads, max_len, self.head_dim)
        kp = self._tensor(k, shape, "k") if max_len > 0 else None
        vp = self._tensor(v, shape, "v") if max_len > 0 else None
        lens_c = (ctypes.c_int32 * B)(*lens)
        mask_c = None
        if mask is not None:
            mask = [int(bool(x)) for x in mask]
            if len(mask) != B:
                raise ValueError("mask must have %d entries" % B)
            mask_c = (ctypes.c_int32 * B)(*mask)
        _check(self.lib.raas_prefill_ragged(self._h, layer, kp, vp, lens_c, mask_c, max_len,
                                            _stream_handle(stream)), "raas_prefill_ragged")

    def prepare_step(self, layer: int, q, k_new, v_new, out, page_table=None, timestamps=None,
                     evicted=None, stream=None, active=None) -> tuple:
        """Checks and converts the arguments of one raas_decode_step_masked call
        once, so a loop can replay them with decode_prepared(). active: None, or
        a device int32 tensor [batch] (nonzero = the sequence takes the step)."""
        B, Hq, Hkv, d = self.batch, self.n_q_heads, self.n_kv_heads, self.head_dim
        return (
            self._h, layer,
            self._tensor(q, (B, Hq, d), "q"),
            self._tensor(k_new, (B, Hkv, d), "k_new"),
            self._tensor(v_new, (B, Hkv, d), "v_new"),
            self._tensor(out, (B, Hq, d), "out"),
            self._i32(page_table, (B, Hkv, self.slots), "page_table"),
            self._i32(timestamps, (B, Hkv, self.slots), "timestamps"),
            self._i32(evicted, (B, Hkv), "evicted"),
            self._i32(active, (B,), "active"),
            _stream_handle(stream),
        )

    def decode_prepared(self, args: tuple):
        _check(self.lib.raas_decode_step_masked(*args), "raas_decode_step_masked")

    def decode_step(self, layer: int, q, k_new, v_new, out, page_table=None, timestamps=None,
                    evicted=None, stream=None):
        """One decode step of one layer for every unit (raas_decode_step)."""
        self.decode_prepared(self.prepare_step(layer, q, k_new, v_new, out, page_table, timestamps,
                                               evicted, stream))

    def decode_step_static(self, layer: int, q, k_new, v_new, out, page_table=None, timestamps=None,
                           evicted=None, stream=None):
        """raas_decode_step with the step's scratch in the library's fixed
        device array (raas_decode_step_static): allocates nothing."""
        args = self.prepare_step(layer, q, k_new, v_new, out, page_table, timestamps, evicted, stream)
        _check(self.lib.raas_decode_step_static(*(args[:9] + args[10:])), "raas_decode_step_static")

    def export_state(self, layer: int, stream=None) -> dict:
        import numpy as np

        U, S = self.units, self.slots
        buf = np.empty(U * (4 * S + 4), np.int32)
        _check(self.lib.raas_export_state(self._h, layer, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                          buf.size, _stream_handle(stream)), "raas_export_state")
        n = U * S
        unit = buf[4 * n:].reshape(U, 4)
        return dict(lid=buf[:n].reshape(U, S), ts=buf[n:2 * n].reshape(U, S),
                    state=buf[2 * n:3 * n].reshape(U, S), fill=buf[3 * n:4 * n].reshape(U, S),
                    tail=unit[:, 0].copy(), next_lid=unit[:, 1].copy(), clock=unit[:, 2].copy(),
                    evicted=unit[:, 3].copy())

    def save_layer(self, layer: int, stream=None):
        """One layer's whole state as a host byte array (raas_save_layer)."""
        import numpy as np

        buf = np.empty(int(self.lib.raas_layer_checkpoint_bytes(self._h)), np.uint8)
        _check(self.lib.raas_save_layer(self._h, layer, ctypes.c_void_p(buf.ctypes.data), buf.size,
                                        _stream_handle(stream)), "raas_save_layer")
        return buf

    def load_layer(self, layer: int, buf, stream=None):
        """Replaces one layer's state by a saved one (raas_load_layer); keep
        `buf` alive until the stream has run the copies."""
        import numpy as np

        buf = np.ascontiguousarray(buf, np.uint8)
        _check(self.lib.raas_load_layer(self._h, layer, ctypes.c_void_p(buf.ctypes.data), buf.size,
                                        _stream_handle(stream)), "raas_load_layer")
        return buf

    def pool_bytes(self) -> int:
        return int(self.lib.raas_pool_bytes(self._h))

    def set_attention_splits(self, splits: int):
        _check(self.lib.raas_set_attention_splits(self._h, splits), "raas_set_attention_splits")

    def profile(self, mask: int):
        _check(self.lib.raas_profile(self._h, mask), "raas_profile")

    def profile_read(self, kernel: int):
        ms = ctypes.c_double()
        n = ctypes.c_int64()
        _check(self.lib.raas_profile_read(self._h, kernel, ctypes.byref(ms), ctypes.byref(n)),
               "raas_profile_read")
        return ms.value, n.value
