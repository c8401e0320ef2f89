"""Python binding of libags (include/ags.h): argument marshalling only.

Every function here has the name of the C function it calls and forwards
plain pointers and sizes; all arithmetic of the step runs in the HIP
kernels of libags.so.  PyTorch is used for device memory and streams only,
in the convenience class :class:`AGS`.

The library is loaded from ``paper_2603_18112_amd/_lib/libags.so``; build it
with ``python -m paper_2603_18112_amd._build`` (or ``__graft_entry__.build()``).
A missing library is an error: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import numpy as np

from . import _build

# ---------------------------------------------------------------- C types --

AGS_OK, AGS_E_ARG, AGS_E_LAYOUT, AGS_E_ALIGN, AGS_E_NOMEM, AGS_E_DEVICE, AGS_E_STATE = range(7)
STATUS_NAMES = {0: "AGS_OK", 1: "AGS_E_ARG", 2: "AGS_E_LAYOUT", 3: "AGS_E_ALIGN",
                4: "AGS_E_NOMEM", 5: "AGS_E_DEVICE", 6: "AGS_E_STATE"}
AGS_F32, AGS_BF16 = 0, 1
AGS_MODE_SGD, AGS_MODE_AGS, AGS_MODE_LARS, AGS_MODE_STATIC = 0, 1, 2, 3
AGS_LAYER_SCALE, AGS_LAYER_DECAY = 1, 2
AGS_DELTA_GLOBAL, AGS_DELTA_LAYER = 0, 1
DELTA_SCOPES = {"global": AGS_DELTA_GLOBAL, "layer": AGS_DELTA_LAYER}
AGS_ALIGN_ELEMS = 8
AGS_MAX_K = 1024
AGS_N_KERNELS = 3
KERNEL_NAMES = ("step", "finalize", "second_pass")
MODES = {"sgd": AGS_MODE_SGD, "ags": AGS_MODE_AGS, "lars": AGS_MODE_LARS,
         "static": AGS_MODE_STATIC}
DTYPES = {"f32": AGS_F32, "bf16": AGS_BF16}


class ags_layer(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_int64), ("numel", ctypes.c_int64),
                ("flags", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]


class ags_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("layers", ctypes.POINTER(ags_layer)),
                ("n_flat", ctypes.c_int64), ("K", ctypes.c_int32),
                ("grad_dtype", ctypes.c_int), ("mode", ctypes.c_int),
                ("lr", ctypes.c_double), ("momentum", ctypes.c_double),
                ("weight_decay", ctypes.c_double), ("delta", ctypes.c_double),
                ("eps", ctypes.c_double), ("s_max", ctypes.c_double),
                ("trust_coef", ctypes.c_double), ("refresh_every", ctypes.c_int32),
                ("small_replica", ctypes.c_int32), ("static_scale", ctypes.c_double),
                ("elementwise", ctypes.c_int32), ("delta_scope", ctypes.c_int32),
                ("reuse_w_norms", ctypes.c_int32)]


class ags_layer_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in
                ("w_sq", "g_sq", "var", "gsmall_sq", "noise_ratio", "coef_a", "coef_b", "gradscale",
                 "delta")] + [("sensitive", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class ags_global_stats(ctypes.Structure):
    _fields_ = [("step", ctypes.c_int64), ("g_sq", ctypes.c_double),
                ("g_sq_prev", ctypes.c_double), ("delta", ctypes.c_double),
                ("sensitive", ctypes.c_int32), ("nonfinite", ctypes.c_int32)]


LAYER_STATS_FIELDS = tuple(n for n, _ in ags_layer_stats._fields_ if n != "reserved")
#: every function the header declares
EXPORTS = ("ags_workspace_bytes", "ags_init", "ags_stats", "ags_step", "ags_read_stats",
           "ags_set_lr", "ags_get_state", "ags_set_state", "ags_get_layer_state",
           "ags_set_layer_state", "ags_get_last_decision", "ags_set_last_decision",
           "ags_get_elementwise_scale",
           "ags_set_elementwise_scale", "ags_invalidate_weight_norms", "ags_set_profiling",
           "ags_get_kernel_times", "ags_stats_noalloc", "ags_status_string", "ags_last_error",
           "ags_destroy")

_lib = None


class AGSError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def library_path() -> str:
    return _build.LIB


def load_library(path: str | None = None):
    """Load libags.so (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or _build.LIB
    # PyTorch for ROCm ships its own HIP runtime with the same soname as
    # /opt/rocm's.  Loading torch first makes libags bind to that runtime,
    # so one HIP runtime (and one set of streams and allocations) serves
    # both; loading libags first would bring in a second runtime.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(path):
        raise ImportError(f"libags.so is not built ({path}); run python -m paper_2603_18112_amd._build")
    lib = ctypes.CDLL(path)
    P, c_int, c_i64, c_dbl, vp = ctypes.POINTER, ctypes.c_int, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
    h = vp
    sig = {
        "ags_workspace_bytes": (c_int, [P(ags_config), P(ctypes.c_size_t)]),
        "ags_init": (c_int, [P(ags_config), vp, vp, vp, P(vp)]),
        "ags_stats": (c_int, [h, vp, c_i64, vp]),
        "ags_step": (c_int, [h, vp, c_i64, vp]),
        "ags_read_stats": (c_int, [h, vp, P(ags_global_stats)]),
        "ags_set_lr": (c_int, [h, c_dbl]),
        "ags_get_state": (c_int, [h, vp, P(c_dbl), P(c_i64)]),
        "ags_set_state": (c_int, [h, vp, c_dbl, c_i64]),
        "ags_invalidate_weight_norms": (c_int, [h]),
        "ags_stats_noalloc": (c_int, [P(ags_config), vp, vp, c_i64, vp, P(ags_global_stats), vp]),
        "ags_get_layer_state": (c_int, [h, vp]),
        "ags_set_layer_state": (c_int, [h, vp]),
        "ags_get_last_decision": (c_int, [h, vp, vp]),
        "ags_set_last_decision": (c_int, [h, ctypes.c_int32, vp]),
        "ags_get_elementwise_scale": (c_int, [h, vp, c_i64]),
        "ags_set_elementwise_scale": (c_int, [h, vp, c_i64]),
        "ags_set_profiling": (c_int, [h, c_int]),
        "ags_get_kernel_times": (c_int, [h, vp, P(c_i64)]),
        "ags_status_string": (ctypes.c_char_p, [c_int]),
        "ags_last_error": (ctypes.c_char_p, [h]),
        "ags_destroy": (None, [h]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(status: int, handle=None):
    if status != AGS_OK:
        msg = load_library().ags_last_error(handle)
        raise AGSError(status, msg.decode() if msg else "")


# ------------------------------------------------------------ thin calls --
# Same names and arguments as the C functions; pointers are ints.


def make_config(layers, n_flat, K, *, grad_dtype="f32", mode="ags", lr=0.1, momentum=0.9,
                weight_decay=5e-4, delta=0.5, eps=1e-8, s_max=0.0, trust_coef=1e-3,
                refresh_every=1, small_replica=0, static_scale=2.0, elementwise=False,
                delta_scope="global", reuse_w_norms=False):
    """An ags_config (plus the layer array it points to, kept alive on it)."""
    arr = (ags_layer * max(len(layers), 1))()
    for i, (o, n, f) in enumerate(layers):
        arr[i].offset, arr[i].numel, arr[i].flags, arr[i].reserved = int(o), int(n), int(f), 0
    cfg = ags_config(n_layers=len(layers), layers=ctypes.cast(arr, ctypes.POINTER(ags_layer)),
                     n_flat=int(n_flat), K=int(K), grad_dtype=DTYPES[grad_dtype], mode=MODES[mode],
                     lr=float(lr), momentum=float(momentum), weight_decay=float(weight_decay),
                     delta=float(delta), eps=float(eps), s_max=float(s_max),
                     trust_coef=float(trust_coef), refresh_every=int(refresh_every),
                     small_replica=int(small_replica), static_scale=float(static_scale),
                     elementwise=int(bool(elementwise)), delta_scope=DELTA_SCOPES[delta_scope],
                     reuse_w_norms=int(bool(reuse_w_norms)))
    cfg._layers_keepalive = arr
    return cfg


def ags_status_string(status: int) -> str:
    return load_library().ags_status_string(int(status)).decode()


def ags_last_error(handle=None) -> str:
    r = load_library().ags_last_error(handle)
    return r.decode() if r else ""


def ags_workspace_bytes(cfg) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().ags_workspace_bytes(ctypes.byref(cfg), ctypes.byref(out)))
    return int(out.value)


def ags_init(cfg, d_w: int, d_m: int, stream: int = 0):
    h = ctypes.c_void_p(0)
    _check(load_library().ags_init(ctypes.byref(cfg), d_w, d_m, stream, ctypes.byref(h)))
    return h


def ags_stats(handle, d_grads: int, replica_stride: int, stream: int = 0):
    _check(load_library().ags_stats(handle, d_grads, int(replica_stride), stream), handle)


def ags_step(handle, d_grads: int, replica_stride: int, stream: int = 0):
    _check(load_library().ags_step(handle, d_grads, int(replica_stride), stream), handle)


def ags_read_stats(handle, n_layers: int):
    arr = (ags_layer_stats * max(n_layers, 1))()
    g = ags_global_stats()
    _check(load_library().ags_read_stats(handle, ctypes.cast(arr, ctypes.c_void_p), ctypes.byref(g)), handle)
    layer = {f: np.array([getattr(arr[i], f) for i in range(n_layers)]) for f in LAYER_STATS_FIELDS}
    glob = {"step": int(g.step), "g_sq": g.g_sq, "g_sq_prev": g.g_sq_prev, "delta": g.delta,
            "sensitive": int(g.sensitive), "nonfinite": int(g.nonfinite)}
    return layer, glob


def ags_set_lr(handle, lr: float):
    _check(load_library().ags_set_lr(handle, float(lr)), handle)


def ags_get_state(handle, n_layers: int):
    gs = np.zeros(max(n_layers, 1))
    gp = ctypes.c_double(0)
    st = ctypes.c_int64(0)
    _check(load_library().ags_get_state(handle, gs.ctypes.data, ctypes.byref(gp), ctypes.byref(st)), handle)
    return gs[:n_layers].copy(), float(gp.value), int(st.value)


def ags_set_state(handle, gradscale, g_sq_prev: float, step: int):
    if gradscale is None:
        ptr = None
    else:
        gs = np.ascontiguousarray(gradscale, dtype=np.float64)
        ptr = gs.ctypes.data
    _check(load_library().ags_set_state(handle, ptr, float(g_sq_prev), int(step)), handle)


def ags_stats_noalloc(cfg, d_w: int, d_grads: int, replica_stride: int, stream: int = 0):
    """Statistics of one replica set without a handle and without any device
    allocation; returns (per-layer dict, global dict) like ags_read_stats."""
    n = int(cfg.n_layers)
    arr = (ags_layer_stats * max(n, 1))()
    g = ags_global_stats()
    _check(load_library().ags_stats_noalloc(ctypes.byref(cfg), d_w, d_grads, int(replica_stride),
                                            ctypes.cast(arr, ctypes.c_void_p), ctypes.byref(g),
                                            stream))
    layer = {f: np.array([getattr(arr[i], f) for i in range(n)]) for f in LAYER_STATS_FIELDS}
    glob = {"step": int(g.step), "g_sq": g.g_sq, "g_sq_prev": g.g_sq_prev, "delta": g.delta,
            "sensitive": int(g.sensitive), "nonfinite": int(g.nonfinite)}
    return layer, glob


def ags_invalidate_weight_norms(handle):
    _check(load_library().ags_invalidate_weight_norms(handle), handle)


def ags_get_layer_state(handle, n_layers: int):
    out = np.zeros(max(int(n_layers), 1))
    _check(load_library().ags_get_layer_state(handle, out.ctypes.data), handle)
    return out[:int(n_layers)].copy()


def ags_set_layer_state(handle, g_sq_prev):
    a = np.ascontiguousarray(g_sq_prev, dtype=np.float64).reshape(-1)
    _check(load_library().ags_set_layer_state(handle, a.ctypes.data), handle)


def ags_get_last_decision(handle, n_layers: int):
    """(global sensitive bit, per-layer bits) of the last committed step."""
    g = np.zeros(1, np.int32)
    per = np.zeros(max(int(n_layers), 1), np.int32)
    _check(load_library().ags_get_last_decision(handle, g.ctypes.data, per.ctypes.data), handle)
    return int(g[0]), per[:int(n_layers)].copy()


def ags_set_last_decision(handle, sensitive: int, sensitive_l=None):
    if sensitive_l is None:
        _check(load_library().ags_set_last_decision(handle, int(sensitive), None), handle)
        return
    a = np.ascontiguousarray(sensitive_l, dtype=np.int32).reshape(-1)
    _check(load_library().ags_set_last_decision(handle, int(sensitive), a.ctypes.data), handle)


def ags_get_elementwise_scale(handle, n: int):
    out = np.empty(max(int(n), 1), np.float32)
    _check(load_library().ags_get_elementwise_scale(handle, out.ctypes.data, int(n)), handle)
    return out[:int(n)].copy()


def ags_set_elementwise_scale(handle, scale):
    a = np.ascontiguousarray(scale, dtype=np.float32).reshape(-1)
    _check(load_library().ags_set_elementwise_scale(handle, a.ctypes.data, int(a.size)), handle)


def ags_set_profiling(handle, enable: bool):
    _check(load_library().ags_set_profiling(handle, int(bool(enable))), handle)


def ags_get_kernel_times(handle):
    ms = np.zeros(AGS_N_KERNELS)
    n = ctypes.c_int64(0)
    _check(load_library().ags_get_kernel_times(handle, ms.ctypes.data, ctypes.byref(n)), handle)
    return ms, int(n.value)


def ags_destroy(handle):
    if handle is not None and handle.value:
        load_library().ags_destroy(handle)


# ------------------------------------------------------- torch convenience --


@dataclass
class StepStats:
    layer: dict
    glob: dict


class AGS:
    """A libags handle over torch tensors (device memory and streams only).

    ``w`` and ``m`` are contiguous fp32 CUDA tensors of ``n_flat`` elements,
    updated in place by :meth:`step`.  ``grads`` passed to :meth:`step` /
    :meth:`stats` is a contiguous [K, stride] tensor, fp32 or bf16 (bf16 may
    also be passed as int16/uint16 bit patterns).
    """

    def __init__(self, layers, w, m, K, *, grad_dtype="f32", mode="ags", stream=None, **hyper):
        import torch
        self.torch = torch
        for name, t in (("w", w), ("m", m)):
            if not (t.is_cuda and t.dtype == torch.float32 and t.is_contiguous()):
                raise ValueError(f"{name} must be a contiguous float32 CUDA tensor")
        if w.numel() != m.numel():
            raise ValueError("w and m differ in size")
        self.layers = [(int(o), int(n), int(f)) for o, n, f in layers]
        self.n_layers = len(self.layers)
        self.K = int(K)
        self.grad_dtype = grad_dtype
        self.w, self.m = w, m
        self.cfg = make_config(self.layers, w.numel(), K, grad_dtype=grad_dtype, mode=mode, **hyper)
        self.handle = ags_init(self.cfg, w.data_ptr(), m.data_ptr(), self._stream(stream))

    def _stream(self, stream):
        if stream is None:
            stream = self.torch.cuda.current_stream(self.w.device)
        return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)

    def _grads(self, grads):
        t = self.torch
        want = {"f32": (t.float32,), "bf16": (t.bfloat16, t.int16, t.uint16)}[self.grad_dtype]
        if grads.dtype not in want or not grads.is_cuda or not grads.is_contiguous() or grads.dim() != 2:
            raise ValueError(f"grads must be a contiguous 2-D CUDA tensor of dtype {want}")
        if grads.shape[0] != self.K:
            raise ValueError(f"grads has {grads.shape[0]} replicas, the handle has K={self.K}")
        return grads.data_ptr(), grads.shape[1]

    def step(self, grads, stream=None):
        p, stride = self._grads(grads)
        ags_step(self.handle, p, stride, self._stream(stream))

    def stats(self, grads, stream=None):
        p, stride = self._grads(grads)
        ags_stats(self.handle, p, stride, self._stream(stream))

    def read_stats(self) -> StepStats:
        layer, glob = ags_read_stats(self.handle, self.n_layers)
        return StepStats(layer, glob)

    def set_lr(self, lr):
        ags_set_lr(self.handle, lr)

    def get_state(self):
        return ags_get_state(self.handle, self.n_layers)

    def set_state(self, gradscale, g_sq_prev, step):
        # the C function reads n_layers values; with element scales it reads
        # none (gradscale may be None)
        if gradscale is not None:
            gradscale = np.asarray(gradscale, dtype=np.float64).reshape(-1)
            if gradscale.size != self.n_layers:
                raise ValueError(f"expected {self.n_layers} gradscale values, got {gradscale.size}")
        ags_set_state(self.handle, gradscale, g_sq_prev, step)

    def invalidate_weight_norms(self):
        ags_invalidate_weight_norms(self.handle)

    def get_layer_state(self):
        return ags_get_layer_state(self.handle, self.n_layers)

    def set_layer_state(self, g_sq_prev):
        g = np.asarray(g_sq_prev, dtype=np.float64).reshape(-1)
        if g.size != self.n_layers:
            raise ValueError(f"expected {self.n_layers} values, got {g.size}")
        ags_set_layer_state(self.handle, g)

    def get_last_decision(self):
        return ags_get_last_decision(self.handle, self.n_layers)

    def set_last_decision(self, sensitive, sensitive_l=None):
        if sensitive_l is not None:
            sensitive_l = np.asarray(sensitive_l, dtype=np.int32).reshape(-1)
            if sensitive_l.size != self.n_layers:
                raise ValueError(f"expected {self.n_layers} values, got {sensitive_l.size}")
        ags_set_last_decision(self.handle, sensitive, sensitive_l)

    def get_elementwise_scale(self):
        return ags_get_elementwise_scale(self.handle, self.w.numel())

    def set_elementwise_scale(self, scale):
        ags_set_elementwise_scale(self.handle, scale)

    def set_profiling(self, enable=True):
        ags_set_profiling(self.handle, enable)

    def kernel_times(self):
        return ags_get_kernel_times(self.handle)

    def close(self):
        if getattr(self, "handle", None) is not None:
            ags_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
