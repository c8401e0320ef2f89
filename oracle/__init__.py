"""Float64 CPU oracle of the AGS step (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg use
this package.  It is the reference the GPU library is checked against and is
never called by the library.  The arithmetic lives in ``ags_oracle.c``
(plain C, float64, single thread); this module compiles it with gcc when no
build is present and wraps it with ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ags_oracle.c")
# AGS_ORACLE_LIB names another build of the same source (the sanitizer
# test loads an AddressSanitizer / UBSan build through it).
_LIB = os.environ.get("AGS_ORACLE_LIB") or os.path.join(_HERE, "liboracle_ags.so")
_lock = threading.Lock()
_lib = None

MODES = {"sgd": 0, "ags": 1, "lars": 2, "static": 3}
LAYER_FIELDS = ("w_sq", "g_sq", "var", "gsmall_sq", "noise_ratio", "coef_a",
                "coef_b", "gradscale", "delta", "sensitive")
DELTA_SCOPES = {"global": 0, "layer": 1}
GLOBAL_FIELDS = ("g_sq", "g_sq_prev", "delta", "sensitive", "nonfinite")


class _Layer(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_int64), ("numel", ctypes.c_int64),
                ("flags", ctypes.c_uint32), ("pad_", ctypes.c_uint32)]


class _Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("K", ctypes.c_int32),
                ("grad_is_bf16", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("refresh_every", ctypes.c_int32), ("small_replica", ctypes.c_int32),
                ("n_flat", ctypes.c_int64), ("replica_stride", ctypes.c_int64),
                ("lr", ctypes.c_double), ("momentum", ctypes.c_double),
                ("weight_decay", ctypes.c_double), ("delta", ctypes.c_double),
                ("eps", ctypes.c_double), ("s_max", ctypes.c_double),
                ("trust_coef", ctypes.c_double), ("static_scale", ctypes.c_double),
                ("elementwise", ctypes.c_int32), ("delta_scope", ctypes.c_int32)]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain -O2, no fast-math)."""
    with _lock:
        if os.environ.get("AGS_ORACLE_LIB"):
            return _LIB
        if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            tmp = _LIB + f".tmp{os.getpid()}"
            subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared",
                                   "-fno-fast-math", "-ffp-contract=off",
                                   _SRC, "-o", tmp, "-lm"])
            os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_ags_step.restype = ctypes.c_int
        lib.oracle_ags_step.argtypes = [
            ctypes.POINTER(_Config), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.POINTER(ctypes.c_double), ctypes.c_void_p,
            ctypes.POINTER(ctypes.c_int64), ctypes.c_int, ctypes.POINTER(_Layer), ctypes.c_void_p,
            ctypes.c_void_p]
        _lib = lib
    return _lib


class OracleAGS:
    """Stateful float64 oracle: weights, momentum and AGS state in float64.

    ``layers`` is a list of (offset, numel, flags); ``w0``/``m0`` are the
    initial flat buffers (any float dtype, converted exactly to float64).
    """

    def __init__(self, layers, n_flat, K, w0, m0=None, *, mode="ags",
                 grad_dtype="f32", lr=0.1, momentum=0.9, weight_decay=5e-4,
                 delta=0.5, eps=1e-8, s_max=0.0, trust_coef=1e-3, static_scale=2.0,
                 refresh_every=1, small_replica=0, elementwise=False, delta_scope="global"):
        self.lib = _load()
        self.layers = [(int(o), int(n), int(f)) for o, n, f in layers]
        self.L = len(self.layers)
        self.n_flat = int(n_flat)
        self.K = int(K)
        self.grad_dtype = grad_dtype
        self.cfg = dict(mode=mode, lr=lr, momentum=momentum, weight_decay=weight_decay,
                        delta=delta, eps=eps, s_max=s_max, trust_coef=trust_coef,
                        static_scale=static_scale, elementwise=bool(elementwise),
                        refresh_every=refresh_every, small_replica=small_replica,
                        delta_scope=DELTA_SCOPES[delta_scope])
        self.w = np.array(w0, dtype=np.float64, copy=True).reshape(-1)
        self.m = (np.zeros(self.n_flat) if m0 is None
                  else np.array(m0, dtype=np.float64, copy=True).reshape(-1))
        if self.w.size != self.n_flat or self.m.size != self.n_flat:
            raise ValueError("w/m size does not match n_flat")
        # one scale per layer, or per element of the flat buffer
        self.gradscale = np.ones(self.n_flat if elementwise else self.L)
        self.g_prev = ctypes.c_double(0.0)
        self.g_prev_layers = np.zeros(max(self.L, 1))
        self.step_count = ctypes.c_int64(0)
        arr = (_Layer * max(self.L, 1))()
        for i, (o, n, f) in enumerate(self.layers):
            arr[i].offset, arr[i].numel, arr[i].flags = o, n, f
        self._layers_c = arr

    @property
    def step_index(self) -> int:
        return int(self.step_count.value)

    def get_state(self):
        return self.gradscale.copy(), float(self.g_prev.value), int(self.step_count.value)

    def set_state(self, gradscale, g_prev, step):
        self.gradscale[:] = np.asarray(gradscale, dtype=np.float64)
        self.g_prev.value = float(g_prev)
        self.step_count.value = int(step)

    def get_layer_state(self):
        """Per-layer ||gbar_l||^2 of the last committed step."""
        return self.g_prev_layers[:self.L].copy()

    def set_layer_state(self, g_prev_layers):
        self.g_prev_layers[:self.L] = np.asarray(g_prev_layers, dtype=np.float64)

    def _run(self, grads, commit, lr=None):
        g = np.ascontiguousarray(grads)
        if self.grad_dtype == "bf16":
            if g.dtype != np.uint16:
                raise TypeError("bf16 gradients are passed as uint16 bit patterns")
        elif g.dtype != np.float32:
            raise TypeError("f32 gradients must be float32")
        if g.ndim != 2 or g.shape[0] != self.K or g.shape[1] < self.n_flat:
            raise ValueError("gradients must be [K, stride >= n_flat]")
        c = self.cfg
        cfg = _Config(n_layers=self.L, K=self.K, grad_is_bf16=int(self.grad_dtype == "bf16"),
                      mode=MODES[c["mode"]], refresh_every=int(c["refresh_every"]),
                      small_replica=int(c["small_replica"]), n_flat=self.n_flat,
                      replica_stride=int(g.shape[1]),
                      lr=float(c["lr"] if lr is None else lr), momentum=float(c["momentum"]),
                      weight_decay=float(c["weight_decay"]), delta=float(c["delta"]),
                      eps=float(c["eps"]), s_max=float(c["s_max"]),
                      trust_coef=float(c["trust_coef"]),
                      static_scale=float(c["static_scale"]),
                      elementwise=int(c["elementwise"]), delta_scope=int(c["delta_scope"]))
        out_l = np.zeros((self.L, len(LAYER_FIELDS)))
        out_g = np.zeros(len(GLOBAL_FIELDS))
        rc = self.lib.oracle_ags_step(
            ctypes.byref(cfg), self.w.ctypes.data, self.m.ctypes.data, g.ctypes.data,
            self.gradscale.ctypes.data, ctypes.byref(self.g_prev), self.g_prev_layers.ctypes.data,
            ctypes.byref(self.step_count), int(commit), self._layers_c,
            out_l.ctypes.data, out_g.ctypes.data)
        if rc != 0:
            raise RuntimeError(f"oracle_ags_step failed ({rc})")
        layer_stats = {k: out_l[:, i].copy() for i, k in enumerate(LAYER_FIELDS)}
        glob = {k: float(out_g[i]) for i, k in enumerate(GLOBAL_FIELDS)}
        layer_stats["sensitive"] = layer_stats["sensitive"].astype(np.int64)
        glob["sensitive"] = int(glob["sensitive"])
        glob["nonfinite"] = int(glob["nonfinite"])
        return layer_stats, glob

    def step(self, grads, lr=None):
        """One AGS step: statistics, decision, update, refresh."""
        return self._run(grads, commit=True, lr=lr)

    def stats(self, grads):
        """Statistics and coefficients only; no state changes."""
        return self._run(grads, commit=False)
