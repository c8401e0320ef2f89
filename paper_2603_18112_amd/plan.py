"""Python binding of the libags planner (include/ags_plan.h): argument
marshalling only; the model fit, the time and cost estimates, the memory
bound and the selection policy run in the library.
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import ags

AGS_SYNC_NONE, AGS_SYNC_RING, AGS_SYNC_PS = 0, 1, 2
SYNC = {"none": AGS_SYNC_NONE, "ring": AGS_SYNC_RING, "ps": AGS_SYNC_PS}
AGS_PLAN_INTERCEPT, AGS_PLAN_COMPUTE, AGS_PLAN_SYNC = 1, 2, 4
SHAPES = {"concave_inc": 0, "concave_dec": 1, "convex_inc": 2, "convex_dec": 3}
OBJECTIVES = {"time": 0, "cost": 1, "knee": 2}
EXPORTS = ("ags_plan_fit", "ags_plan_step_time", "ags_plan_time_cost", "ags_plan_max_local_batch",
           "ags_plan_knee", "ags_plan_select")


class ags_plan_sample(ctypes.Structure):
    _fields_ = [("nodes", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("local_batch", ctypes.c_double), ("t_step", ctypes.c_double)]


class ags_plan_model(ctypes.Structure):
    _fields_ = [("sync", ctypes.c_int), ("terms", ctypes.c_uint32), ("c0", ctypes.c_double),
                ("c_compute", ctypes.c_double), ("c_sync", ctypes.c_double),
                ("rms_residual", ctypes.c_double), ("n_samples", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]

    def as_dict(self):
        return {"sync": self.sync, "terms": self.terms, "c0": self.c0, "c_compute": self.c_compute,
                "c_sync": self.c_sync, "rms_residual": self.rms_residual,
                "n_samples": self.n_samples}


class ags_plan_candidate(ctypes.Structure):
    _fields_ = [("nodes", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("global_batch", ctypes.c_double)]


_sig_done = False


def _lib():
    global _sig_done
    lib = ags.load_library()
    if not _sig_done:
        P, c_int, c_i32, c_i64, c_dbl, vp = (ctypes.POINTER, ctypes.c_int, ctypes.c_int32,
                                              ctypes.c_int64, ctypes.c_double, ctypes.c_void_p)
        sig = {
            "ags_plan_fit": [vp, c_i32, c_int, ctypes.c_uint32, P(ags_plan_model)],
            "ags_plan_step_time": [P(ags_plan_model), c_i32, c_dbl, P(c_dbl)],
            "ags_plan_time_cost": [P(ags_plan_model), c_i32, c_dbl, c_dbl, c_dbl, c_dbl, P(c_dbl),
                                   P(c_dbl)],
            "ags_plan_max_local_batch": [c_dbl, c_dbl, c_dbl, P(c_i64)],
            "ags_plan_knee": [vp, vp, c_i32, c_int, c_dbl, P(c_i32)],
            "ags_plan_select": [P(ags_plan_model), vp, c_i32, c_dbl, c_dbl, c_dbl, c_dbl, c_int, c_dbl,
                                P(c_i32), vp, vp],
        }
        for name, args in sig.items():
            f = getattr(lib, name)
            f.restype = c_int
            f.argtypes = args
        _sig_done = True
    return lib


def _check(status):
    if status != ags.AGS_OK:
        raise ags.AGSError(status, ags.ags_last_error(None))


def ags_plan_fit(samples, sync="ring", terms=AGS_PLAN_INTERCEPT | AGS_PLAN_COMPUTE | AGS_PLAN_SYNC):
    """samples: iterable of (nodes, local_batch, t_step)."""
    samples = list(samples)
    arr = (ags_plan_sample * max(len(samples), 1))()
    for i, (n, b, t) in enumerate(samples):
        arr[i].nodes, arr[i].reserved, arr[i].local_batch, arr[i].t_step = int(n), 0, float(b), float(t)
    m = ags_plan_model()
    _check(_lib().ags_plan_fit(ctypes.cast(arr, ctypes.c_void_p), len(samples), SYNC[sync],
                               int(terms), ctypes.byref(m)))
    return m


def ags_plan_step_time(model, nodes, local_batch):
    out = ctypes.c_double()
    _check(_lib().ags_plan_step_time(ctypes.byref(model), int(nodes), float(local_batch),
                                     ctypes.byref(out)))
    return out.value


def ags_plan_time_cost(model, nodes, global_batch, epochs, dataset_size, price_per_node_hour):
    T, C = ctypes.c_double(), ctypes.c_double()
    _check(_lib().ags_plan_time_cost(ctypes.byref(model), int(nodes), float(global_batch),
                                     float(epochs), float(dataset_size), float(price_per_node_hour),
                                     ctypes.byref(T), ctypes.byref(C)))
    return T.value, C.value


def ags_plan_max_local_batch(capacity, m_static, m_per_sample):
    out = ctypes.c_int64()
    _check(_lib().ags_plan_max_local_batch(float(capacity), float(m_static), float(m_per_sample),
                                           ctypes.byref(out)))
    return int(out.value)


def ags_plan_knee(x, y, shape="convex_dec", sensitivity=1.0):
    """Index of the Kneedle knee, or None."""
    xa = np.ascontiguousarray(x, dtype=np.float64)
    ya = np.ascontiguousarray(y, dtype=np.float64)
    if xa.shape != ya.shape or xa.ndim != 1:
        raise ValueError("x and y must be 1-D arrays of one length")
    out = ctypes.c_int32()
    _check(_lib().ags_plan_knee(xa.ctypes.data, ya.ctypes.data, len(xa), SHAPES[shape],
                                float(sensitivity), ctypes.byref(out)))
    return None if out.value < 0 else int(out.value)


def ags_plan_select(model, candidates, epochs, dataset_size, price_per_node_hour,
                    max_local_batch=float("inf"), objective="time", sensitivity=1.0):
    """candidates: iterable of (nodes, global_batch).  Returns (index or
    None, T array, C array)."""
    candidates = list(candidates)
    n = len(candidates)
    arr = (ags_plan_candidate * max(n, 1))()
    for i, (nn, B) in enumerate(candidates):
        arr[i].nodes, arr[i].reserved, arr[i].global_batch = int(nn), 0, float(B)
    T = np.zeros(max(n, 1))
    C = np.zeros(max(n, 1))
    best = ctypes.c_int32()
    _check(_lib().ags_plan_select(ctypes.byref(model), ctypes.cast(arr, ctypes.c_void_p), n,
                                  float(epochs), float(dataset_size), float(price_per_node_hour),
                                  float(max_local_batch), OBJECTIVES[objective], float(sensitivity),
                                  ctypes.byref(best), T.ctypes.data, C.ctypes.data))
    return (None if best.value < 0 else int(best.value)), T[:n].copy(), C[:n].copy()
