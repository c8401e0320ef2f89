"""Parity harness: the HIP path (through the C-ABI) against the float64
oracle on the same seeded input bytes.  Test infrastructure only.

Tolerances:
* parameters and momentum, per element:
    |x - y| <= 1e-5 * max(|y|, rms_l(y), |y_prev|)
  with rms_l the oracle RMS of layer l and y_prev the oracle's value before
  the step (relative error of fp32 state, guarded near zero by the layer
  scale; a new w or m is a sum whose largest term has the size of the
  previous value, and an fp32 sum's rounding is relative to that term, which
  matters where the terms cancel in a layer of one or a few elements);
* statistics (W, G, V, S, rho, a, b, gradscale, global G and Delta):
    |x - y| <= 1e-4 * |y|, and exact where the oracle's value is exactly 0
  (the spread of identical replicas, a single replica) or infinite;
* the per-layer Delta_l = |G_l - G_l,prev| / G_l,prev cancels when the
  layer's norm barely changes, so its bound adds the error of the two fp32
  per-layer norms (relative error below 1e-6 each: tile sums of at most
  2048 terms, then fp64):  |x - y| <= 1e-4 * |y| + 2e-6 * (1 + y);
* the sensitive bit is compared exactly, and the harness asserts that the
  oracle's Delta is not within 1e-6 * delta of the threshold, where fp32
  and fp64 sums could legitimately take different branches;
* element scales (elementwise AGS), per element: |x - y| <= 1e-5 * |y|,
  exact where the oracle's scale is 0.  The GPU forms each scale's
  denominator from an fp64 replica sum and rounds it once, then divides in
  fp32, so the scale carries about two fp32 roundings (1.2e-7 relative;
  3e-7 with the root-mean-square numerator) however close gbar_j is to 0.
"""
from __future__ import annotations

import math
import sys
import time

import numpy as np

from oracle import OracleAGS
from paper_2603_18112_amd import ags, layouts, synth

PARAM_RTOL = 1e-5
STAT_RTOL = 1e-4
SCALE_RTOL = 1e-5


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_device(arr: np.ndarray):
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16)).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


def check_params(x: np.ndarray, y: np.ndarray, table, what: str, rtol: float = PARAM_RTOL,
                 y_prev: np.ndarray | None = None):
    """Per-element check with the layer-RMS and previous-value guards;
    returns the worst error over tolerance scale."""
    worst = 0.0
    for l, (o, n, _) in enumerate(table):
        yy = y[o:o + n]
        xx = x[o:o + n].astype(np.float64)
        rms = math.sqrt(float(np.mean(yy * yy)))
        scale = np.maximum(np.abs(yy), rms)
        if y_prev is not None:
            scale = np.maximum(scale, np.abs(y_prev[o:o + n]))
        err = np.abs(xx - yy)
        bad = err > rtol * scale
        if np.any(~np.isfinite(xx)) or np.any(bad):
            i = int(np.argmax(np.where(np.isfinite(err), err / np.maximum(scale, 1e-300), np.inf)))
            raise AssertionError(
                f"{what}: layer {l} element {i}: got {xx[i]!r}, oracle {yy[i]!r}, "
                f"rms {rms:.3e}, {int(bad.sum())} of {n} out of tolerance")
        if n:
            r = float(np.max(err / np.maximum(scale, 1e-300)))
            worst = max(worst, r)
    return worst


def check_scales(x: np.ndarray, y: np.ndarray, table, what: str, rtol: float = SCALE_RTOL):
    """Element scales of every layer (elements outside the layers are not
    compared: the kernels never read or write them)."""
    for l, (o, n, _) in enumerate(table):
        xx = x[o:o + n].astype(np.float64)
        yy = y[o:o + n]
        bad = ~(np.abs(xx - yy) <= rtol * np.abs(yy))
        if np.any(bad):
            i = int(np.argmax(bad))
            raise AssertionError(f"{what}: layer {l} element {i}: scale {xx[i]!r}, oracle {yy[i]!r}, "
                                 f"{int(bad.sum())} of {n} out of tolerance")


def _close(x, y, rtol):
    if math.isinf(y) or math.isnan(y):
        return (math.isinf(x) and math.isinf(y) and (x > 0) == (y > 0)) or (math.isnan(x) and math.isnan(y))
    if y == 0.0:
        return x == 0.0
    return abs(x - y) <= rtol * abs(y)


def _close_delta_l(x, y, rtol):
    if math.isinf(y):
        return math.isinf(x) and x > 0
    return abs(x - y) <= rtol * abs(y) + DELTA_L_ABS * (1.0 + y)


DELTA_L_ABS = 2e-6


def check_stats(gpu_layer, gpu_glob, ora_layer, ora_glob, delta_thr, what="", rtol=STAT_RTOL,
                fields=ags.LAYER_STATS_FIELDS, layer_scope=False, scaled=None):
    for f in fields:
        for l, (x, y) in enumerate(zip(gpu_layer[f], ora_layer[f])):
            if f == "sensitive":
                ok = int(x) == int(y)
            elif f == "delta":
                ok = _close_delta_l(float(x), float(y), rtol)
            else:
                ok = _close(float(x), float(y), rtol)
            if not ok:
                raise AssertionError(f"{what} {f}[{l}]: got {x!r}, oracle {y!r}")
    if layer_scope:
        # A layer whose Delta_l lies within the error bound of the threshold
        # could legitimately take either branch: the case is reseeded.
        for l, y in enumerate(ora_layer["delta"]):
            if math.isfinite(y) and (scaled is None or scaled[l]):
                assert abs(y - delta_thr) > DELTA_L_ABS * (1 + y) + 1e-6 * delta_thr, \
                    f"{what}: oracle Delta_{l} {y} is within the error bound of the threshold; reseed"
    for f in ("g_sq", "g_sq_prev", "delta"):
        if not _close(float(gpu_glob[f]), float(ora_glob[f]), rtol):
            raise AssertionError(f"{what} global {f}: got {gpu_glob[f]!r}, oracle {ora_glob[f]!r}")
    d = ora_glob["delta"]
    if math.isfinite(d):
        assert abs(d - delta_thr) > 1e-6 * delta_thr, \
            f"{what}: oracle Delta {d} is within 1e-6 of the threshold; reseed"
    assert gpu_glob["sensitive"] == ora_glob["sensitive"], f"{what}: sensitive differs"
    assert gpu_glob["nonfinite"] == ora_glob["nonfinite"], f"{what}: nonfinite differs"


class Pair:
    """A GPU handle and an oracle started from the same weights."""

    def __init__(self, layout: layouts.Layout, K: int, *, dtype="f32", mode="ags", seed=0,
                 w0=None, stride=None, **hyper):
        import torch
        self.torch = torch
        self.layout = layout
        self.table = layout.table()
        self.K, self.dtype = K, dtype
        self.stride = stride or layout.n_flat
        self.hyper = dict(lr=0.1, momentum=0.9, weight_decay=5e-4, delta=0.5, eps=1e-8,
                          s_max=0.0, trust_coef=1e-3, refresh_every=1, small_replica=0)
        self.hyper.update(hyper)
        self.ew = bool(self.hyper.get("elementwise", False))
        self.layer_scope = self.hyper.get("delta_scope", "global") == "layer"
        self.scaled = [bool(f & layouts.LAYER_SCALE) for _, _, f in self.table]
        self.w0 = synth.init_weights(layout, seed) if w0 is None else np.asarray(w0, np.float32)
        self.w = torch.from_numpy(self.w0.copy()).cuda()
        self.m = torch.zeros_like(self.w)
        self.gpu = ags.AGS(self.table, self.w, self.m, K, grad_dtype=dtype, mode=mode, **self.hyper)
        # reuse_w_norms only chooses where the GPU takes W_l from
        ora_hyper = {k: v for k, v in self.hyper.items() if k != "reuse_w_norms"}
        self.ora = OracleAGS(self.table, layout.n_flat, K, self.w0, mode=mode, grad_dtype=dtype,
                             **ora_hyper)

    def step(self, grads: np.ndarray, commit=True, check=True, what=""):
        g = to_device(grads)
        self.prev_w, self.prev_m = self.ora.w.copy(), self.ora.m.copy()
        if commit:
            self.gpu.step(g)
            ol, og = self.ora.step(grads)
        else:
            self.gpu.stats(g)
            ol, og = self.ora.stats(grads)
        s = self.gpu.read_stats()
        if check:
            check_stats(s.layer, s.glob, ol, og, self.hyper["delta"], what,
                        layer_scope=self.layer_scope, scaled=self.scaled)
        return s, (ol, og)

    def check_state(self, what=""):
        self.torch.cuda.synchronize()
        w = self.w.cpu().numpy()
        m = self.m.cpu().numpy()
        pw, pm = getattr(self, "prev_w", None), getattr(self, "prev_m", None)
        rw = check_params(w, self.ora.w, self.table, what + " w", y_prev=pw)
        rm = check_params(m, self.ora.m, self.table, what + " m", y_prev=pm)
        gs, gp, st = self.gpu.get_state()
        ogs, ogp, ost = self.ora.get_state()
        assert st == ost
        if self.ew:
            check_scales(self.gpu.get_elementwise_scale(), ogs, self.table, what + " scales")
            ogs = np.array([np.mean(ogs[o:o + n]) for o, n, _ in self.table])
        for x, y in zip(gs, ogs):
            assert _close(float(x), float(y), STAT_RTOL), (x, y)
        assert _close(gp, ogp, STAT_RTOL)
        for x, y in zip(self.gpu.get_layer_state(), self.ora.get_layer_state()):
            assert _close(float(x), float(y), STAT_RTOL), (x, y)
        return rw, rm

    def close(self):
        self.gpu.close()


def run_steps(layout, K, steps, *, dtype="f32", mode="ags", seed=0, noise=0.5, check_each=True,
              label="", **hyper):
    """Run ``steps`` fresh-gradient steps on both sides and check them.  The
    next step's gradients are drawn on a helper thread while the current
    step runs (the draw is keyed by the step, so the bytes are the same)."""
    from concurrent.futures import ThreadPoolExecutor
    t0 = time.time()
    p = Pair(layout, K, dtype=dtype, mode=mode, seed=seed, **hyper)
    sig = synth.layer_sigmas(layout, seed)
    worst = (0.0, 0.0)

    def draw(t):
        return synth.replica_grads(layout, K, t, seed, noise=noise, dtype=dtype, sigmas=sig,
                                   stride=p.stride)

    try:
        with ThreadPoolExecutor(1) as ex:
            nxt = ex.submit(draw, 0)
            for t in range(steps):
                g = nxt.result()
                if t + 1 < steps:
                    nxt = ex.submit(draw, t + 1)
                p.step(g, what=f"{label} step {t + 1}")
                del g
                if check_each or t == steps - 1:
                    r = p.check_state(f"{label} step {t + 1}")
                    worst = (max(worst[0], r[0]), max(worst[1], r[1]))
                log(f"  {label}: step {t + 1}/{steps} ok ({time.time() - t0:.1f}s)")
    finally:
        p.close()
    return worst
