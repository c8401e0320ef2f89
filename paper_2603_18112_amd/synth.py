"""Seeded synthetic inputs for the AGS step: weights and replica gradients.

This module only *draws* inputs; it holds none of the method's arithmetic and
is shared by the GPU path's tests/bench and by the float64 oracle's tests, so
that both sides read the very same bytes.

Recipe (the paper trains CNNs on ImageNet-1K / CIFAR100 / CalTech, Sec. IV-B;
neither the datasets nor trained weights are needed, only the parameter
shapes and gradients of a realistic scale):

* weights: Kaiming-normal, std = sqrt(2 / fan_in) for conv and fc weights;
  biases U(-1/sqrt(fan_in), 1/sqrt(fan_in)); BN gamma = 1, beta = 0 (or,
  with ``perturb_bn``, gamma ~ 1 + N(0, 0.1^2), beta ~ N(0, 0.1^2));
* per-layer gradient scale sigma_l, log-uniform in [1e-4, 1e-1];
* replica gradients g[k, l] = mu_l + eps[k, l] with a shared mean
  mu_l ~ N(0, sigma_l^2) and per-replica noise eps ~ N(0, (c sigma_l)^2),
  drawn fresh for every step; the replicas stand in for the K data-parallel
  workers' local gradients of one step (Eq. (1c)), and their spread plays
  the role of the small/large-batch noise term of Eq. (6);
* generated in fp32; bf16 gradients are the fp32 values rounded to nearest
  even.

Randomness is counter based: every (purpose, step, layer, replica) draws from
its own Philox-4x64 stream (Salmon et al., SC'11) whose 128-bit key is
(seed, packed tuple), so any piece can be regenerated on its own, in any
order, on any machine.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .layouts import Layout

_P_WEIGHT, _P_SIGMA, _P_MEAN, _P_NOISE, _P_BN = 1, 2, 3, 4, 5
#: replica id used for the shared per-layer mean stream
_SHARED = 0xFFFF


def _rng(seed: int, purpose: int, step: int = 0, layer: int = 0,
         replica: int = 0) -> np.random.Generator:
    if not (0 <= step < (1 << 24) and 0 <= layer < (1 << 16) and 0 <= replica < (1 << 16)):
        raise ValueError("generator key out of range")
    k1 = (purpose << 56) | (step << 32) | (layer << 16) | replica
    return np.random.Generator(np.random.Philox(key=[int(seed) & ((1 << 64) - 1), k1]))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def layer_sigmas(layout: Layout, seed: int = 0) -> np.ndarray:
    """sigma_l, log-uniform in [1e-4, 1e-1], one draw per layer (float64)."""
    out = np.empty(layout.n_layers)
    for l in range(layout.n_layers):
        u = _rng(seed, _P_SIGMA, 0, l).random()
        out[l] = 10.0 ** (-4.0 + 3.0 * u)
    return out


def init_weights(layout: Layout, seed: int = 0, perturb_bn: bool = False) -> np.ndarray:
    """fp32 weights [n_flat]; padding between layers is zero."""
    w = np.zeros(layout.n_flat, np.float32)
    for l, t in enumerate(layout.tensors):
        o, n = int(layout.offsets[l]), int(layout.numels[l])
        g = _rng(seed, _P_WEIGHT, 0, l)
        if t.kind in ("conv", "fc"):
            w[o:o + n] = g.standard_normal(n, dtype=np.float32) * np.float32(np.sqrt(2.0 / t.fan_in))
        elif t.kind == "bias":
            b = 1.0 / np.sqrt(t.fan_in)
            w[o:o + n] = g.uniform(-b, b, n).astype(np.float32)
        elif t.kind == "bn_weight":
            w[o:o + n] = 1.0
            if perturb_bn:
                w[o:o + n] += g.standard_normal(n, dtype=np.float32) * np.float32(0.1)
        elif t.kind == "bn_bias":
            if perturb_bn:
                w[o:o + n] = g.standard_normal(n, dtype=np.float32) * np.float32(0.1)
        else:  # pragma: no cover
            raise ValueError(t.kind)
    return w


def replica_grads(layout: Layout, K: int, step: int, seed: int = 0,
                  noise: float = 0.5, dtype: str = "f32",
                  stride: int | None = None, sigmas: np.ndarray | None = None,
                  threads: int | None = None) -> np.ndarray:
    """K replica gradients for one step, shape [K, stride].

    ``dtype`` "f32" gives float32, "bf16" gives uint16 bf16 bit patterns.
    Padding between layers is zero.  ``noise`` is c, the per-replica noise
    std in units of sigma_l.
    """
    stride = layout.n_flat if stride is None else int(stride)
    if stride < layout.n_flat:
        raise ValueError("stride shorter than the layout")
    if sigmas is None:
        sigmas = layer_sigmas(layout, seed)
    if dtype == "f32":
        out = np.zeros((K, stride), np.float32)
    elif dtype == "bf16":
        out = np.zeros((K, stride), np.uint16)
    else:
        raise ValueError(dtype)

    L = layout.n_layers
    means = [None] * L

    def mean_task(l):
        n = int(layout.numels[l])
        mu = _rng(seed, _P_MEAN, step, l, _SHARED).standard_normal(n, dtype=np.float32)
        mu *= np.float32(sigmas[l])
        means[l] = mu

    def noise_task(lk):
        l, k = lk
        o, n = int(layout.offsets[l]), int(layout.numels[l])
        g = _rng(seed, _P_NOISE, step, l, k)
        buf = out[k, o:o + n] if dtype == "f32" else np.empty(n, np.float32)
        g.standard_normal(n, dtype=np.float32, out=buf)
        buf *= np.float32(noise * sigmas[l])
        buf += means[l]
        if dtype == "bf16":
            out[k, o:o + n] = to_bf16_bits(buf)

    nt = threads or _threads()
    # Big tensors first keeps the pool busy until the end.
    order = sorted(range(L), key=lambda l: -int(layout.numels[l]))
    with ThreadPoolExecutor(nt) as ex:
        list(ex.map(mean_task, order))
        list(ex.map(noise_task, [(l, k) for l in order for k in range(K)]))
    return out
