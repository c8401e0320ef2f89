"""Plain float64 oracle of the host-side planner (test infrastructure only).

Only the test-suite and the benchmark's planning leg use this module; the
library's planner (``ags_plan_*``) never calls it.  Each function follows
the passage it implements (Tula, arXiv 2603.18112):

* step-time model, Eq. (2a)-(2c), Sec. III-A:
    t_step = c0 + c_compute * b + c_sync * s(N)
  with b the per-node batch, s(N) = N for a centralized parameter server,
  1 - 1/N for ring all-reduce (0 for no synchronisation); c0 is an optional
  intercept for fixed per-step costs, the other terms are proportional as in
  the paper.  Fitted by least squares on profiled samples (full search: all
  profiled configurations; partial search: the extremes only);
* memory bound, Eq. (3): M = M_static + m_per_sample * b <= capacity, with
  the parameter, gradient and optimizer terms static and the activation and
  batch terms linear in b;
* training time and cost, Eq. (4a), (4b): T = (E D / B) t_step,
  C = T N p (p per node per hour, T in hours);
* selection: minimum T, minimum C, or the knee of the T-B curve with the
  Kneedle algorithm (Satopaa, Albrecht, Irwin, Raghavan, "Finding a
  'Kneedle' in a Haystack", ICDCS workshops 2011), written from that paper.
"""
from __future__ import annotations

import math

import numpy as np

SYNC = {"none": 0, "ring": 1, "ps": 2}
TERM_INTERCEPT, TERM_COMPUTE, TERM_SYNC = 1, 2, 4
SHAPES = {"concave_inc": 0, "concave_dec": 1, "convex_inc": 2, "convex_dec": 3}


def sync_term(nodes: int, sync: str) -> float:
    """s(N) of Eq. (2c)."""
    if sync == "ps":
        return float(nodes)
    if sync == "ring":
        return 1.0 - 1.0 / nodes
    return 0.0


def design_row(nodes, local_batch, sync, terms):
    row = []
    if terms & TERM_INTERCEPT:
        row.append(1.0)
    if terms & TERM_COMPUTE:
        row.append(float(local_batch))
    if terms & TERM_SYNC:
        row.append(sync_term(nodes, sync))
    return row


def fit(samples, sync="ring", terms=TERM_INTERCEPT | TERM_COMPUTE | TERM_SYNC):
    """Least-squares fit of Eq. (2).  samples: iterable of (N, b, t_step).
    Returns dict(c0, c_compute, c_sync, rms_residual)."""
    X = np.array([design_row(n, b, sync, terms) for n, b, _ in samples], dtype=np.float64)
    y = np.array([t for _, _, t in samples], dtype=np.float64)
    coef, *_ = np.linalg.lstsq(X, y, rcond=None)
    r = y - X @ coef
    out = {"c0": 0.0, "c_compute": 0.0, "c_sync": 0.0}
    i = 0
    for bit, name in ((TERM_INTERCEPT, "c0"), (TERM_COMPUTE, "c_compute"), (TERM_SYNC, "c_sync")):
        if terms & bit:
            out[name] = float(coef[i])
            i += 1
    out["rms_residual"] = float(math.sqrt(np.mean(r * r)))
    return out


def step_time(model, nodes, local_batch, sync="ring"):
    return model["c0"] + model["c_compute"] * local_batch + model["c_sync"] * sync_term(nodes, sync)


def time_cost(model, nodes, global_batch, epochs, dataset_size, price_per_node_hour, sync="ring"):
    """Eq. (4a), (4b): seconds of training and its cost."""
    t = step_time(model, nodes, global_batch / nodes, sync)
    T = epochs * dataset_size / global_batch * t
    C = T / 3600.0 * nodes * price_per_node_hour
    return T, C


def max_local_batch(capacity, m_static, m_per_sample):
    """Largest b with M_static + m_per_sample * b <= capacity (Eq. (3)); 0
    when not even the static memory fits."""
    return max(0, math.floor((capacity - m_static) / m_per_sample))


def knee(x, y, shape="convex_dec", sensitivity=1.0):
    """Kneedle: index of the knee of (x, y), or None.

    Steps of the method: normalise both axes to [0, 1]; bring the curve to
    the concave increasing form (flip y for a convex curve, flip x for a
    decreasing concave one, both for an increasing convex one); take the
    difference curve y' - x'; each of its local maxima sets a threshold
    that much below it, sensitivity times the mean spacing of the
    normalised x; a local maximum is a knee if the difference curve falls
    below its threshold before the next local maximum.
    """
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    n = len(x)
    if n < 3 or y.max() == y.min():
        return None
    xn = (x - x[0]) / (x[-1] - x[0])
    yn = (y - y.min()) / (y.max() - y.min())
    flip_x = shape in ("concave_dec", "convex_inc")
    flip_y = shape in ("convex_dec", "convex_inc")
    xt = 1.0 - xn if flip_x else xn
    yt = 1.0 - yn if flip_y else yn
    order = list(range(n - 1, -1, -1)) if flip_x else list(range(n))
    xs = [xt[i] for i in order]
    d = [yt[i] - xt[i] for i in order]
    step = sensitivity * (xs[-1] - xs[0]) / (n - 1)
    threshold = None
    lmx = None
    for j in range(1, n):
        if j < n - 1 and d[j - 1] < d[j] >= d[j + 1]:
            lmx = j
            threshold = d[j] - step
            continue
        if threshold is not None and d[j] < threshold:
            return order[lmx]
    return None


def select(model, candidates, epochs, dataset_size, price_per_node_hour, sync="ring",
           objective="time", max_local=math.inf, sensitivity=1.0):
    """Pick a candidate (N, B): 'time' = min T, 'cost' = min C (first on a
    tie), 'knee' = Kneedle knee of T over B (one cluster size, increasing
    B).  Candidates whose per-node batch exceeds max_local are infeasible.
    Returns (index or None, [T], [C])."""
    Ts, Cs, feas = [], [], []
    for n, B in candidates:
        ok = B / n <= max_local
        T, C = time_cost(model, n, B, epochs, dataset_size, price_per_node_hour, sync)
        Ts.append(T if ok else math.inf)
        Cs.append(C if ok else math.inf)
        feas.append(ok)
    idx = [i for i, ok in enumerate(feas) if ok]
    if not idx:
        return None, Ts, Cs
    if objective == "time":
        return min(idx, key=lambda i: (Ts[i], i)), Ts, Cs
    if objective == "cost":
        return min(idx, key=lambda i: (Cs[i], i)), Ts, Cs
    xs = [candidates[i][1] for i in idx]
    k = knee(xs, [Ts[i] for i in idx], "convex_dec", sensitivity)
    return (None if k is None else idx[k]), Ts, Cs
