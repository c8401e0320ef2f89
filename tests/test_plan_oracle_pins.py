"""Pins of the planner oracle (Eq. (2)-(4), Kneedle) against closed forms,
hand-worked numbers and properties that do not come from the oracle."""
import math

import numpy as np
import pytest

from oracle import plan_oracle as po

ALL = po.TERM_INTERCEPT | po.TERM_COMPUTE | po.TERM_SYNC


def _grid_samples(c0, cc, cs, sync, nodes=(1, 2, 4, 8, 16), batches=(32, 64, 128, 256)):
    return [(n, b, c0 + cc * b + cs * po.sync_term(n, sync)) for n in nodes for b in batches]


# ----------------------------------------------------------- Eq. (2) fit --


def test_fit_hand_example_exactly_determined():
    # ring: s(1) = 0, s(2) = 1/2.  c0 + 10 cc = 1; c0 + 10 cc + cs/2 = 1.5;
    # c0 + 20 cc = 2  =>  cc = 0.1, c0 = 0, cs = 1.
    m = po.fit([(1, 10, 1.0), (2, 10, 1.5), (1, 20, 2.0)], "ring", ALL)
    assert abs(m["c0"]) < 1e-12 and abs(m["c_compute"] - 0.1) < 1e-12
    assert abs(m["c_sync"] - 1.0) < 1e-12 and m["rms_residual"] < 1e-12


@pytest.mark.parametrize("sync", ["ring", "ps"])
def test_fit_recovers_noise_free_coefficients_full_and_partial(sync):
    c0, cc, cs = 0.012, 0.0021, 0.047
    full = _grid_samples(c0, cc, cs, sync)
    part = [s for s in full if s[0] in (1, 16) and s[1] in (32, 256)]
    for samples in (full, part):
        m = po.fit(samples, sync, ALL)
        assert abs(m["c0"] - c0) < 1e-12 and abs(m["c_compute"] - cc) < 1e-14
        assert abs(m["c_sync"] - cs) < 1e-12


def test_fit_residual_is_orthogonal_to_the_terms_and_order_free():
    rng = np.random.default_rng(0)
    samples = [(n, b, 0.01 + 0.002 * b + 0.05 * (1 - 1 / n) + rng.normal(0, 0.003))
               for n in (1, 2, 4, 8) for b in (16, 48, 96, 200)]
    m = po.fit(samples, "ring", ALL)
    X = np.array([[1.0, b, 1 - 1 / n] for n, b, _ in samples])
    r = np.array([t for *_, t in samples]) - X @ [m["c0"], m["c_compute"], m["c_sync"]]
    assert np.max(np.abs(X.T @ r)) < 1e-10          # normal equations
    assert abs(m["rms_residual"] - math.sqrt(np.mean(r * r))) < 1e-15
    m2 = po.fit(samples[::-1], "ring", ALL)
    for k in ("c0", "c_compute", "c_sync"):
        assert abs(m[k] - m2[k]) < 1e-12


def test_fit_term_subsets_and_sync_terms():
    # t = 3 N exactly (parameter server, proportional to N): no intercept
    m = po.fit([(n, 8, 3.0 * n) for n in (1, 2, 4)], "ps", po.TERM_SYNC)
    assert abs(m["c_sync"] - 3.0) < 1e-12 and m["c0"] == 0.0 and m["c_compute"] == 0.0
    assert po.sync_term(4, "ring") == 0.75 and po.sync_term(4, "ps") == 4.0
    assert po.sync_term(4, "none") == 0.0


# ------------------------------------------------- Eq. (3), (4): bound, T, C --


def test_time_and_cost_hand_example():
    # c_compute 1 ms per sample, ring sync 0.1 s * (1 - 1/N); N = 4, B = 1024:
    # b = 256, t = 0.256 + 0.075 = 0.331 s; E = 90 epochs of D = 1,281,167
    # samples: 112,602.568359375 steps, T = 37,271.450126953125 s; at 2.48
    # per node-hour, C = 37,271.45... / 3600 * 4 * 2.48 = 102.7035514609375.
    m = {"c0": 0.0, "c_compute": 0.001, "c_sync": 0.1}
    T, C = po.time_cost(m, 4, 1024, 90, 1281167, 2.48, "ring")
    assert abs(T - 37271.450126953125) < 1e-8
    assert abs(C - 102.7035514609375) < 1e-10


def test_memory_bound_hand_example():
    # 288 GB card, 40 GB static (parameters, gradients, optimizer state),
    # 0.75 GB per sample of activations and batch: b_max = floor(248/0.75)
    assert po.max_local_batch(288.0, 40.0, 0.75) == 330


# ------------------------------------------------------------- Kneedle --


def test_knee_concave_increasing_closed_forms():
    x = np.linspace(0, 1, 101)
    # sqrt: d/dx (sqrt(x) - x) = 0 at x = 1/4
    assert po.knee(x, np.sqrt(x), "concave_inc") == 25
    # 1 - (1 - x)^2: 2 (1 - x) = 1 at x = 1/2
    assert po.knee(x, 1 - (1 - x) ** 2, "concave_inc") == 50
    # a corner at x = 0.3
    y = np.where(x <= 0.3, x, 0.3 + 0.1 * (x - 0.3))
    assert po.knee(x, y, "concave_inc") == 30


def test_knee_convex_decreasing_exponential():
    # normalised e^{-5x}: the slope is -1 where e^{-5x} = (1 - e^{-5}) / 5
    x = np.linspace(0, 1, 1001)
    k = po.knee(x, np.exp(-5 * x), "convex_dec")
    x_star = math.log(5 / (1 - math.exp(-5))) / 5
    assert abs(x[k] - x_star) <= 0.5e-3 + 1e-12


def test_knee_mirrored_shapes():
    x = np.linspace(0, 1, 101)
    # sqrt(1 - x) is sqrt mirrored in x: its knee is at 1 - 1/4
    assert po.knee(x, np.sqrt(1 - x), "concave_dec") == 75
    # 1 - sqrt(1 - x) is sqrt mirrored in both axes: knee at 3/4 too
    assert po.knee(x, 1 - np.sqrt(1 - x), "convex_inc") == 75
    # scaling and shifting the data changes nothing (normalisation)
    assert po.knee(3 * x + 7, 5 * np.sqrt(x) - 2, "concave_inc") == 25


def test_knee_threshold_rule_and_sensitivity():
    # Difference curve (y - x on the unit square) with a small local maximum
    # at index 1 that never drops by the threshold before the larger one at
    # index 4, which does (0.1 = one mean spacing): knee at 4.  With
    # sensitivity 3 the threshold 0.3 - 0.3 = 0 is never crossed: no knee.
    x = np.linspace(0, 1, 11)
    d = np.array([0, 0.05, 0.04, 0.045, 0.3, 0.2, 0.1, 0.05, 0.02, 0.01, 0])
    assert po.knee(x, x + d, "concave_inc") == 4
    assert po.knee(x, x + d, "concave_inc", sensitivity=3.0) is None
    # a straight line has no knee, nor a constant
    assert po.knee(x, 2 * x, "concave_inc") is None
    assert po.knee(x, np.ones_like(x), "concave_inc") is None


# Exact curves on x = k/8 whose y spans [0, 1], so the normalisation is the
# identity and the difference curve d = y - x holds the chosen dyadic values.
X8 = np.arange(9) / 8.0
D_TIE = np.array([0, 0.25, 0.125, 0.25, 0, 0, 0, 0, 0])       # d meets the threshold
D_PLATEAU = np.array([0, 0.25, 0.25, 0, 0, 0, 0, 0, 0])       # a flat maximum


def test_knee_threshold_is_strict_and_plateaus_count_from_their_first_point():
    # The maximum at 1 sets the threshold 0.25 - 1/8 = 0.125; d[2] equals
    # it, which is not a fall below it, and the next maximum (3) is the knee.
    assert po.knee(X8, X8 + D_TIE, "concave_inc") == 3
    # A maximum held over two points is a local maximum at its first point.
    assert po.knee(X8, X8 + D_PLATEAU, "concave_inc") == 1


def test_memory_bound_is_zero_when_the_static_part_does_not_fit():
    assert po.max_local_batch(16.0, 20.0, 1.0) == 0
    assert po.max_local_batch(20.0, 20.0, 1.0) == 0
    assert po.max_local_batch(20.5, 20.0, 0.25) == 2


# ------------------------------------------------------------ selection --


def test_select_min_time_min_cost_and_memory_bound():
    # 1 ms per sample, ring sync 0.2 s: more nodes cut compute time but pay
    # the sync and the node-hours.
    m = {"c0": 0.0, "c_compute": 0.001, "c_sync": 0.2}
    cands = [(1, 256), (2, 256), (4, 256), (8, 256), (16, 256)]
    i, T, C = po.select(m, cands, 1, 25600, 1.0, "ring", "time")
    # t(N) = 0.256 / N + 0.2 (1 - 1/N): 0.256, 0.228, 0.214, 0.207, 0.2035
    assert i == 4
    i, T, C = po.select(m, cands, 1, 25600, 1.0, "ring", "cost")
    assert i == 0                       # one node: 100 steps * 0.256 s * 1 node
    i, T, C = po.select(m, cands, 1, 25600, 1.0, "ring", "time", max_local=100)
    assert i == 4 and math.isinf(T[0]) and math.isinf(T[1])   # b = 256, 128 > 100
    i, _, _ = po.select(m, cands, 1, 25600, 1.0, "ring", "time", max_local=1)
    assert i is None


def test_select_cost_tie_takes_the_first_candidate():
    # Constant step time: doubling N and B halves T and keeps C = T N p / 3600
    # exactly (powers of two), so both candidates cost the same.
    m = {"c0": 0.5, "c_compute": 0.0, "c_sync": 0.0}
    for cands in ([(1, 128), (2, 256)], [(2, 256), (1, 128)]):
        i, T, C = po.select(m, cands, 2, 1e5, 3.0, "none", "cost")
        assert C[0] == C[1] and i == 0


def test_select_knee_on_time_versus_batch():
    # Fixed per-step cost 1 s plus 1 ms per sample: T(B) = E D (1/B + 0.001),
    # convex decreasing.  On the grid B = 16 ... 16384 (powers of 2), the
    # normalised x = (B - 16) / 16368 and y = (1/B - 1/16384) / (1/16 -
    # 1/16384) are mirror images of each other about B = sqrt(16 * 16384) =
    # 512, so the difference curve 1 - x - y peaks there (0.9394), and two
    # points later (B = 2048: 0.869, B = 4096: 0.748) falls below the
    # threshold 0.9394 - 1/10: the knee is B = 512.
    m = {"c0": 1.0, "c_compute": 0.001, "c_sync": 0.0}
    Bs = [2 ** k for k in range(4, 15)]
    cands = [(1, B) for B in Bs]
    i, T, _ = po.select(m, cands, 1, 1e6, 1.0, "none", "knee")
    assert Bs[i] == 512
