"""The library's planner (include/ags_plan.h, through its binding) against the
float64 planner oracle, on the CPU: the fit of Eq. (2), Eq. (3), Eq. (4),
Kneedle and the selection policy, plus argument errors."""
import itertools
import math

import numpy as np
import pytest

from oracle import plan_oracle as po
from paper_2603_18112_amd import _build, ags, plan
import os

ALL = po.TERM_INTERCEPT | po.TERM_COMPUTE | po.TERM_SYNC


@pytest.fixture(scope="module", autouse=True)
def lib():
    if not os.path.exists(_build.LIB):
        _build.build()
    return ags.load_library()


def _close(x, y, rtol=1e-9, scale=1.0):
    return abs(x - y) <= rtol * max(abs(y), scale)


TERM_SETS = [ALL, po.TERM_INTERCEPT | po.TERM_SYNC, po.TERM_INTERCEPT | po.TERM_COMPUTE,
             po.TERM_COMPUTE | po.TERM_SYNC, po.TERM_SYNC, po.TERM_COMPUTE]


@pytest.mark.parametrize("sync", ["ring", "ps"])
@pytest.mark.parametrize("terms", TERM_SETS)
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_fit_matches_oracle(sync, terms, seed):
    rng = np.random.default_rng(seed)
    samples = [(int(n), float(b), float(0.01 + 0.002 * b + 0.05 * po.sync_term(n, sync)
                                          + rng.normal(0, 0.004)))
               for n in (1, 2, 4, 8, 16) for b in rng.uniform(8, 512, 3)]
    m = plan.ags_plan_fit(samples, sync, terms)
    o = po.fit(samples, sync, terms)
    scale = max(abs(o["c0"]), abs(o["c_compute"]) * 512, abs(o["c_sync"]) * 16, 1e-3)
    assert _close(m.c0, o["c0"], 1e-9, scale)
    assert _close(m.c_compute * 512, o["c_compute"] * 512, 1e-9, scale)
    assert _close(m.c_sync * 16, o["c_sync"] * 16, 1e-9, scale)
    assert _close(m.rms_residual, o["rms_residual"], 1e-9, scale)
    assert m.n_samples == len(samples) and m.terms == terms


def test_partial_search_extremes_match_oracle():
    full = [(n, b, 0.02 + 0.001 * b + 0.3 * (1 - 1 / n)) for n in (2, 4, 8, 16)
            for b in (64, 128, 256, 512)]
    part = [s for s in full if s[0] in (2, 16) and s[1] in (64, 512)]
    for samples in (full, part):
        m = plan.ags_plan_fit(samples, "ring")
        o = po.fit(samples, "ring", ALL)
        for k in ("c0", "c_compute", "c_sync"):
            assert _close(getattr(m, k), o[k], 1e-10, 1e-3), k


@pytest.mark.parametrize("samples,sync,terms", [
    ([(4, b, 0.1 * b) for b in (1, 2, 3)], "ring", ALL),            # one cluster size
    ([(n, 8, 0.1 * n) for n in (1, 2, 3)], "none", ALL),            # no sync term exists
    ([(n, 8.0, 0.1 * n) for n in (1, 2, 3)], "ps", po.TERM_INTERCEPT | po.TERM_COMPUTE),  # b constant
    ([(1, 1, 1.0)], "ring", ALL),                                   # fewer samples than terms
    ([(0, 1, 1.0), (2, 1, 1.0), (4, 2, 1.0)], "ring", ALL),         # nodes < 1
    ([(1, -1, 1.0), (2, 1, 1.0), (4, 2, 1.0)], "ring", ALL),        # b < 0
    ([(1, 1, math.nan), (2, 1, 1.0), (4, 2, 1.0)], "ring", ALL),    # t not finite
    ([(1, 1, 1.0), (2, 1, 1.0), (4, 2, 1.0)], "ring", 0),           # no terms
    ([(1, 1, 1.0), (2, 1, 1.0), (4, 2, 1.0)], "ring", 8),           # unknown term
])
def test_fit_argument_errors(samples, sync, terms):
    with pytest.raises(ags.AGSError) as e:
        plan.ags_plan_fit(samples, sync, terms)
    assert e.value.status == ags.AGS_E_ARG
    assert ags.ags_last_error(None)


def test_time_cost_and_step_time_match_oracle():
    rng = np.random.default_rng(3)
    for sync in ("ring", "ps", "none"):
        samples = [(n, b, 0.05 + 0.001 * b + 0.02 * po.sync_term(n, sync) + rng.normal(0, 1e-3))
                   for n in (1, 2, 8, 32) for b in (16, 64, 256)]
        terms = ALL if sync != "none" else po.TERM_INTERCEPT | po.TERM_COMPUTE
        m = plan.ags_plan_fit(samples, sync, terms)
        om = m.as_dict()
        for n, B in itertools.product((1, 3, 16, 64), (64, 1000, 8192)):
            assert _close(plan.ags_plan_step_time(m, n, B / n), po.step_time(om, n, B / n, sync), 1e-14)
            T, C = plan.ags_plan_time_cost(m, n, B, 90, 1.28e6, 2.48)
            oT, oC = po.time_cost(om, n, B, 90, 1.28e6, 2.48, sync)
            assert _close(T, oT, 1e-14) and _close(C, oC, 1e-14)


def test_max_local_batch_matches_oracle():
    for cap, st, per in ((288.0, 40.0, 0.75), (80.0, 79.9, 0.05), (16.0, 20.0, 1.0), (1e3, 0.0, 3.0),
                         (20.0, 20.0, 1.0), (20.5, 20.0, 0.25)):
        assert plan.ags_plan_max_local_batch(cap, st, per) == po.max_local_batch(cap, st, per)
    with pytest.raises(ags.AGSError):
        plan.ags_plan_max_local_batch(10.0, 1.0, 0.0)


def _curves():
    x = np.linspace(0, 1, 101)
    rng = np.random.default_rng(4)
    yield x, np.sqrt(x), "concave_inc"
    yield x, 1 - (1 - x) ** 2, "concave_inc"
    yield x, np.sqrt(1 - x), "concave_dec"
    yield x, 1 - np.sqrt(1 - x), "convex_inc"
    yield np.linspace(0, 1, 1001), np.exp(-5 * np.linspace(0, 1, 1001)), "convex_dec"
    Bs = np.array([2.0 ** k for k in range(4, 15)])
    yield Bs, 1 / Bs + 0.001, "convex_dec"
    for p in (0.2, 0.5, 2.0, 5.0):
        yield x, x ** p, ("concave_inc" if p < 1 else "convex_inc")
        yield x, (1 - x) ** p, ("concave_dec" if p < 1 else "convex_dec")
    for _ in range(20):
        xs = np.sort(rng.uniform(0, 10, 40))
        xs = np.unique(xs)
        y = np.exp(-xs / rng.uniform(0.5, 3)) + rng.normal(0, 0.01, len(xs))
        yield xs, y, "convex_dec"
        yield xs, -y, "concave_inc"
    x8 = np.arange(9) / 8.0                 # exact threshold tie and plateau
    yield x8, x8 + np.array([0, 0.25, 0.125, 0.25, 0, 0, 0, 0, 0]), "concave_inc"
    yield x8, x8 + np.array([0, 0.25, 0.25, 0, 0, 0, 0, 0, 0]), "concave_inc"
    yield x, 2 * x, "concave_inc"
    yield x, np.ones_like(x), "convex_dec"
    yield x[:2], x[:2], "concave_inc"


def test_knee_matches_oracle():
    n = 0
    for x, y, shape in _curves():
        for s in (0.0, 0.5, 1.0, 3.0):
            assert plan.ags_plan_knee(x, y, shape, s) == po.knee(x, y, shape, s), (shape, s)
            n += 1
    assert n > 200


def test_knee_argument_errors():
    with pytest.raises(ags.AGSError):
        plan.ags_plan_knee([0, 2, 1], [0, 1, 2])            # x not increasing
    with pytest.raises(ags.AGSError):
        plan.ags_plan_knee([0, 1, 2], [0, math.inf, 2])     # not finite
    with pytest.raises(ags.AGSError):
        plan.ags_plan_knee([0, 1, 2], [0, 1, 2], sensitivity=-1)


@pytest.mark.parametrize("objective", ["time", "cost", "knee"])
def test_select_matches_oracle(objective):
    rng = np.random.default_rng(5)
    for trial in range(10):
        sync = ("ring", "ps")[trial % 2]
        m = plan.ags_plan_fit([(n, b, 0.2 + 0.002 * b + rng.uniform(0.01, 0.3) * po.sync_term(n, sync))
                               for n in (1, 2, 4, 8, 16) for b in (32, 64, 128, 256)], sync)
        om = m.as_dict()
        if objective == "knee":
            N = int(rng.choice([2, 4, 8, 16]))
            cands = [(N, float(2 ** k)) for k in range(5, 16)]
        else:
            cands = [(int(n), float(B)) for n in (1, 2, 4, 8, 16) for B in (256, 1024, 4096)]
        max_local = float(rng.choice([64.0, 512.0, math.inf]))
        i, T, C = plan.ags_plan_select(m, cands, 90, 1.28e6, 2.48, max_local, objective)
        oi, oT, oC = po.select(om, cands, 90, 1.28e6, 2.48, sync, objective, max_local)
        assert i == oi, (trial, i, oi)
        for a, b in zip(T, oT):
            assert (math.isinf(a) and math.isinf(b)) or _close(a, b, 1e-13)
        for a, b in zip(C, oC):
            assert (math.isinf(a) and math.isinf(b)) or _close(a, b, 1e-13)


def test_select_cost_tie_takes_the_first_candidate():
    # Constant step time: the two candidates cost exactly the same.
    m = plan.ags_plan_fit([(1, 32.0, 0.5), (1, 64.0, 0.5)], "none", po.TERM_INTERCEPT)
    for cands in ([(1, 128.0), (2, 256.0)], [(2, 256.0), (1, 128.0)]):
        i, T, C = plan.ags_plan_select(m, cands, 2, 1e5, 3.0, math.inf, "cost")
        oi, _, oC = po.select(m.as_dict(), cands, 2, 1e5, 3.0, "none", "cost")
        assert C[0] == C[1] and oC[0] == oC[1] and i == oi == 0


def test_select_argument_errors():
    m = plan.ags_plan_fit([(1, 8, 1.0), (2, 8, 1.5), (1, 16, 2.0)], "ring")
    with pytest.raises(ags.AGSError):
        plan.ags_plan_select(m, [(2, 64.0), (4, 128.0)], 1, 1, 1, objective="knee")  # two sizes
    with pytest.raises(ags.AGSError):
        plan.ags_plan_select(m, [(2, 128.0), (2, 64.0)], 1, 1, 1, objective="knee")  # B falls
    with pytest.raises(ags.AGSError):
        plan.ags_plan_select(m, [(0, 64.0)], 1, 1, 1)
    i, T, C = plan.ags_plan_select(m, [], 1, 1, 1)
    assert i is None and len(T) == 0
