"""Why the parameter tolerance carries the previous value (CPU tier).

The parity harness checks every element of w and m against the float64
oracle within 1e-5 * max(|y|, rms_l(y), |y_prev|), y_prev being the oracle's
value before the step.  The |y_prev| term is there because a new w or m is a
sum whose largest term has the size of the previous value, and an fp32 sum
is rounded relative to its largest term: where the terms cancel, any fp32
implementation of the momentum step misses a bound taken relative to the
result alone.  On a layer of one element the layer-RMS guard is the result
itself and cannot help.

These tests run a plain float32 momentum-SGD step (numpy, d = g + lambda w,
m <- mu m + d, w <- w - eta m, every operation rounded to fp32) beside the
oracle on one-element layers whose new m (or new w) cancels to about 1e-4
of the previous one: the fp32 step fails the bound without |y_prev| and
passes it with it, by a wide margin.
"""
import numpy as np
import pytest

from ags_parity import check_params
from oracle import OracleAGS

LR, MU, WD = 0.1, 0.9, 5e-4
TABLE = [(0, 1, 2)]  # one element, weight decay on, no scaling


def fp32_momentum_step(w, m, g):
    """The momentum-SGD step of the wrapped optimizer in float32 arithmetic
    (no fused multiply-add: each product and sum is rounded)."""
    f = np.float32
    d = g + f(WD) * w
    m = f(MU) * m + d
    w = w - f(LR) * m
    return w.astype(np.float32), m.astype(np.float32)


def run_two_steps(w0, g1, g2_of):
    """Step 1 with g1, step 2 with g2_of(oracle state after step 1), on the
    oracle (float64) and on the float32 step; returns both states after each
    step."""
    o = OracleAGS(TABLE, 1, 1, np.array([w0], np.float32), mode="sgd", lr=LR, momentum=MU,
                  weight_decay=WD)
    w32 = np.array([w0], np.float32)
    m32 = np.zeros(1, np.float32)
    g1 = np.array([[g1]], np.float32)
    o.step(g1)
    w32, m32 = fp32_momentum_step(w32, m32, g1[0])
    w1, m1 = o.w.copy(), o.m.copy()
    g2 = np.array([[g2_of(w1[0], m1[0])]], np.float32)
    o.step(g2)
    w32b, m32b = fp32_momentum_step(w32, m32, g2[0])
    return (w1, m1), (o.w.copy(), o.m.copy()), (w32b, m32b)


def test_cancelling_momentum_needs_the_previous_value():
    # m2 = mu m1 + g2 + lambda w1 is made to cancel to ~1e-4 of mu m1.
    (w1, m1), (w2, m2), (w32, m32) = run_two_steps(
        1.0, 0.3, lambda w1, m1: -(MU * m1 + WD * w1) + 1e-4 * MU * m1)
    assert abs(m2[0]) < 2e-4 * abs(m1[0])
    err = abs(float(m32[0]) - m2[0])
    # fails the bound relative to the result (and to the one-element RMS) ...
    assert err > 1e-5 * abs(m2[0])
    with pytest.raises(AssertionError):
        check_params(m32, m2, TABLE, "m")
    # ... and passes with the previous value, with room to spare
    assert err <= 1e-5 * abs(m1[0])
    assert check_params(m32, m2, TABLE, "m", y_prev=m1) < 0.05


def test_cancelling_weight_needs_the_previous_value():
    # w1 = w0 - eta m1 is made to cancel to ~1e-4 of w0 (m1 = g1 + lambda w0).
    w0 = 0.03
    g1 = (w0 * (1 - 1e-4)) / LR - WD * w0
    o = OracleAGS(TABLE, 1, 1, np.array([w0], np.float32), mode="sgd", lr=LR, momentum=MU,
                  weight_decay=WD)
    w_prev = o.w.copy()
    o.step(np.array([[g1]], np.float32))
    w32, _ = fp32_momentum_step(np.array([w0], np.float32), np.zeros(1, np.float32),
                                np.array([g1], np.float32))
    w1 = o.w
    assert abs(w1[0]) < 2e-4 * abs(w_prev[0])
    err = abs(float(w32[0]) - w1[0])
    assert err > 1e-5 * abs(w1[0])
    with pytest.raises(AssertionError):
        check_params(w32, w1, TABLE, "w")
    assert check_params(w32, w1, TABLE, "w", y_prev=w_prev) < 0.05


def test_without_cancellation_the_guard_is_not_needed():
    # The same fp32 step on terms that do not cancel meets the plain bound.
    (w1, m1), (w2, m2), (w32, m32) = run_two_steps(1.0, 0.3, lambda w1, m1: 0.2)
    assert check_params(m32, m2, TABLE, "m") < 0.05
    assert check_params(w32, w2, TABLE, "w") < 0.05
