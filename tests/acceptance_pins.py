"""Pins for the oracle's acceptance rule (oracle.tolerance / oracle.check).

Every parity verdict rests on these two functions, so they are fixed here by
hand-worked values rather than by re-typing their formula.  The rule is the
workload specification's bound for an fp32 result r of the convolution whose
exact value is `out`:

    |r - out| <= 1e-4 * (1 + S / (C_in * K * K))   element by element,

S being the sum of |products| of the element's C_in*K*K terms (bias
excluded; padding taps add 0 to S but still count in the divisor).  A result
that is NaN or infinite never passes.

Each pin takes the module under test (the real `oracle`, or a copy with a
planted mistake, see test_oracle_mutants.py) and raises AssertionError on
failure.
"""
from __future__ import annotations

import numpy as np


def _raises(fn, exc):
    try:
        fn()
    except exc:
        return True
    return False


def pin_tolerance_1x1_hand(mod):
    """C_in = 2, K = 1, S = 3: divisor 2*1*1 = 2, bound 1e-4 * (1 + 1.5) = 2.5e-4."""
    t = float(mod.tolerance(np.float64(3.0), 2, 1))
    assert abs(t - 2.5e-4) <= 1e-16, t


def pin_tolerance_3x3_hand(mod):
    """C_in = 4, K = 3, S = 72: divisor 4*3*3 = 36, bound 1e-4 * (1 + 2) = 3e-4.
    (With C_in alone as the divisor it would be 1e-4 * 19 = 1.9e-3.)"""
    t = float(mod.tolerance(np.float64(72.0), 4, 3))
    assert abs(t - 3e-4) <= 1e-16, t


def pin_tolerance_zero_sum(mod):
    """S = 0 (all products zero, e.g. an all-padding window): the bound is the
    absolute floor 1e-4, never 0."""
    t = float(mod.tolerance(np.float64(0.0), 7, 5))
    assert abs(t - 1e-4) <= 1e-18, t


def pin_tolerance_elementwise(mod):
    """The bound is taken per element: S = [0, 25, 50] at C_in = 1, K = 5
    gives [1e-4, 2e-4, 3e-4]."""
    t = np.asarray(mod.tolerance(np.array([0.0, 25.0, 50.0]), 1, 5), dtype=np.float64)
    np.testing.assert_allclose(t, [1e-4, 2e-4, 3e-4], rtol=1e-12, atol=0)


def pin_check_inside_and_outside(mod):
    """Against ref = [1, -2, 0.5] with the 3x3 bound of pin_tolerance_3x3_hand
    (3e-4 per element): an error of 0.99 bound passes, 1.01 bound fails, in
    either direction from the reference."""
    ref = np.array([1.0, -2.0, 0.5])
    s = np.full(3, 72.0)
    tol = 3e-4
    for sign in (1.0, -1.0):
        ok, ratio, _ = mod.check(ref + sign * 0.99 * tol, ref, s, 4, 3)
        assert ok and 0.98 < ratio < 1.0, (sign, ok, ratio)
        ok, ratio, _ = mod.check(ref + sign * 1.01 * tol, ref, s, 4, 3)
        assert (not ok) and 1.0 < ratio < 1.02, (sign, ok, ratio)


def pin_check_exactly_at_bound(mod):
    """An error equal to the bound is accepted (the rule is <=)."""
    ref = np.zeros(2)
    s = np.array([10.0, 0.0])
    bound = np.asarray(mod.tolerance(s, 2, 1), dtype=np.float64)
    ok, ratio, _ = mod.check(ref + bound, ref, s, 2, 1)
    assert ok and ratio == 1.0, (ok, ratio)


def pin_check_below_reference(mod):
    """A result twice the bound below the reference fails (the difference is
    taken in absolute value)."""
    ref = np.array([5.0, 5.0])
    s = np.zeros(2)
    ok, ratio, i = mod.check(ref - np.array([0.0, 2e-4]), ref, s, 3, 3)
    assert not ok and i == 1 and abs(ratio - 2.0) < 1e-9, (ok, ratio, i)


def pin_check_reports_worst(mod):
    """Among errors of 0.2, 0.9 and 0.5 bound, the worst is element 1, ratio 0.9."""
    ref = np.zeros(3)
    s = np.zeros(3)
    ok, ratio, i = mod.check(np.array([0.2e-4, 0.9e-4, 0.5e-4]), ref, s, 1, 1)
    assert ok and i == 1 and abs(ratio - 0.9) < 1e-9, (ok, ratio, i)


def pin_check_non_finite_fails(mod):
    """NaN and +-inf results fail whatever the bound, reported as ratio inf at
    the first such element."""
    ref = np.array([1.0, 2.0, 3.0, 4.0])
    s = np.full(4, 1e6)  # a huge bound: only the non-finite value can fail
    for bad in (np.nan, np.inf, -np.inf):
        r = ref.copy()
        r[2] = bad
        ok, ratio, i = mod.check(r, ref, s, 1, 3)
        assert (not ok) and ratio == float("inf") and i == 2, (bad, ok, ratio, i)


def pin_check_float32_result(mod):
    """A float32 result is compared in float64: 1 + 2^-23 (one fp32 ulp above
    1) against 1 is an error of 1.19e-7, inside the 1e-4 floor."""
    r = np.array([np.float32(1.0) + np.float32(2.0 ** -23)], dtype=np.float32)
    ok, ratio, _ = mod.check(r, np.ones(1), np.zeros(1), 1, 1)
    assert ok and abs(ratio - 2.0 ** -23 / 1e-4) < 1e-9, (ok, ratio)


def pin_check_shape_mismatch(mod):
    """Results and references of different sizes are an error, not a broadcast."""
    assert _raises(lambda: mod.check(np.zeros(4), np.zeros(1), np.zeros(1), 1, 1), ValueError)
    assert _raises(lambda: mod.check(np.zeros((2, 3)), np.zeros(5), np.zeros(5), 1, 1), ValueError)


def pin_check_empty(mod):
    """No elements: nothing to reject."""
    ok, _, _ = mod.check(np.zeros(0), np.zeros(0), np.zeros(0), 3, 3)
    assert ok


ALL_ACCEPTANCE_PINS = [pin_tolerance_1x1_hand, pin_tolerance_3x3_hand, pin_tolerance_zero_sum,
                       pin_tolerance_elementwise, pin_check_inside_and_outside, pin_check_exactly_at_bound,
                       pin_check_below_reference, pin_check_reports_worst, pin_check_non_finite_fails,
                       pin_check_float32_result, pin_check_shape_mismatch, pin_check_empty]
