"""Pins of the parity checker itself: `oracle.compare` (the error statistics every GPU parity
assertion reads) and `gpu_helpers.assert_close` (the pass/fail rule built on them).

Each pin feeds hand-built GPU bit patterns and float64 reference values whose statistics are
known in closed form: exact bf16 values against references offset by chosen amounts, NaN and Inf
on either side, an empty selection, and references rounded to bf16 (at most half an ulp away).
The bf16 values used here are built from their sign, exponent and mantissa fields, not through
the oracle's own conversion routines.  `ALL_PINS` lists them for the planted-mistake tests.
"""
from __future__ import annotations

import math

import numpy as np

import oracle
from gpu_helpers import LSE_ABS, MAX_ABS, MEAN_ABS, assert_close


def bf16(sign: int, exp: int, mant: int) -> int:
    """Bit pattern of (-1)^sign * 2^exp * (1 + mant / 128), a normal bf16 number."""
    assert 0 <= mant < 128 and -126 <= exp <= 127
    return (sign << 15) | ((exp + 127) << 7) | mant


def bf16_value(sign: int, exp: int, mant: int) -> float:
    return (-1.0) ** sign * 2.0 ** exp * (1.0 + mant / 128.0)


NAN_BITS = 0x7FC0
INF_BITS = 0x7F80


def _raises(fn) -> bool:
    try:
        fn()
    except AssertionError:
        return True
    return False


def pin_known_offsets():
    """Four exact bf16 outputs against references offset by 0.011, 0, -0.004, 0.002: max-abs
    0.011, mean-abs 0.017 / 4, all four compared, nothing non-finite."""
    vals = [(0, 0, 0), (0, 1, 0), (1, -1, 0), (0, -2, 64)]          # 1, 2, -0.5, 0.375
    g = np.array([bf16(*v) for v in vals], np.uint16)
    x = np.array([bf16_value(*v) for v in vals])
    offs = np.array([0.011, 0.0, -0.004, 0.002])
    st = oracle.compare(g, x - offs)
    assert st["n"] == 4, st
    assert abs(st["max_abs"] - 0.011) < 1e-15, st
    assert abs(st["mean_abs"] - 0.017 / 4) < 1e-15, st
    assert st["nonfinite_gpu"] == 0, st


def pin_max_is_absolute():
    """The largest deviation is negative (GPU below the reference): max-abs still reports it."""
    g = np.array([bf16(0, 0, 0), bf16(0, 0, 0)], np.uint16)          # 1, 1
    st = oracle.compare(g, np.array([1.02, 1.001]))
    assert abs(st["max_abs"] - 0.02) < 1e-15, st
    assert abs(st["mean_abs"] - 0.0105) < 1e-15, st


def pin_ulp_units():
    """Error in bf16 ulps of the reference: ulp(x) = 2^(floor(log2 |x|) - 7).  The bf16
    neighbours 4 and 4 + 2^-5 are one ulp of 4 apart; 3.5 against 3.5 + 2^-7 is half an ulp of
    3.5 (ulp 2^-6)."""
    g = np.array([bf16(0, 2, 1)], np.uint16)                          # 4 + 2^-5
    st = oracle.compare(g, np.array([4.0]))
    assert abs(st["max_ulp"] - 1.0) < 1e-12, st
    g = np.array([bf16(0, 1, 96)], np.uint16)                         # 3.5
    st = oracle.compare(g, np.array([3.5 + 2.0 ** -7]))
    assert abs(st["max_ulp"] - 0.5) < 1e-12, st


def pin_gpu_nan_counts():
    """A NaN or Inf GPU output at a finite reference is counted, the max-abs statistic on its own
    fails the bar too (a non-finite error is never reported as small), and assert_close fails even
    though every other element is exact."""
    for bad in (NAN_BITS, INF_BITS, INF_BITS | 0x8000):
        g = np.array([bf16(0, 0, 0), bad, bf16(0, 1, 0)], np.uint16)
        ref = np.array([1.0, 0.5, 2.0])
        st = oracle.compare(g, ref)
        assert st["nonfinite_gpu"] == 1 and st["n"] == 3, st
        assert not (st["max_abs"] <= MAX_ABS), st
        assert _raises(lambda: assert_close(g, ref, what="planted non-finite")), hex(bad)


def pin_reference_nan_excluded():
    """Reference entries that are NaN (rows the oracle did not compute) are left out of n and of
    the mean, whatever the GPU holds there."""
    g = np.array([bf16(0, 0, 0), NAN_BITS, bf16(0, 0, 0), bf16(0, 1, 0)], np.uint16)
    ref = np.array([1.0 - 0.008, np.nan, np.nan, 2.0])
    st = oracle.compare(g, ref)
    assert st["n"] == 2, st
    assert st["nonfinite_gpu"] == 0, st
    assert abs(st["max_abs"] - 0.008) < 1e-15, st
    assert abs(st["mean_abs"] - 0.004) < 1e-15, st


def pin_empty_selection():
    """No finite reference at all: nothing is compared, and assert_close refuses to pass."""
    g = np.array([bf16(0, 0, 0)] * 3, np.uint16)
    ref = np.full(3, np.nan)
    st = oracle.compare(g, ref)
    assert st["n"] == 0, st
    assert _raises(lambda: assert_close(g, ref, what="empty"))


def pin_rounded_reference_half_ulp():
    """GPU values that are the reference rounded to the nearest bf16 lie within half an ulp of it.
    The rounding here works on the exponent and a scaled mantissa (numpy's round is half to
    even), independently of the oracle's conversion."""
    rng = np.random.default_rng(17)
    x = rng.standard_normal(4000) * np.exp2(rng.integers(-6, 6, 4000))
    e = np.floor(np.log2(np.abs(x)))
    ulp = np.exp2(e - 7)
    r = np.round(x / ulp) * ulp                                        # nearest multiple, ties even
    # r is a bf16 value (it may carry into the next binade, still representable): take its bits
    g = (r.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal((g.astype(np.uint32) << 16).view(np.float32).astype(np.float64), r)
    st = oracle.compare(g, x)
    assert st["max_ulp"] <= 0.5 + 1e-12, st
    assert st["max_abs"] <= 0.5 * ulp.max() + 1e-15, st
    assert st["n"] == x.size and st["nonfinite_gpu"] == 0


def pin_assert_close_bars():
    """assert_close passes at the bars and fails just beyond them: one element at 0.0099 passes
    and at 0.0101 fails (max-abs 1e-2); a uniform offset of 0.0011 fails the mean bar (1e-3)."""
    assert MAX_ABS == 1e-2 and MEAN_ABS == 1e-3 and LSE_ABS == 1e-3
    n = 64
    g = np.array([bf16(0, 0, 0)] * n, np.uint16)                      # all 1.0
    ref = np.ones(n)
    ref[5] = 1.0 - 0.0099
    assert_close(g, ref, what="at the max bar")
    ref[5] = 1.0 - 0.0101
    assert _raises(lambda: assert_close(g, ref, what="past the max bar"))
    assert _raises(lambda: assert_close(g, np.full(n, 1.0 - 0.0011), what="past the mean bar"))
    assert_close(g, np.full(n, 1.0 - 0.0009), what="under the mean bar")


def pin_peaked_bound():
    """The stress-case bar: max(1e-2, half an ulp of the reference + 2^-8 vmax + 1e-4).  With
    vmax = 5: at 3.0 (ulp 2^-6) the bar is 2^-7 + 5/256 + 1e-4 = 0.027444, so 0.0274 passes and
    0.0275 fails; at 6.0 (ulp 2^-5) it is 2^-6 + 5/256 + 1e-4 = 0.035256, so 0.0352 passes and
    0.0353 fails.  With vmax = 2 at 2^-5 the bound (0.00797) is below 1e-2, so the plain bar
    holds: 0.0099 passes and 0.0101 fails."""
    n = 400
    ones = [bf16(0, 0, 0)] * (n - 1)
    for top, vmax, err_ok, err_bad in (((0, 1, 64), 5.0, 0.0274, 0.0275), ((0, 2, 64), 5.0, 0.0352, 0.0353),
                                       ((0, -5, 0), 2.0, 0.0099, 0.0101)):
        g = np.array([bf16(*top)] + ones, np.uint16)
        ref = np.ones(n)
        ref[0] = bf16_value(*top) - err_ok
        assert_close(g, ref, what="peaked ok", peaked_vmax=vmax)
        ref[0] = bf16_value(*top) - err_bad
        assert _raises(lambda: assert_close(g, ref, what="peaked bad", peaked_vmax=vmax))
    g = np.array([bf16(0, 1, 64)] + ones, np.uint16)
    ref = np.ones(n)
    ref[0] = 3.0 - 0.0274
    assert _raises(lambda: assert_close(g, ref, what="no peaked bound"))


def pin_lse_bar():
    """The LSE bar: 9e-4 off passes, 1.1e-3 off fails, and a NaN GPU LSE at a finite reference
    fails."""
    g = np.array([bf16(0, 0, 0)] * 4, np.uint16)
    ref = np.ones(4)
    lref = np.array([2.0, 3.0, 4.0, 5.0])
    assert_close(g, ref, (lref + 9e-4).astype(np.float32), lref, what="lse ok")
    assert _raises(lambda: assert_close(g, ref, (lref + 1.1e-3).astype(np.float32), lref, what="lse off"))
    bad = lref.astype(np.float32)
    bad[2] = np.nan
    assert _raises(lambda: assert_close(g, ref, bad, lref, what="lse nan"))


ALL_PINS = [pin_known_offsets, pin_max_is_absolute, pin_ulp_units, pin_gpu_nan_counts,
            pin_reference_nan_excluded, pin_empty_selection, pin_rounded_reference_half_ulp,
            pin_assert_close_bars, pin_peaked_bound, pin_lse_bar]

assert math.isclose(bf16_value(0, -2, 64), 0.375)
