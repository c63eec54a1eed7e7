"""The parity checker (`oracle.compare`, `gpu_helpers.assert_close`) against its pins, and planted
mistakes in it that the pins must catch: each mutation is a plausible slip that would let GPU
parity tests pass vacuously or report wrong statistics."""
import numpy as np
import pytest

import oracle
from compare_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_compare_pin(pin):
    pin()


_orig = oracle.compare


def _stats(g, ref, mask, diff_fn=lambda g, r: np.abs(g - r), ulp_shift=7):
    diff = diff_fn(g[mask], ref[mask])
    r = ref[mask]
    if diff.size == 0:
        return {"max_abs": 0.0, "mean_abs": 0.0, "max_ulp": 0.0, "n": 0, "nonfinite_gpu": 0}
    ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(r), 2.0 ** -126))) - ulp_shift)
    return {"max_abs": float(diff.max()), "mean_abs": float(diff.mean()), "max_ulp": float((diff / ulp).max()),
            "n": int(diff.size), "nonfinite_gpu": int((~np.isfinite(g[mask])).sum())}


def _mask_by_gpu_finite(gpu_bits, ref):
    g = oracle.bf16_bits_to_f64(gpu_bits)
    return _stats(g, ref, np.isfinite(g) & np.isfinite(ref))


def _nan_to_zero_diff(gpu_bits, ref):
    g = oracle.bf16_bits_to_f64(gpu_bits)
    return _stats(g, ref, np.isfinite(ref), diff_fn=lambda a, b: np.nan_to_num(np.abs(a - b)))


def _signed_max(gpu_bits, ref):
    g = oracle.bf16_bits_to_f64(gpu_bits)
    st = _stats(g, ref, np.isfinite(ref))
    m = np.isfinite(ref)
    if m.any():
        st["max_abs"] = float((g[m] - ref[m]).max())
    return st


def _mean_over_all(gpu_bits, ref):
    st = _orig(gpu_bits, ref)
    if st["n"]:
        st["mean_abs"] = st["mean_abs"] * st["n"] / np.asarray(ref).size
        st["n"] = int(np.asarray(ref).size)
    return st


def _ulp_off_by_one(gpu_bits, ref):
    g = oracle.bf16_bits_to_f64(gpu_bits)
    return _stats(g, ref, np.isfinite(ref), ulp_shift=8)


def _against_rounded_reference(gpu_bits, ref):
    return _orig(gpu_bits, oracle.bf16_bits_to_f64(oracle.f64_to_bf16_bits(ref)))


def _empty_reports_one(gpu_bits, ref):
    st = _orig(gpu_bits, ref)
    if st["n"] == 0:
        st["n"] = 1
    return st


MUTATIONS = {
    "mask_by_gpu_finiteness": _mask_by_gpu_finite,
    "nan_difference_as_zero": _nan_to_zero_diff,
    "signed_max": _signed_max,
    "mean_over_unselected_entries": _mean_over_all,
    "ulp_exponent_off_by_one": _ulp_off_by_one,
    "reference_rounded_to_bf16": _against_rounded_reference,
    "empty_selection_counted": _empty_reports_one,
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_compare_mutation_is_caught(name, monkeypatch):
    monkeypatch.setattr(oracle, "compare", MUTATIONS[name])
    failed = []
    for pin in ALL_PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, "mutation %s passed every pin" % name


def _bound_full_ulp(ref_o, vmax):
    import gpu_helpers
    return np.maximum(gpu_helpers.MAX_ABS, gpu_helpers.bf16_ulp(ref_o) + vmax * 2.0 ** -8 + 1e-4)


def _bound_without_weights(ref_o, vmax):
    import gpu_helpers
    return np.maximum(gpu_helpers.MAX_ABS, 0.5 * gpu_helpers.bf16_ulp(ref_o) + 1e-4)


def _bound_weights_half(ref_o, vmax):
    import gpu_helpers
    return np.maximum(gpu_helpers.MAX_ABS, 0.5 * gpu_helpers.bf16_ulp(ref_o) + vmax * 2.0 ** -9 + 1e-4)


@pytest.mark.parametrize("fn", [_bound_full_ulp, _bound_without_weights, _bound_weights_half],
                         ids=lambda f: f.__name__)
def test_peaked_bound_mutation_is_caught(fn, monkeypatch):
    """A stress bound with a whole ulp for the output rounding, without the bf16-weight term, or
    with that term at half its size, must fail a pin."""
    import gpu_helpers
    import compare_pins
    monkeypatch.setattr(gpu_helpers, "peaked_bound", fn)
    with pytest.raises(AssertionError):
        compare_pins.pin_peaked_bound()
