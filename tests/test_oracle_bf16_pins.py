"""Pins of the oracle's bfloat16 helpers, which set the tolerance of every
gradient comparison: ``bf16_ulp`` (the spacing of bf16 numbers at a value's
magnitude; one ulp is the bar on dlogits) and ``f64_to_bf16_bits`` (correct
rounding to nearest even).

The spacing is checked against the gap to the next representable bf16 number,
computed from the format's fields (sign, 8-bit exponent, 7-bit fraction) with
``math.ldexp`` and no floating-point view of the bits, for every finite bit
pattern; plus hand values. Planted mistakes in the oracle's own source of the
two helpers must each fail one of these pins.
"""

import inspect
import math

import numpy as np
import pytest

import oracle


def _bf16_value(bits: int) -> float:
    """Value of a bf16 bit pattern from its fields (finite patterns only)."""
    sign = -1.0 if bits & 0x8000 else 1.0
    exp = (bits >> 7) & 0xFF
    frac = bits & 0x7F
    assert exp != 0xFF
    if exp == 0:  # subnormal: frac / 2^7 * 2^-126
        return sign * math.ldexp(frac, -126 - 7)
    return sign * math.ldexp(128 + frac, exp - 127 - 7)


def _next_up_gap(bits: int) -> float:
    """|next bf16 number away from zero| - |value| for a finite pattern whose
    magnitude is below the largest finite bf16."""
    mag = bits & 0x7FFF
    return _bf16_value(mag + 1) - _bf16_value(mag)


def _all_finite_patterns():
    mags = np.arange(0, 0x7F7F, dtype=np.uint16)  # 0 .. largest finite - 1
    return np.concatenate([mags, mags | np.uint16(0x8000)])


def test_bf16_ulp_is_the_gap_to_the_next_number_for_every_pattern():
    bits = _all_finite_patterns()
    got = oracle.bf16_ulp(bits)
    want = np.array([_next_up_gap(int(b)) for b in bits])
    assert np.array_equal(got, want)


def test_bf16_ulp_hand_values():
    def ulp_of(x):
        b = int((np.array([x], np.float32).view(np.uint32)[0] >> 16))
        assert _bf16_value(b) == x  # x is exactly a bf16 number
        return float(oracle.bf16_ulp(np.array([b], np.uint16))[0])

    assert ulp_of(1.0) == 2.0 ** -7
    assert ulp_of(1.9921875) == 2.0 ** -7      # largest bf16 below 2
    assert ulp_of(2.0) == 2.0 ** -6
    assert ulp_of(-3.0) == 2.0 ** -6
    assert ulp_of(0.0) == 2.0 ** -133
    assert ulp_of(2.0 ** -126) == 2.0 ** -133  # smallest normal
    assert ulp_of(2.0 ** -130) == 2.0 ** -133  # a subnormal
    assert ulp_of(2.0 ** -125) == 2.0 ** -132
    assert ulp_of(2.0 ** 127) == 2.0 ** 120


def test_bf16_ulp_is_the_rounding_step_of_the_rounding_helper():
    """Between two adjacent bf16 numbers a and a + ulp(a), values below the
    midpoint round to a and values above it to a + ulp(a)."""
    rng = np.random.default_rng(11)
    mags = rng.integers(1, 0x7F7E, 4000).astype(np.uint16)
    a = np.array([_bf16_value(int(m)) for m in mags])
    u = oracle.bf16_ulp(mags)
    lo = oracle.f64_to_bf16_bits(a + 0.49 * u)
    hi = oracle.f64_to_bf16_bits(a + 0.51 * u)
    assert np.array_equal(lo, mags)
    assert np.array_equal(hi, mags + np.uint16(1))


def test_rounding_helper_matches_fields_for_every_pattern():
    """f64_to_bf16_bits maps every finite bf16 value (computed from its
    fields) back to its own pattern, and ties go to the even pattern."""
    bits = _all_finite_patterns()
    vals = np.array([_bf16_value(int(b)) for b in bits])
    back = oracle.f64_to_bf16_bits(vals)
    nonzero = (bits & 0x7FFF) != 0
    assert np.array_equal(back[nonzero], bits[nonzero])
    mags = np.arange(1, 0x7F7E, 7, dtype=np.uint16)
    mid = np.array([(_bf16_value(int(m)) + _bf16_value(int(m) + 1)) / 2 for m in mags])
    want = np.where(mags % 2 == 0, mags, mags + np.uint16(1)).astype(np.uint16)
    assert np.array_equal(oracle.f64_to_bf16_bits(mid), want)


PINS = (test_bf16_ulp_is_the_gap_to_the_next_number_for_every_pattern,
        test_bf16_ulp_hand_values,
        test_bf16_ulp_is_the_rounding_step_of_the_rounding_helper,
        test_rounding_helper_matches_fields_for_every_pattern)

# One-token rewrites of the helpers' source in oracle/__init__.py.
MUTATIONS = {
    "ulp_exponent_off_by_one_up": ("bf16_ulp", "2.0 ** (e - 7)", "2.0 ** (e - 6)"),
    "ulp_exponent_off_by_one_down": ("bf16_ulp", "2.0 ** (e - 7)", "2.0 ** (e - 8)"),
    "ulp_subnormal_spacing": ("bf16_ulp", "2.0 ** -126, 2.0 ** -133", "2.0 ** -126, 2.0 ** -134"),
    "ulp_ceil_not_floor": ("bf16_ulp", "np.floor(np.log2", "np.ceil(np.log2"),
    "ulp_normal_threshold": ("bf16_ulp", "np.where(a < 2.0 ** -126", "np.where(a < 2.0 ** -124"),
    "rounding_truncates": ("f64_to_bf16_bits", "(u + half + ((u >> np.uint64(45)) & np.uint64(1)))",
                           "(u)"),
    "rounding_ties_away": ("f64_to_bf16_bits", "(u + half + ((u >> np.uint64(45)) & np.uint64(1)))",
                           "(u + half + np.uint64(1))"),
}


def test_pins_pass_unmutated():
    for pin in PINS:
        pin()


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    fn_name, old, new = MUTATIONS[name]
    src = inspect.getsource(getattr(oracle, fn_name))
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    ns = dict(vars(oracle))
    exec(compile(src.replace(old, new), f"<mutated {fn_name}>", "exec"), ns)
    monkeypatch.setattr(oracle, fn_name, ns[fn_name])
    caught = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"mutation {name} passed every pin"
