"""Pins for the oracle's storage rounding (Sec. 3.2 formats; Remark after
Thm thm:matrix_rank_compensation: factors rounded individually).

The oracle's binary16 rounding is hand-written bit arithmetic; it is pinned
bit-for-bit against numpy's float64 -> float16 cast (a direct, correctly
rounded conversion) and against exact cases derived from the format
definition (11 significand bits, 5 exponent bits, ties to even)."""
import numpy as np
import pytest

import oracle as O


def _corpus():
    rng = np.random.default_rng([12969, 99, 0])
    parts = [rng.standard_normal(20000) * 10.0 ** rng.uniform(-9, 4.8, 20000)]
    # exact ties and near ties around binary16 quanta at many exponents
    e = np.arange(-24, 16, dtype=np.float64)
    base = 2.0 ** e
    for frac in (1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, 1.5 + 2.0 ** -11,
                 1.0 + 2.0 ** -11 + 2.0 ** -40, 1.0 + 2.0 ** -11 - 2.0 ** -40,
                 1.0 - 2.0 ** -12, 1.999):
        parts.append(base * frac)
    # subnormal range and its boundary
    q = 2.0 ** -24
    parts.append(np.array([q * 0.5, q * 1.5, q * 2.5, q * 0.49, q * 1023.5, q * 1024.0,
                           2.0 ** -14 * (1 - 2.0 ** -12), 2.0 ** -14, 1e-30, 0.0, -0.0]))
    # top of the range (65504 is the largest finite value)
    parts.append(np.array([65504.0, 65503.0, 65519.99, 65519.999999, 60000.0]))
    x = np.concatenate(parts)
    return np.concatenate([x, -x])


def test_f16_bitwise_matches_numpy_cast():
    x = _corpus()
    ours = O.round_to(x, "fp16", allow_overflow=True)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16)
    assert ours.dtype == np.float16
    np.testing.assert_array_equal(ours.view(np.uint16), ref.view(np.uint16))


def test_f32_bitwise_matches_numpy_cast():
    rng = np.random.default_rng([12969, 99, 1])
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.uniform(-40, 38, 20000),
                        np.array([0.0, -0.0, 1.0 + 2.0 ** -24, 1.0 + 3 * 2.0 ** -24, 1e-45, 1.5e-45])])
    ours = O.round_to(x, "fp32")
    np.testing.assert_array_equal(ours.view(np.uint32), x.astype(np.float32).view(np.uint32))


def test_f16_single_rounding_not_double():
    # 1 + 2^-11 + 2^-40 lies just above the midpoint of 1 and 1 + 2^-10, so a
    # single rounding gives 1 + 2^-10.  Rounding first to binary32 lands
    # exactly on the midpoint (2^-40 is below half a binary32 ulp) and the
    # second rounding then ties to even, 1.0.
    x = np.array([1.0 + 2.0 ** -11 + 2.0 ** -40])
    assert float(O.widen(O.round_to(x, "fp16"))[0]) == 1.0 + 2.0 ** -10
    via32 = np.float16(np.float32(x[0]))
    assert float(via32) == 1.0


def test_f16_ties_to_even_and_subnormals():
    cases = {
        1.0 + 2.0 ** -11: 1.0,                       # tie -> even mantissa 0
        1.0 + 3 * 2.0 ** -11: 1.0 + 2.0 ** -9,       # tie -> even mantissa 2
        2.0 ** -24 * 0.5: 0.0,                       # tie at the bottom -> 0
        2.0 ** -24 * 1.5: 2.0 ** -23,                # tie between 1 and 2 quanta -> 2
        2.0 ** -24 * 2.5: 2.0 ** -23,                # tie between 2 and 3 -> 2
        2.0 ** -24 * 1023.5: 2.0 ** -14,             # rounds up into the normal range
        65519.99: 65504.0,
    }
    x = np.array(list(cases.keys()))
    got = O.widen(O.round_to(x, "fp16"))
    np.testing.assert_array_equal(got, np.array(list(cases.values())))


def test_f16_overflow_flagged():
    with pytest.raises(O.OverflowInRounding):
        O.round_to(np.array([65520.0]), "fp16")
    got = O.round_to(np.array([65520.0, -1e6]), "fp16", allow_overflow=True)
    assert np.isinf(got[0]) and got[0] > 0 and np.isinf(got[1]) and got[1] < 0


def test_rounding_is_odd_symmetric():
    # fl(-x) = -fl(x): the reason the SVD sign choice cannot change eta
    x = _corpus()
    for prec in ("fp32", "fp16"):
        a = O.widen(O.round_to(x, prec, allow_overflow=True))
        b = O.widen(O.round_to(-x, prec, allow_overflow=True))
        np.testing.assert_array_equal(a, -b)


def test_widen_is_exact():
    bits = np.arange(0, 0x7C00, dtype=np.uint16)     # every finite non-negative binary16
    h = bits.view(np.float16)
    np.testing.assert_array_equal(O.widen(h), h.astype(np.float64))
    # and rounding the widened value gives the same bits back
    np.testing.assert_array_equal(O.round_to(O.widen(h), "fp16").view(np.uint16), bits)


def test_unit_roundoff_bound():
    # |fl(x) - x| <= u |x| with u = 2^-p (Sec. 3.2-3.3, eq. fl_op_model), p = 11
    # for binary16 and 24 for binary32, in the normal range
    rng = np.random.default_rng([12969, 99, 2])
    x = rng.uniform(1e-3, 6e4, 50000) * np.sign(rng.standard_normal(50000))
    for prec, p in (("fp16", 11), ("fp32", 24)):
        err = np.abs(O.widen(O.round_to(x, prec)) - x)
        assert np.all(err <= 2.0 ** -p * np.abs(x))
