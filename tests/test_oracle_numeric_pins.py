"""Pins for the oracle's numeric helpers, which every GPU parity verdict rests on.

* ``bf16_bits_to_f32`` widens bf16 bit patterns to fp32.  bf16 is the upper
  half of an IEEE-754 binary32 word, so the widening is exact; it is checked
  on all 65 536 patterns against torch's own bf16 -> fp32 conversion (an
  implementation that shares nothing with the oracle) and on hand-decoded
  values (sign, exponent and mantissa fields worked out from the IEEE
  format: 0x3F80 = 1.0, 0xC0A0 = -5.0, 0x0001 = 2^-133, 0x7F80 = +inf).
* ``rel_l2`` and ``max_abs_ratio`` (the acceptance measures of the
  element-wise parity bar) are checked on small arrays worked out by hand.
* Planted mistakes -- a shift by 15, a max|got| denominator, a missing
  square root, a missing absolute value -- fail these pins.
"""
import numpy as np
import pytest

from oracle import combine as oc


# ---- bf16 widening ------------------------------------------------------------

HAND_BF16 = [
    (0x3F80, 1.0),                 # sign 0, exponent 127, mantissa 0
    (0xC0A0, -5.0),                # sign 1, exponent 129, mantissa 0x20 -> -(1 + 1/4) * 4
    (0x0001, 2.0 ** -133),         # smallest subnormal: 2^-126 * 2^-7
    (0x7F80, np.inf),              # exponent all ones, mantissa 0
    (0xFF80, -np.inf),
    (0x8000, -0.0),
    (0x4049, 3.140625),            # 1.5703125 * 2: pi rounded down to 8 significant bits
    (0x3C00, 2.0 ** -7),
    (0x7F7F, (2 - 2.0 ** -7) * 2.0 ** 127),   # largest finite bf16
]


def _bf16_pins_hold(fn) -> bool:
    """True when fn widens every bf16 pattern exactly as torch does and
    gives the hand-decoded values."""
    import torch
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    got = np.asarray(fn(bits), dtype=np.float32)
    if got.shape != ref.shape:
        return False
    nan = np.isnan(ref)
    if not np.isnan(got[nan]).all():
        return False
    if not np.array_equal(got.view(np.uint32)[~nan], ref.view(np.uint32)[~nan]):
        return False
    for b, v in HAND_BF16:
        g = np.asarray(fn(np.array([b], dtype=np.uint16)), dtype=np.float32)[0]
        if g != np.float32(v) or np.signbit(g) != np.signbit(np.float32(v)):
            return False
    return True


def test_bf16_widening_matches_torch_and_hand_values():
    assert _bf16_pins_hold(oc.bf16_bits_to_f32)


def test_bf16_widening_keeps_shape_and_accepts_2d():
    bits = np.array([[0x3F80, 0xC0A0], [0x0000, 0x4000]], dtype=np.uint16)
    got = oc.bf16_bits_to_f32(bits)
    assert got.shape == (2, 2) and got.dtype == np.float32
    assert got.tolist() == [[1.0, -5.0], [0.0, 2.0]]


def _shift15(bits):
    b = np.ascontiguousarray(bits).view(np.uint16)
    return (b.astype(np.uint32) << np.uint32(15)).view(np.float32)


def _low_half(bits):
    b = np.ascontiguousarray(bits).view(np.uint16)
    return b.astype(np.uint32).view(np.float32)


def _sign_dropped(bits):
    b = np.ascontiguousarray(bits).view(np.uint16) & np.uint16(0x7FFF)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _value_cast(bits):
    # converts the integer value instead of reinterpreting the bits
    return np.ascontiguousarray(bits).view(np.uint16).astype(np.float32)


@pytest.mark.parametrize("mutant", [_shift15, _low_half, _sign_dropped, _value_cast])
def test_planted_bf16_mistakes_fail_the_pins(mutant):
    assert not _bf16_pins_hold(mutant)


# ---- acceptance measures --------------------------------------------------------

def _metric_pins_hold(rel_l2, max_abs_ratio) -> bool:
    """Hand-worked cases.

    rel_l2: got = [3, 5], ref = [3, 4]: |d| = 1, |ref| = 5 -> 0.2.
            got = [0, 0, 2, 0], ref = [1, 2, 2, 0]: |d| = sqrt(5), |ref| = 3
            -> sqrt(5)/3.  ref = 0: the bare norm of the difference.
    max_abs_ratio: got = [1, 2, 3], ref = [1, 2.5, 2]: max|d| = 1,
            max|ref| = 2.5 -> 0.4.  got = [-3, 1], ref = [-4, 1]: max|d| = 1,
            max|ref| = 4 -> 0.25.  ref = 0: the bare max difference.
    """
    cases_l2 = [
        (np.array([3.0, 5.0], np.float32), np.array([3.0, 4.0], np.float32), 0.2),
        (np.array([0.0, 0.0, 2.0, 0.0], np.float32), np.array([1.0, 2.0, 2.0, 0.0], np.float32),
         np.sqrt(5.0) / 3.0),
        (np.array([[3.0, 4.0]], np.float32), np.zeros((1, 2), np.float32), 5.0),
        (np.array([[1.0, -2.0], [2.0, 4.0]], np.float32),
         np.array([[1.0, -2.0], [2.0, 4.0]], np.float32), 0.0),
    ]
    cases_max = [
        (np.array([1.0, 2.0, 3.0], np.float32), np.array([1.0, 2.5, 2.0], np.float32), 0.4),
        (np.array([-3.0, 1.0], np.float32), np.array([-4.0, 1.0], np.float32), 0.25),
        (np.array([[0.5, -0.25]], np.float32), np.zeros((1, 2), np.float32), 0.5),
        (np.array([[7.0, 1.0], [1.0, 1.0]], np.float32),
         np.array([[8.0, 1.0], [1.0, -16.0]], np.float32), 17.0 / 16.0),
    ]
    for got, ref, want in cases_l2:
        if abs(rel_l2(got, ref) - want) > 1e-12 * max(1.0, want):
            return False
    for got, ref, want in cases_max:
        if abs(max_abs_ratio(got, ref) - want) > 1e-12 * max(1.0, want):
            return False
    return True


def test_acceptance_measures_on_hand_worked_arrays():
    assert _metric_pins_hold(oc.rel_l2, oc.max_abs_ratio)


def test_acceptance_measures_are_symmetric_in_sign_and_scale_free():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((17, 9)).astype(np.float32)
    got = ref + 1e-3 * rng.standard_normal(ref.shape).astype(np.float32)
    for s in (2.0, 0.5, -1.0):   # powers of two: exact in fp32
        assert oc.rel_l2(s * got, s * ref) == pytest.approx(oc.rel_l2(got, ref), rel=1e-12)
        assert oc.max_abs_ratio(s * got, s * ref) == pytest.approx(
            oc.max_abs_ratio(got, ref), rel=1e-12)


def _max_over_got(got, ref):
    m = float(np.abs(got).max())
    d = float(np.abs(got.astype(np.float64) - ref).max())
    return d / m if m > 0 else d


def _max_without_abs(got, ref):
    m = float(ref.max())
    d = float(np.abs(got.astype(np.float64) - ref).max())
    return d / m if m > 0 else d


def _mean_diff(got, ref):
    m = float(np.abs(ref).max())
    d = float(np.abs(got.astype(np.float64) - ref).mean())
    return d / m if m > 0 else d


def _l2_no_sqrt(got, ref):
    ref64 = ref.astype(np.float64)
    den = float(np.sum(ref64 ** 2))
    num = float(np.sum((got.astype(np.float64) - ref64) ** 2))
    return num / den if den > 0 else num


def _l2_over_got(got, ref):
    g64 = got.astype(np.float64)
    den = np.linalg.norm(g64)
    num = np.linalg.norm(g64 - ref.astype(np.float64))
    return float(num / den) if den > 0 else float(num)


@pytest.mark.parametrize("rel,mab", [
    (oc.rel_l2, _max_over_got),
    (oc.rel_l2, _max_without_abs),
    (oc.rel_l2, _mean_diff),
    (_l2_no_sqrt, oc.max_abs_ratio),
    (_l2_over_got, oc.max_abs_ratio),
])
def test_planted_metric_mistakes_fail_the_pins(rel, mab):
    assert not _metric_pins_hold(rel, mab)


def test_tolerances_are_the_stated_bar():
    # rel-L2 <= 5e-3 and max|d| <= 1e-2 max|ref| for bf16 inputs, fp32 accumulation
    assert oc.REL_L2_TOL == 5e-3
    assert oc.MAX_ABS_TOL == 1e-2
